// Shared pieces of the score kernels: MFMA tile traits, work mapping and the
// LDS K tiles (gfx950).
#pragma once

#include "sg_internal.h"

namespace sg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int SC_CHUNK = 2048;     // keys per workgroup
constexpr int SC_MAXR = 512;       // rows per unit (G * W): at most 8 wavefronts
constexpr float SC_LOG2E = 1.4426950408889634f;
constexpr float SC_LN2 = 0.6931471805599453f;

typedef float f32x16 __attribute__((ext_vector_type(16)));

// MFMA tile traits.  bf16 runs v_mfma_f32_32x32x16_bf16 (32 x 32 outputs, 16
// products per instruction and output; on gfx950 its issue overlaps the
// exponential / add work of the score passes far better than the 16x16x32
// form); fp32 runs v_mfma_f32_16x16x4_f32.
//
// For both operand slots a lane holds row (or column) lane % BM and the
// contraction slice ks of its lane group, so the same registers serve as A
// or B: mma(Q, K) gives C[row][key], mma(K, Q) gives C[key][row].  Output
// register v of a lane holds C[crow(v, lane)][lane % BM].
template <typename T, int D>
struct MT;

template <int D>
struct MT<uint16_t, D> {
    static constexpr int BM = 32;                 // rows (and columns) of one output tile
    static constexpr int KS = D / 16;             // instructions per contraction
    static constexpr int NV = 16;                 // outputs per lane
    static constexpr int ROWB = D * 2 + 16;       // padded LDS row bytes (conflict-free column reads)
    using A = bf16x8;
    using C = f32x16;
    __device__ static int crow(int v, int lane) { return 8 * (v / 4) + 4 * (lane / 32) + v % 4; }
    __device__ static A load_global(const uint16_t *row, int ks, int lane) {
        return *reinterpret_cast<const A *>(row + ks * 16 + 8 * (lane / 32));
    }
    __device__ static A load_lds(const char *img, int row, int ks, int lane) {
        return *reinterpret_cast<const A *>(img + row * ROWB + (ks * 16 + 8 * (lane / 32)) * 2);
    }
    __device__ static C mma(const A &a, const A &b, const C &c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
    __device__ static C zero() { return C{}; }
};

template <int D>
struct MT<float, D> {
    static constexpr int BM = 16;
    static constexpr int KS = D / 4;
    static constexpr int NV = 4;
    static constexpr int ROWB = D * 4 + 16;
    using A = float;
    using C = f32x4;
    __device__ static int crow(int v, int lane) { return 4 * (lane / 16) + v; }
    __device__ static A load_global(const float *row, int ks, int lane) { return row[ks * 4 + lane / 16]; }
    __device__ static A load_lds(const char *img, int row, int ks, int lane) {
        return *reinterpret_cast<const float *>(img + row * ROWB + (ks * 4 + lane / 16) * 4);
    }
    __device__ static C mma(const A &a, const A &b, const C &c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    __device__ static C zero() { return C{}; }
};

// Workgroup -> (unit, chunk).  Workgroups are dealt to the 8 XCDs round-robin
// by their linear id; this mapping gives the chunks of one unit consecutive
// slots on one XCD, so the unit's queries are fetched into that XCD's L2 once.
__device__ __forceinline__ void unit_chunk(int64_t units, int nchunk, int64_t &u, int &c) {
    const int64_t id = blockIdx.x;
    const int64_t total = units * nchunk;
    const int64_t full = total / 8 * 8;        // ids in the XCD-interleaved part
    if (id < full) {
        const int64_t xcd = id % 8, j = id / 8;          // j-th workgroup of this XCD
        const int64_t lin = xcd * (full / 8) + j;       // contiguous range per XCD
        u = lin / nchunk;
        c = (int)(lin % nchunk);
    } else {
        u = id / nchunk;
        c = (int)(id % nchunk);
    }
}

struct UnitGeom {
    int b, l, h;
    int64_t s0, N;
};

__device__ __forceinline__ UnitGeom unit_geom(int64_t u, int B, int Hkv, const int32_t *cu_seqlens, int64_t T) {
    UnitGeom g;
    g.b = (int)(u % B);
    const int64_t lh = u / B;
    g.l = (int)(lh / Hkv);
    g.h = (int)(lh % Hkv);
    const int64_t s0 = cu_seqlens[g.b], s1 = cu_seqlens[g.b + 1];
    g.s0 = s0;
    g.N = (s0 >= 0 && s1 >= s0 && s1 <= T) ? s1 - s0 : 0;
    return g;
}

// Direct global->LDS load as dma16, addressed by a wavefront-uniform base in
// scalar registers and a 32-bit per-lane offset.  The base reaches the
// instruction in scalar registers only in an optimising compile (readfirstlane
// results stay scalar there); an unoptimised device compile (the sanitised
// library for host-side checks) keeps the 64-bit form.
#if defined(__OPTIMIZE__)
constexpr bool SC_SCALAR_BASE = true;
#else
constexpr bool SC_SCALAR_BASE = false;
#endif
__device__ __forceinline__ void dma16_sbase(const char *base, unsigned off, unsigned lds) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "{m0}"(lds) : "memory");
}

// K tiles in LDS.  A tile is TK keys of D elements, stored without padding;
// the 16-byte vector v of key j sits at slot j * VPR + (v ^ (j % VPR)), so the
// 32 (or 16) lanes reading one fragment column hit distinct banks.  Tiles
// arrive through direct global->LDS loads (lane i of an instruction lands at
// base + 16 i; the swizzle is applied to the global address each lane reads).
template <typename T, int D, int TKEYS = (sizeof(T) == 2 ? 128 : 64)>
struct KTile {
    static constexpr int VPR = D * (int)sizeof(T) / 16;          // 16-byte vectors per key
    static constexpr int TK = TKEYS;                              // keys per tile
    static constexpr int BYTES = TK * VPR * 16;
    static constexpr int NKB = TK / MT<T, D>::BM;                 // key blocks per tile

    // Issue the loads of keys [key0, key0 + TK) (clamped to the prompt's last
    // key) into `buf`; the NW wavefronts share the work.  Completion is tracked
    // by the vector memory counter of the issuing wavefront.
    template <int NW>
    __device__ static void load(char *buf, const T *kunit, int key0, int N, int wave, int lane) {
        constexpr int KPI = 64 / VPR;                              // keys per instruction
        constexpr int KPW = TK / NW;                               // keys per wavefront
        static_assert(KPW % KPI == 0, "tile keys must split evenly over the wavefronts");
        // recompute the per-lane offsets at every call instead of keeping them
        // live across the caller's loop (registers are the scarce resource)
        asm volatile("" : "+v"(lane));
        const unsigned kl = (unsigned)lane / VPR, vl = (unsigned)lane % VPR;
        const char *tb = reinterpret_cast<const char *>(kunit) + (int64_t)key0 * (VPR * 16);   // wavefront-uniform
        if constexpr (sizeof(T) == 2 && SC_SCALAR_BASE && KPW % VPR == 0) {
            // A whole bf16 tile: every wavefront's first key is a multiple of VPR
            // and the swizzle repeats every PER instructions, so the lane's 32-bit
            // offsets of PER instructions serve them all, each instruction taking
            // a wavefront-uniform base in scalar registers (no 64-bit address
            // arithmetic per lane and instruction).
            static_assert(KPW % VPR == 0 && (VPR % KPI == 0 || KPI % VPR == 0), "swizzle period");
            constexpr int NI = KPW / KPI, PER0 = VPR % KPI == 0 ? VPR / KPI : 1, PER = PER0 < NI ? PER0 : NI;
            if (key0 + TK <= N) {
                unsigned off[PER];
#pragma unroll
                for (int p = 0; p < PER; ++p)
                    off[p] = (p * KPI + kl) * (VPR * 16) + ((vl ^ ((p * KPI + kl) % VPR)) << 4);
                // the base is uniform by construction; readfirstlane puts it in the
                // scalar registers the instruction form requires
                const uint64_t b0 = reinterpret_cast<uint64_t>(tb + (int64_t)wave * KPW * (VPR * 16));
                const uint64_t sb = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(b0 >> 32)) << 32) |
                                    (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b0);
#pragma unroll
                for (int j = 0; j < NI; ++j) {
                    const char *base = reinterpret_cast<const char *>(sb + (uint64_t)((j / PER) * PER * KPI * VPR * 16));
                    dma16_sbase(base, off[j % PER], lds_addr(buf + (wave * KPW + j * KPI) * VPR * 16));
                }
                return;
            }
        }
        // the last key of the prompt relative to key0: keys past it read it instead
        const unsigned last = (unsigned)max(0, min(TK - 1, N - 1 - key0));
        const bool whole = key0 + TK <= N;
#pragma unroll
        for (int j = 0; j < KPW / KPI; ++j) {
            const unsigned key = (unsigned)(wave * KPW + j * KPI) + kl;
            const unsigned v = vl ^ (key % VPR);
            const unsigned row = whole ? key : min(key, last);
            dma16(tb + (row * (VPR * 16) + v * 16), lds_addr(buf + (wave * KPW + j * KPI) * VPR * 16));
        }
    }

    // Operand fragment (key block kb, contraction slice ks) of a lane.
    __device__ static typename MT<T, D>::A frag(const char *buf, int kb, int ks, int lane) {
        using M = MT<T, D>;
        const int key = kb * M::BM + lane % M::BM;
        if constexpr (sizeof(T) == 2) {
            const int v = ks * 2 + lane / 32;                     // elements ks * 16 + 8 * (lane / 32) ..
            return *reinterpret_cast<const typename M::A *>(buf + (key * VPR + (v ^ (key % VPR))) * 16);
        } else {
            const int e = ks * 4 + lane / 16;                     // element of the key row
            const int v = e / 4;
            return *reinterpret_cast<const float *>(buf + (key * VPR + (v ^ (key % VPR))) * 16 + (e % 4) * 4);
        }
    }
};

// Workgroup barrier after this wavefront's LDS operations and vector memory
// operations (direct LDS loads included) have completed.  The asm's memory
// clobber keeps the compiler from moving memory accesses across it.
__device__ __forceinline__ void barrier_after_loads() {
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace sg
