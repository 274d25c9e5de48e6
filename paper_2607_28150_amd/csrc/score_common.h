// Shared pieces of the score kernels: MFMA operand fragments, the K-tile
// stager and the query-fragment loader (gfx950).
#pragma once

#include "sg_internal.h"

namespace sg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int SC_TK = 64;          // keys per tile
constexpr int SC_TPC = 16;         // tiles per chunk
constexpr int SC_CHUNK = SC_TK * SC_TPC;
constexpr int SC_MAXR = 512;       // rows per unit (G * W): at most 8 wavefronts
constexpr float SC_LOG2E = 1.4426950408889634f;
constexpr float SC_LN2 = 0.6931471805599453f;

template <typename T, int D>
struct Frag;

template <int D>
struct Frag<uint16_t, D> {  // bfloat16 operands, K = 32 per instruction
    static constexpr int KSTEPS = D / 32;
    static constexpr int ROWB = D * 2 + 16;  // padded LDS row bytes
    using A = bf16x8;
    __device__ static A zero() { return A{}; }
    __device__ static A load_global(const uint16_t *row, int ks, int lane) {
        return *reinterpret_cast<const A *>(row + ks * 32 + 8 * (lane / 16));
    }
    __device__ static A load_lds(const char *tile, int key, int ks, int lane) {
        return *reinterpret_cast<const A *>(tile + key * ROWB + (ks * 32 + 8 * (lane / 16)) * 2);
    }
    __device__ static f32x4 mma(const A &a, const A &b, const f32x4 &c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

template <int D>
struct Frag<float, D> {  // fp32 operands, K = 4 per instruction
    static constexpr int KSTEPS = D / 4;
    static constexpr int ROWB = D * 4 + 16;
    using A = float;
    __device__ static A zero() { return 0.f; }
    __device__ static A load_global(const float *row, int ks, int lane) { return row[ks * 4 + lane / 16]; }
    __device__ static A load_lds(const char *tile, int key, int ks, int lane) {
        return *reinterpret_cast<const float *>(tile + key * ROWB + (ks * 4 + lane / 16) * 4);
    }
    __device__ static f32x4 mma(const A &a, const A &b, const f32x4 &c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
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

// Stage one 64-key tile of K (rows [key0, key0+64) of the unit) into LDS.
template <typename T, int D>
__device__ __forceinline__ void stage_tile(char *tile, const T *kunit, int64_t key0, int64_t N) {
    constexpr int ESZ = sizeof(T);
    constexpr int VPR = D * ESZ / 16;  // 16-byte vectors per key row
    for (int i = threadIdx.x; i < SC_TK * VPR; i += blockDim.x) {
        const int key = i / VPR, v = i % VPR;
        v4u x = v4u{0u, 0u, 0u, 0u};
        if (key0 + key < N) x = reinterpret_cast<const v4u *>(kunit + (key0 + key) * D)[v];
        *reinterpret_cast<v4u *>(tile + key * Frag<T, D>::ROWB + v * 16) = x;
    }
}

// acc[rb][kb] = Q(rows of row-block rb) . K(tile keys of key-block kb); the
// first k-step multiplies with a zero accumulator operand (no separate clear)
template <typename T, int D>
__device__ __forceinline__ void tile_mma(const typename Frag<T, D>::A (&qa)[4][Frag<T, D>::KSTEPS],
                                         const char *tile, int lane, f32x4 (&acc)[4][4]) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        const auto bf = Frag<T, D>::load_lds(tile, kb * 16 + lane % 16, 0, lane);
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) acc[rb][kb] = Frag<T, D>::mma(qa[rb][0], bf, f32x4{0.f, 0.f, 0.f, 0.f});
    }
#pragma unroll
    for (int ks = 1; ks < Frag<T, D>::KSTEPS; ++ks) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            const auto bf = Frag<T, D>::load_lds(tile, kb * 16 + lane % 16, ks, lane);
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) acc[rb][kb] = Frag<T, D>::mma(qa[rb][ks], bf, acc[rb][kb]);
        }
    }
}

template <typename T, int D>
__device__ __forceinline__ void load_q(const T *qunit, int R, int wave, int lane,
                                       typename Frag<T, D>::A (&qa)[4][Frag<T, D>::KSTEPS]) {
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
        const int r = wave * 64 + rb * 16 + lane % 16;
#pragma unroll
        for (int ks = 0; ks < Frag<T, D>::KSTEPS; ++ks)
            qa[rb][ks] = r < R ? Frag<T, D>::load_global(qunit + (int64_t)r * D, ks, lane) : Frag<T, D>::zero();
    }
}


}  // namespace sg
