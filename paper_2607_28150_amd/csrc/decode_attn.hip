// sg_decode_attn: GQA decode attention over a partial, page-addressed KV set.
//
// Grid: x = (sequence, KV head) unit, y = split of the unit's rows (one split
// whenever there are at least as many units as compute units).  A workgroup
// of WAVES wavefronts serves all G q heads of the group, so each K/V row is
// read from HBM once per step.  Wavefront w walks 32-row sub-tiles w,
// w + WAVES, ...; within a sub-tile CPR = 16 / esize * d / 16 lanes cover one
// row with one 16-byte vector each (fully coalesced K and V loads), and a
// wavefront step covers 64 / CPR rows.  Per sub-tile:
//   logits : each lane dots its slice of q (held in registers) with its K
//            slice (v_dot2_f32_bf16 for bf16, fp32 accumulation); DPP adds sum
//            the partials over the row's lanes;
//   softmax: online, with a wavefront-uniform running max m (exp2 with
//            log2(e) folded into the scale); the sums l and the outputs o stay
//            per-lane partials rescaled by the same factor, reduced once at
//            the end, so only the max crosses lanes per sub-tile;
//   values : each lane accumulates its V slice weighted by the row's
//            probability for the G heads in fp32.
// The wavefronts' (m, l, o) are merged through LDS at the end.  With one split
// the normalised output is written directly; otherwise the split's state goes
// to the workspace and a merge kernel combines the splits in a fixed order.
// All reductions have a fixed order, so results are deterministic.
#include "sg_internal.h"

namespace sg {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// reinterpret a 32-bit word as two bf16 lanes (element 0 = low half); a copy
// through a local word, not a bit_cast of a vector element
__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t w) {
    bf16x2 r;
    __builtin_memcpy(&r, &w, sizeof(r));
    return r;
}

// partial dot product of one 16-byte slice of q with the same slice of a K row
template <typename T>
struct SliceDot;
template <>
struct SliceDot<uint16_t> {   // bf16: four v_dot2_f32_bf16, fp32 accumulation
    __device__ static float run(const v4u &q, const v4u &k) {
        float a = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.x), as_bf16x2(k.x), 0.f, false);
        float b = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.y), as_bf16x2(k.y), 0.f, false);
        a = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.z), as_bf16x2(k.z), a, false);
        b = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.w), as_bf16x2(k.w), b, false);
        return a + b;
    }
};
template <>
struct SliceDot<float> {
    __device__ static float run(const v4u &q, const v4u &k) {
        float a = __uint_as_float(q.x) * __uint_as_float(k.x);
        float b = __uint_as_float(q.y) * __uint_as_float(k.y);
        a = fmaf(__uint_as_float(q.z), __uint_as_float(k.z), a);
        b = fmaf(__uint_as_float(q.w), __uint_as_float(k.w), b);
        return a + b;
    }
};

template <typename T>
struct Elem;
template <>
struct Elem<float> {
    static constexpr int PER16 = 4;
    __device__ static void unpack(const v4u &w, float *x) {
        x[0] = __uint_as_float(w.x); x[1] = __uint_as_float(w.y);
        x[2] = __uint_as_float(w.z); x[3] = __uint_as_float(w.w);
    }
};
template <>
struct Elem<uint16_t> {  // bfloat16 bits
    static constexpr int PER16 = 8;
    __device__ static void unpack(const v4u &w, float *x) {
        x[0] = bf16_lo(w.x); x[1] = bf16_hi(w.x); x[2] = bf16_lo(w.y); x[3] = bf16_hi(w.y);
        x[4] = bf16_lo(w.z); x[5] = bf16_hi(w.z); x[6] = bf16_lo(w.w); x[7] = bf16_hi(w.w);
    }
};

template <int G>
struct DecodeShape {
    // wavefronts per workgroup: sixteen (four per SIMD at <= 128 registers)
    // keep enough loads in flight per CU; more heads need more accumulators
    // and LDS for the final merge, so fewer wavefronts
    static constexpr int WAVES = G <= 4 ? 16 : (G == 8 ? 8 : 4);
    // rows per wavefront sub-tile (register budget: K, V slices and logits)
    static constexpr int SUB = G <= 2 ? 32 : 16;
    static constexpr int64_t ROWS_PER_PASS = (int64_t)SUB * WAVES;
};

// partial state of one split: per head (m, l) then o[d]
__device__ __forceinline__ float *part_ptr(float *ws, int64_t unit, int nsplit, int split, int G, int d) {
    return ws + ((unit * nsplit + split) * G) * (int64_t)(d + 2);
}

// DPP lane moves (gfx9 encodings): quad_perm, row rotate, row half-mirror
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int DPP_XOR1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int DPP_XOR2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141;
constexpr int DPP_ROR4 = 0x124;
constexpr int DPP_ROR8 = 0x128;

// sum over each group of N consecutive lanes (N = 8, 16 or 32); every lane of
// the group receives the group's sum
template <int N>
__device__ __forceinline__ float group_sum(float x) {
    x += dpp<DPP_XOR1>(x);
    x += dpp<DPP_XOR2>(x);
    if constexpr (N == 8) {
        x += dpp<DPP_HALF_MIRROR>(x);
    } else {
        x += dpp<DPP_ROR4>(x);
        x += dpp<DPP_ROR8>(x);
        if constexpr (N == 32) x += __shfl_xor(x, 16, 64);
    }
    return x;
}

template <typename T, int D, int G, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void decode_kernel(
    int Hq, int Hkv, float scale_log2, const T *__restrict__ q, const v4u *__restrict__ k_pool,
    const v4u *__restrict__ v_pool, int64_t pool_rows, const int32_t *__restrict__ page_table,
    const int32_t *__restrict__ n_rows, int page_size, int page_shift, int max_pages, int64_t split_rows,
    float *__restrict__ out, float *__restrict__ ws) {
    constexpr int PER16 = Elem<T>::PER16;  // elements per 16-byte vector
    constexpr int CPR = D / PER16;         // lanes per row (one vector each)
    constexpr int RPS = 64 / CPR;          // rows per wavefront step
    constexpr int SUB = DecodeShape<G>::SUB;
    constexpr int STEPS = SUB / RPS;       // steps per sub-tile
    __shared__ float m_s[WAVES][G], l_s[WAVES][G];
    __shared__ float o_s[WAVES][G][D];

    const int64_t unit = blockIdx.x;        // b * Hkv + h
    const int b = (int)(unit / Hkv), h = (int)(unit % Hkv);
    const int split = blockIdx.y, nsplit = gridDim.y;
    const int tid = threadIdx.x, lane = tid % 64;
    const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
    const int cg = lane % CPR, rsub = lane / CPR;
    int64_t n = n_rows[unit];
    n = max<int64_t>(0, min<int64_t>(n, (int64_t)max_pages * page_size));
    const int64_t r0 = (int64_t)split * split_rows;
    const int64_t r1 = min<int64_t>(n, r0 + split_rows);
    const int32_t *pt = page_table + unit * max_pages;

    // this lane's 16-byte slice (vector cg) of each of the G query vectors
    v4u qs[G];
    {
        const v4u *qv = reinterpret_cast<const v4u *>(q + ((int64_t)b * Hq + (int64_t)h * G) * D);
#pragma unroll
        for (int g = 0; g < G; ++g) qs[g] = qv[g * CPR + cg];
    }
    // running state: m is wavefront-uniform; l and o are per-lane partials
    // (over the rows this lane visits) and are reduced at the end
    float m[G], l[G], o[G][PER16];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        m[g] = -INFINITY;
        l[g] = 0.f;
#pragma unroll
        for (int e = 0; e < PER16; ++e) o[g][e] = 0.f;
    }

    for (int64_t t0 = r0 + (int64_t)wave * SUB; t0 < r1; t0 += (int64_t)SUB * WAVES) {
        int prow[STEPS];
        v4u kv[STEPS], vv[STEPS];
#pragma unroll
        for (int st = 0; st < STEPS; ++st) {
            // logical rows fit in 31 bits and pool rows too (host checks)
            const int lr = (int)(t0 + st * RPS + rsub);
            int pr = -1;
            if (lr < r1) {
                const int pg = page_shift >= 0 ? (lr >> page_shift) : lr / page_size;
                const int64_t x = (int64_t)pt[pg] + (lr - pg * page_size);
                if (x >= 0 && x < pool_rows) pr = (int)x;
            }
            prow[st] = pr;
        }
#pragma unroll
        for (int st = 0; st < STEPS; ++st)
            kv[st] = prow[st] >= 0 ? k_pool[(int64_t)prow[st] * CPR + cg] : v4u{0u, 0u, 0u, 0u};
#pragma unroll
        for (int st = 0; st < STEPS; ++st)
            vv[st] = prow[st] >= 0 ? v_pool[(int64_t)prow[st] * CPR + cg] : v4u{0u, 0u, 0u, 0u};

        // logits: partial dot over this lane's vector, summed over the row's lanes
        float z[STEPS][G];
#pragma unroll
        for (int st = 0; st < STEPS; ++st) {
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const float a = group_sum<CPR>(SliceDot<T>::run(qs[g], kv[st]));
                z[st][g] = prow[st] >= 0 ? a * scale_log2 : -INFINITY;
            }
        }
        // online softmax with a wavefront-wide running max
#pragma unroll
        for (int g = 0; g < G; ++g) {
            float mx = z[0][g];
#pragma unroll
            for (int st = 1; st < STEPS; ++st) mx = fmaxf(mx, z[st][g]);
#pragma unroll
            for (int off = CPR; off < 64; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
            const float mn = fmaxf(m[g], mx);
            if (mn == -INFINITY) continue;            // nothing usable yet (uniform)
            const float alpha = __builtin_amdgcn_exp2f(m[g] - mn);
            m[g] = mn;
            float ls = 0.f;
#pragma unroll
            for (int st = 0; st < STEPS; ++st) {
                z[st][g] = __builtin_amdgcn_exp2f(z[st][g] - mn);   // z now holds p
                ls += z[st][g];
            }
            l[g] = l[g] * alpha + ls;
#pragma unroll
            for (int e = 0; e < PER16; ++e) o[g][e] *= alpha;
        }
        // values
#pragma unroll
        for (int st = 0; st < STEPS; ++st) {
            float x[PER16];
            Elem<T>::unpack(vv[st], x);
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const float p = m[g] == -INFINITY ? 0.f : z[st][g];
#pragma unroll
                for (int e = 0; e < PER16; ++e) o[g][e] = fmaf(p, x[e], o[g][e]);
            }
        }
    }
    // reduce l and o over the row groups of the wavefront (lanes sharing cg)
#pragma unroll
    for (int off = CPR; off < 64; off <<= 1)
#pragma unroll
        for (int g = 0; g < G; ++g) {
            l[g] += __shfl_xor(l[g], off, 64);
#pragma unroll
            for (int e = 0; e < PER16; ++e) o[g][e] += __shfl_xor(o[g][e], off, 64);
        }
    if (rsub == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < PER16; ++e) o_s[wave][g][cg * PER16 + e] = o[g][e];
    }
    if (lane == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) { m_s[wave][g] = m[g]; l_s[wave][g] = l[g]; }
    }
    __syncthreads();

    // combine the wavefronts; thread t handles (g, c) pairs
    for (int i = tid; i < G * D; i += 64 * WAVES) {
        const int g = i / D, c = i % D;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) M = fmaxf(M, m_s[w][g]);
        float Lsum = 0.f, O = 0.f;
        if (M > -INFINITY) {
#pragma unroll
            for (int w = 0; w < WAVES; ++w) {
                const float a = m_s[w][g] > -INFINITY ? __builtin_amdgcn_exp2f(m_s[w][g] - M) : 0.f;
                Lsum += a * l_s[w][g];
                O += a * o_s[w][g][c];
            }
        }
        if (nsplit == 1) {
            out[((int64_t)b * Hq + (int64_t)h * G + g) * D + c] = Lsum > 0.f ? O / Lsum : 0.f;
        } else {
            float *pp = part_ptr(ws, unit, nsplit, split, G, D) + (int64_t)g * (D + 2);
            if (c == 0) { pp[0] = M; pp[1] = Lsum; }
            pp[2 + c] = O;
        }
    }
}

template <int D, int G>
__global__ __launch_bounds__(256) void decode_merge_kernel(int Hq, int Hkv, int nsplit, const float *__restrict__ ws,
                                                          float *__restrict__ out) {
    const int64_t unit = blockIdx.x;
    const int b = (int)(unit / Hkv), h = (int)(unit % Hkv);
    float *w = const_cast<float *>(ws);
    for (int i = threadIdx.x; i < G * D; i += 256) {
        const int g = i / D, c = i % D;
        float M = -INFINITY;
        for (int s = 0; s < nsplit; ++s) M = fmaxf(M, part_ptr(w, unit, nsplit, s, G, D)[g * (D + 2)]);
        float Lsum = 0.f, O = 0.f;
        if (M > -INFINITY) {
            for (int s = 0; s < nsplit; ++s) {
                const float *pp = part_ptr(w, unit, nsplit, s, G, D) + (int64_t)g * (D + 2);
                if (pp[0] > -INFINITY) {
                    const float a = __builtin_amdgcn_exp2f(pp[0] - M);
                    Lsum += a * pp[1];
                    O += a * pp[2 + c];
                }
            }
        }
        out[((int64_t)b * Hq + (int64_t)h * G + g) * D + c] = Lsum > 0.f ? O / Lsum : 0.f;
    }
}

static int device_cus() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0, v = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
            cus = v;
        else
            cus = 256;
    }
    return cus;
}

template <int G>
static int max_splits(int64_t max_rows) {
    return (int)std::max<int64_t>(1, ceil_div(max_rows, DecodeShape<G>::ROWS_PER_PASS));
}

template <typename T, int D, int G>
static int launch_decode(hipStream_t s, int B, int Hq, int Hkv, float scale_log2, const void *q, const void *k_pool,
                         const void *v_pool, int64_t pool_rows, const int32_t *page_table, const int32_t *n_rows,
                         int page_size, int max_pages, float *out, float *ws, size_t ws_bytes) {
    constexpr int WAVES = DecodeShape<G>::WAVES;
    const int64_t units = (int64_t)B * Hkv;
    const int64_t max_rows = (int64_t)max_pages * page_size;
    const int cap = max_splits<G>(max_rows);
    int nsplit = 1;
    if (units < device_cus()) nsplit = (int)std::min<int64_t>(cap, ceil_div(device_cus(), units));
    const int64_t split_rows = ceil_div(ceil_div(max_rows, nsplit), 32) * 32;
    nsplit = (int)ceil_div(max_rows, split_rows);
    const size_t need = nsplit > 1 ? (size_t)units * nsplit * G * (D + 2) * sizeof(float) : 0;
    if (need > ws_bytes || (need && !ws)) {
        set_error("sg_decode_attn: workspace %zu < %zu", ws_bytes, need);
        return SG_EWORKSPACE;
    }
    // page sizes that are powers of two index with a shift (-1: divide)
    const int page_shift = (page_size & (page_size - 1)) == 0 ? __builtin_ctz((unsigned)page_size) : -1;
    dim3 grid((unsigned)units, (unsigned)nsplit);
    decode_kernel<T, D, G, WAVES><<<grid, 64 * WAVES, 0, s>>>(
        Hq, Hkv, scale_log2, reinterpret_cast<const T *>(q), reinterpret_cast<const v4u *>(k_pool),
        reinterpret_cast<const v4u *>(v_pool), pool_rows, page_table, n_rows, page_size, page_shift, max_pages,
        split_rows, out, ws);
    if (nsplit > 1) decode_merge_kernel<D, G><<<(unsigned)units, 256, 0, s>>>(Hq, Hkv, nsplit, ws, out);
    return launch_status("sg_decode_attn");
}

template <typename T, int D>
static int dispatch_g(int G, hipStream_t s, int B, int Hq, int Hkv, float sl2, const void *q, const void *kp,
                      const void *vp, int64_t pr, const int32_t *pt, const int32_t *nr, int ps, int mp, float *out,
                      float *ws, size_t wsb) {
    switch (G) {
        case 1: return launch_decode<T, D, 1>(s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, wsb);
        case 2: return launch_decode<T, D, 2>(s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, wsb);
        case 4: return launch_decode<T, D, 4>(s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, wsb);
        case 8: return launch_decode<T, D, 8>(s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, wsb);
        case 16: return launch_decode<T, D, 16>(s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, wsb);
        default: set_error("sg_decode_attn: group size %d not supported (1, 2, 4, 8, 16)", G); return SG_EUNSUPPORTED;
    }
}

}  // namespace sg

using namespace sg;

extern "C" size_t sg_decode_attn_workspace_size(int B, int Hq, int Hkv, int d, int max_pages, int page_size) {
    if (B <= 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv != 0 || d <= 0 || max_pages <= 0 || page_size <= 0) return 0;
    const int G = Hq / Hkv;
    const int64_t max_rows = (int64_t)max_pages * page_size;
    int cap = 1;
    switch (G) {
        case 1: cap = max_splits<1>(max_rows); break;
        case 2: cap = max_splits<2>(max_rows); break;
        case 4: cap = max_splits<4>(max_rows); break;
        case 8: cap = max_splits<8>(max_rows); break;
        default: cap = max_splits<16>(max_rows); break;
    }
    if (cap <= 1) return 0;
    return (size_t)B * Hkv * cap * G * (size_t)(d + 2) * sizeof(float);
}

extern "C" int sg_decode_attn(void *stream, sg_dtype dt, int B, int Hq, int Hkv, int d, float scale, const void *q,
                              const void *k_pool, const void *v_pool, int64_t pool_rows, const int32_t *page_table,
                              const int32_t *n_rows, int page_size, int max_pages, float *out, void *ws,
                              size_t ws_bytes) {
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "sg_decode_attn: unknown dtype %d", (int)dt);
    SG_REQUIRE(B >= 0 && Hq >= 1 && Hkv >= 1 && Hq % Hkv == 0, SG_EINVAL,
               "sg_decode_attn: need Hq %% Hkv == 0 (Hq=%d, Hkv=%d)", Hq, Hkv);
    SG_REQUIRE(d == 64 || d == 128, SG_EUNSUPPORTED, "sg_decode_attn: head dimension %d not supported", d);
    SG_REQUIRE(page_size >= 1 && max_pages >= 1 && pool_rows >= 0, SG_EINVAL, "sg_decode_attn: bad page geometry");
    SG_REQUIRE((int64_t)max_pages * page_size <= (1ll << 30), SG_EINVAL, "sg_decode_attn: page table too large");
    SG_REQUIRE(pool_rows <= 0x7fffffffll, SG_EUNSUPPORTED, "sg_decode_attn: pool above 2^31 rows");
    SG_REQUIRE(scale == scale && scale > 0.f, SG_EINVAL, "sg_decode_attn: scale must be positive");
    if (B == 0) return SG_OK;
    SG_REQUIRE(q && k_pool && v_pool && page_table && n_rows && out, SG_EINVAL, "sg_decode_attn: null pointer");
    SG_REQUIRE(aligned16(k_pool) && aligned16(v_pool) && aligned16(q), SG_EINVAL,
               "sg_decode_attn: q and pools must be 16-byte aligned");
    SG_REQUIRE((int64_t)B * Hkv <= 0x7fffffffll, SG_EINVAL, "sg_decode_attn: too many units");
    const float sl2 = scale * 1.4426950408889634f;  // log2(e)
    const int G = Hq / Hkv;
    hipStream_t s = as_stream(stream);
    float *w = reinterpret_cast<float *>(ws);
    if (dt == SG_F32) {
        if (d == 64) return dispatch_g<float, 64>(G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, ws_bytes);
        return dispatch_g<float, 128>(G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, ws_bytes);
    }
    if (d == 64) return dispatch_g<uint16_t, 64>(G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, ws_bytes);
    return dispatch_g<uint16_t, 128>(G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, ws_bytes);
}
