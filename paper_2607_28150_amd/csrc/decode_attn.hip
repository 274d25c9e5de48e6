// sg_decode_attn: GQA decode attention over a partial, page-addressed KV set.
//
// Grid: x = (sequence, KV head) unit, y = split of the unit's rows.  A 256-
// thread workgroup handles SPLIT = 256 rows of one unit for all G q heads of
// the group, so every K/V row is read from HBM exactly once per step.
//   scores: lane i of wavefront w owns row w*64 + i of the split and computes
//           its logits for the G heads (q in LDS, broadcast reads);
//   softmax: wavefront max / sum per head (exp2 with log2(e) folded in);
//   values: CPR lanes cover one V row with 16-byte vectors, 64/CPR rows per
//           step, each lane accumulating its 16/esize columns for G heads;
//   merge:  the four wavefronts combine (max, sum, o) through LDS; with one
//           split the normalised output is written directly, otherwise the
//           partial state goes to the workspace and a merge kernel combines
//           the splits (fixed order, so results are deterministic).
#include "sg_internal.h"

namespace sg {

constexpr int DA_THREADS = 256;
constexpr int DA_WAVES = DA_THREADS / 64;
constexpr int DA_SPLIT = DA_THREADS;  // rows per split: one per lane
constexpr int DA_MAXG = 16;

template <typename T>
struct Elem;
template <>
struct Elem<float> {
    static constexpr int PER16 = 4;
    __device__ static void unpack(const v4u &w, float *x) {
        x[0] = __uint_as_float(w.x); x[1] = __uint_as_float(w.y);
        x[2] = __uint_as_float(w.z); x[3] = __uint_as_float(w.w);
    }
    __device__ static float load1(const void *p, int64_t i) { return reinterpret_cast<const float *>(p)[i]; }
};
template <>
struct Elem<uint16_t> {  // bfloat16 bits
    static constexpr int PER16 = 8;
    __device__ static void unpack(const v4u &w, float *x) {
        x[0] = bf16_lo(w.x); x[1] = bf16_hi(w.x); x[2] = bf16_lo(w.y); x[3] = bf16_hi(w.y);
        x[4] = bf16_lo(w.z); x[5] = bf16_hi(w.z); x[6] = bf16_lo(w.w); x[7] = bf16_hi(w.w);
    }
    __device__ static float load1(const void *p, int64_t i) {
        return __uint_as_float(((uint32_t)reinterpret_cast<const uint16_t *>(p)[i]) << 16);
    }
};

// partial state of one split: per head (m, l) then o[d]
__device__ __forceinline__ float *part_ptr(float *ws, int64_t unit, int nsplit, int split, int G, int d) {
    return ws + ((unit * nsplit + split) * G) * (int64_t)(d + 2);
}

template <typename T, int D, int G>
__global__ __launch_bounds__(DA_THREADS) void decode_kernel(
    int Hq, int Hkv, float scale_log2, const T *__restrict__ q, const v4u *__restrict__ k_pool,
    const v4u *__restrict__ v_pool, int64_t pool_rows, const int32_t *__restrict__ page_table,
    const int32_t *__restrict__ n_rows, int page_size, int max_pages, float *__restrict__ out,
    float *__restrict__ ws) {
    constexpr int PER16 = Elem<T>::PER16;
    constexpr int CPR = D / PER16;         // 16-byte vectors per row
    constexpr int RPS = 64 / CPR;          // rows per wavefront step in the value phase
    __shared__ float q_s[G][D];
    __shared__ float p_s[DA_WAVES][G][64];
    __shared__ int64_t row_s[DA_WAVES][64];
    __shared__ float m_s[DA_WAVES][G], l_s[DA_WAVES][G];
    __shared__ float o_s[DA_WAVES][G][D];

    const int64_t unit = blockIdx.x;        // b * Hkv + h
    const int b = (int)(unit / Hkv), h = (int)(unit % Hkv);
    const int split = blockIdx.y, nsplit = gridDim.y;
    const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
    int64_t n = n_rows[unit];
    n = max<int64_t>(0, min<int64_t>(n, (int64_t)max_pages * page_size));

    for (int i = tid; i < G * D; i += DA_THREADS)
        q_s[i / D][i % D] = Elem<T>::load1(q, ((int64_t)b * Hq + h * G) * D + i);
    __syncthreads();

    // ---- logits: lane owns one row
    const int64_t lr = (int64_t)split * DA_SPLIT + wave * 64 + lane;
    int64_t prow = -1;
    if (lr < n) {
        const int64_t pr = (int64_t)page_table[unit * max_pages + lr / page_size] + lr % page_size;
        if (pr >= 0 && pr < pool_rows) prow = pr;
    }
    row_s[wave][lane] = prow;
    float s[G];
#pragma unroll
    for (int g = 0; g < G; ++g) s[g] = 0.f;
    if (prow >= 0) {
        const v4u *kr = k_pool + prow * CPR;
#pragma unroll 4
        for (int c = 0; c < CPR; ++c) {
            float x[PER16];
            Elem<T>::unpack(kr[c], x);
#pragma unroll
            for (int g = 0; g < G; ++g) {
#pragma unroll
                for (int e = 0; e < PER16; ++e) s[g] = fmaf(q_s[g][c * PER16 + e], x[e], s[g]);
            }
        }
    }
    // ---- softmax statistics of this wavefront's 64 rows (log2 domain)
    float m[G], l[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const float z = prow >= 0 ? s[g] * scale_log2 : -INFINITY;
        m[g] = wave_max(z);
        const float p = prow >= 0 ? __builtin_amdgcn_exp2f(z - m[g]) : 0.f;
        l[g] = wave_sum(p);
        p_s[wave][g][lane] = p;
    }
    __syncthreads();

    // ---- values: CPR lanes per row, RPS rows per step
    const int cg = lane % CPR, rsub = lane / CPR;
    float o[G][PER16];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < PER16; ++e) o[g][e] = 0.f;
#pragma unroll 2
    for (int r = rsub; r < 64; r += RPS) {
        const int64_t pr = row_s[wave][r];
        if (pr < 0) continue;
        float x[PER16];
        Elem<T>::unpack(v_pool[pr * CPR + cg], x);
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const float p = p_s[wave][g][r];
#pragma unroll
            for (int e = 0; e < PER16; ++e) o[g][e] = fmaf(p, x[e], o[g][e]);
        }
    }
    // reduce over the RPS row groups of the wavefront (lanes sharing cg)
#pragma unroll
    for (int off = CPR; off < 64; off <<= 1)
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < PER16; ++e) o[g][e] += __shfl_xor(o[g][e], off, 64);
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

    // ---- combine the wavefronts; thread t handles (g, c) pairs
    for (int i = tid; i < G * D; i += DA_THREADS) {
        const int g = i / D, c = i % D;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < DA_WAVES; ++w) M = fmaxf(M, m_s[w][g]);
        float Lsum = 0.f, O = 0.f;
        if (M > -INFINITY) {
#pragma unroll
            for (int w = 0; w < DA_WAVES; ++w) {
                const float a = m_s[w][g] > -INFINITY ? __builtin_amdgcn_exp2f(m_s[w][g] - M) : 0.f;
                Lsum += a * l_s[w][g];
                O += a * o_s[w][g][c];
            }
        }
        if (nsplit == 1) {
            out[((int64_t)b * Hq + h * G + g) * D + c] = Lsum > 0.f ? O / Lsum : 0.f;
        } else {
            float *pp = part_ptr(ws, unit, nsplit, split, G, D) + (int64_t)g * (D + 2);
            if (c == 0) { pp[0] = M; pp[1] = Lsum; }
            pp[2 + c] = O;
        }
    }
}

template <int D, int G>
__global__ __launch_bounds__(DA_THREADS) void decode_merge_kernel(int Hq, int Hkv, int nsplit,
                                                                  const float *__restrict__ ws,
                                                                  float *__restrict__ out) {
    const int64_t unit = blockIdx.x;
    const int b = (int)(unit / Hkv), h = (int)(unit % Hkv);
    for (int i = threadIdx.x; i < G * D; i += DA_THREADS) {
        const int g = i / D, c = i % D;
        float M = -INFINITY;
        for (int s = 0; s < nsplit; ++s) M = fmaxf(M, part_ptr(const_cast<float *>(ws), unit, nsplit, s, G, D)[g * (D + 2)]);
        float Lsum = 0.f, O = 0.f;
        if (M > -INFINITY) {
            for (int s = 0; s < nsplit; ++s) {
                const float *pp = part_ptr(const_cast<float *>(ws), unit, nsplit, s, G, D) + (int64_t)g * (D + 2);
                if (pp[0] > -INFINITY) {
                    const float a = __builtin_amdgcn_exp2f(pp[0] - M);
                    Lsum += a * pp[1];
                    O += a * pp[2 + c];
                }
            }
        }
        out[((int64_t)b * Hq + h * G + g) * D + c] = Lsum > 0.f ? O / Lsum : 0.f;
    }
}

template <typename T, int D, int G>
static int launch_decode(hipStream_t s, int B, int Hq, int Hkv, float scale_log2, const void *q,
                         const void *k_pool, const void *v_pool, int64_t pool_rows, const int32_t *page_table,
                         const int32_t *n_rows, int page_size, int max_pages, float *out, float *ws, int nsplit) {
    dim3 grid((unsigned)((int64_t)B * Hkv), (unsigned)nsplit);
    decode_kernel<T, D, G><<<grid, DA_THREADS, 0, s>>>(
        Hq, Hkv, scale_log2, reinterpret_cast<const T *>(q), reinterpret_cast<const v4u *>(k_pool),
        reinterpret_cast<const v4u *>(v_pool), pool_rows, page_table, n_rows, page_size, max_pages, out, ws);
    if (nsplit > 1) decode_merge_kernel<D, G><<<(unsigned)((int64_t)B * Hkv), DA_THREADS, 0, s>>>(Hq, Hkv, nsplit, ws, out);
    return launch_status("sg_decode_attn");
}

template <typename T, int D>
static int dispatch_g(int G, hipStream_t s, int B, int Hq, int Hkv, float sl2, const void *q, const void *kp,
                      const void *vp, int64_t pr, const int32_t *pt, const int32_t *nr, int ps, int mp, float *out,
                      float *ws, int nsplit) {
    switch (G) {
        case 1: return launch_decode<T, D, 1>(s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, nsplit);
        case 2: return launch_decode<T, D, 2>(s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, nsplit);
        case 4: return launch_decode<T, D, 4>(s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, nsplit);
        case 8: return launch_decode<T, D, 8>(s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, nsplit);
        case 16: return launch_decode<T, D, 16>(s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, nsplit);
        default: set_error("sg_decode_attn: group size %d not supported (1, 2, 4, 8, 16)", G); return SG_EUNSUPPORTED;
    }
}

static int num_splits(int max_pages, int page_size) {
    return (int)ceil_div((int64_t)max_pages * page_size, DA_SPLIT);
}

}  // namespace sg

using namespace sg;

extern "C" size_t sg_decode_attn_workspace_size(int B, int Hq, int Hkv, int d, int max_pages, int page_size) {
    if (B <= 0 || Hkv <= 0 || Hq <= 0 || d <= 0 || max_pages <= 0 || page_size <= 0) return 0;
    const int nsplit = num_splits(max_pages, page_size);
    if (nsplit <= 1) return 0;
    const int G = Hq / Hkv;
    return (size_t)B * Hkv * nsplit * G * (size_t)(d + 2) * sizeof(float);
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
    SG_REQUIRE(scale == scale && scale > 0.f, SG_EINVAL, "sg_decode_attn: scale must be positive");
    if (B == 0) return SG_OK;
    SG_REQUIRE(q && k_pool && v_pool && page_table && n_rows && out, SG_EINVAL, "sg_decode_attn: null pointer");
    SG_REQUIRE(aligned16(k_pool) && aligned16(v_pool), SG_EINVAL, "sg_decode_attn: pools must be 16-byte aligned");
    const size_t need = sg_decode_attn_workspace_size(B, Hq, Hkv, d, max_pages, page_size);
    SG_REQUIRE(ws_bytes >= need && (need == 0 || ws), SG_EWORKSPACE, "sg_decode_attn: workspace %zu < %zu", ws_bytes, need);
    const int nsplit = num_splits(max_pages, page_size);
    SG_REQUIRE(nsplit <= 65535, SG_EINVAL, "sg_decode_attn: too many splits");
    const float sl2 = scale * 1.4426950408889634f;  // log2(e)
    const int G = Hq / Hkv;
    hipStream_t s = as_stream(stream);
    float *w = reinterpret_cast<float *>(ws);
    if (dt == SG_F32) {
        if (d == 64) return dispatch_g<float, 64>(G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, nsplit);
        return dispatch_g<float, 128>(G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, nsplit);
    }
    if (d == 64) return dispatch_g<uint16_t, 64>(G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, nsplit);
    return dispatch_g<uint16_t, 128>(G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, nsplit);
}
