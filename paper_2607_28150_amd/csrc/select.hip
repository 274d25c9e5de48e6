// sg_decode_select: decode-time dynamic KV selection (Section 2.3: each step
// the selector picks KV entries from the decode query; Section 5.1: InfiniGen's
// alpha = 5, a partial ratio of 0.3 and a maximum KV selection ratio of 20%).
// Rows are whole heads or a partial set of their channels (32 to 128 wide).
//
// select_logits: z[u][g][j] = scale * q[b][l][g] . k_j for the G q heads of
//   unit u = (b, l, h) and every key j < N_b.  One pass over the unit's keys:
//   LPR lanes per key row, each holding VPL 16-byte slices of it (4 lanes per
//   bf16 row of 128), all of a pass's rows loaded before any use, G dot
//   products per row summed over the lane group by xor shuffles; a wavefront
//   owns consecutive rows and writes each head's logits of them as whole
//   256-byte pieces.  Bound by reading K.
// select_thresh: one 1024-thread workgroup per unit holds its row (up to
//   32 x 1024 keys) in registers: m_g = max_j z[g][j]; r_j = max_g (z[g][j] - m_g); the count of
//   r_j >= -alpha; k = min(count, cap); the exact top-k of r (ties: lower j,
//   select_common.h), ids ascending, the rest of the segment -1.
#include "select_common.h"

namespace sg {

constexpr int SEL_THREADS = 256;
constexpr int SEL_CHUNK = 512;    // keys per workgroup of the logits pass (many rounds of workgroups)
constexpr int SEL_UNROLL = 4;     // key rows in flight per lane group
constexpr int SEL_MAX_G = 8;

constexpr int gcd_c(int a, int b) { return b == 0 ? a : gcd_c(b, a % b); }

// Rows of D elements (a whole head, or a partial set of its channels): VPR
// 16-byte slices, LPR lanes per row (a power of two dividing VPR, at most 4,
// 8 for rows of 32 slices), VPL slices per lane.
template <typename T, int D>
struct SelShape {
    static constexpr int VPR = D * (int)sizeof(T) / 16;
    static constexpr int LPR = gcd_c(VPR, VPR >= 32 ? 8 : 4);
    static constexpr int VPL = VPR / LPR;
    static_assert(D * (int)sizeof(T) % 16 == 0, "rows must be whole 16-byte slices");
};

struct SelUnit {
    int b, l, h;
    int64_t s0, N;
};

__device__ __forceinline__ SelUnit sel_unit(int64_t u, int B, int Hkv, const int32_t *cu_seqlens, int64_t T) {
    SelUnit g;
    g.b = (int)(u % B);
    const int64_t lh = u / B;
    g.l = (int)(lh / Hkv);
    g.h = (int)(lh % Hkv);
    const int64_t s0 = cu_seqlens[g.b], s1 = cu_seqlens[g.b + 1];
    g.s0 = s0;
    g.N = (s0 >= 0 && s1 >= s0 && s1 <= T) ? s1 - s0 : 0;   // bad metadata: an empty request
    return g;
}

template <typename T, int D, int G>
__global__ __launch_bounds__(SEL_THREADS) void select_logits_kernel(int B, int L, int Hq, int Hkv,
                                                                      const int32_t *__restrict__ cu_seqlens,
                                                                      int64_t T_, const T *__restrict__ q,
                                                                      const T *__restrict__ k, int64_t k_layer_rows,
                                                                      float scale, int nchunk, int ldz,
                                                                      float *__restrict__ z,
                                                                      float *__restrict__ zmax) {
    using S = SelShape<T, D>;
    __shared__ float wmax[SEL_THREADS / 64][G];
    const int64_t u = blockIdx.x / nchunk;
    const int chunk = blockIdx.x % nchunk;
    const SelUnit g = sel_unit(u, B, Hkv, cu_seqlens, T_);
    const int N = (int)min<int64_t>(g.N, ldz);
    const int j0 = chunk * SEL_CHUNK;
    if (j0 >= N) return;
    const int j1 = min(N, j0 + SEL_CHUNK);
    // a wavefront owns GPW * SEL_UNROLL consecutive rows of every step: lane
    // group grp (LPR lanes) takes rows grp, grp + GPW, ...
    constexpr int GPW = 64 / S::LPR;
    constexpr int WROWS = GPW * SEL_UNROLL;
    const int lv = threadIdx.x % S::LPR;
    const int lane = threadIdx.x % 64;
    const int grp = lane / S::LPR;
    const int wave = threadIdx.x / 64;
    const v4u *qb = reinterpret_cast<const v4u *>(q + (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * D);
    v4u qs[G][S::VPL];
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
#pragma unroll
        for (int v = 0; v < S::VPL; ++v) qs[hh][v] = qb[hh * S::VPR + lv + v * S::LPR];
    const v4u *ku = reinterpret_cast<const v4u *>(k + ((int64_t)g.l * k_layer_rows + (int64_t)g.h * T_ + g.s0) * D);
    float *zu = z + u * G * (int64_t)ldz;
    float mx[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) mx[hh] = -INFINITY;
    for (int w0 = j0 + wave * WROWS; w0 < j1; w0 += (SEL_THREADS / 64) * WROWS) {   // uniform per wavefront
        v4u kr[SEL_UNROLL][S::VPL];
#pragma unroll
        for (int r = 0; r < SEL_UNROLL; ++r) {
            const int j = min(w0 + r * GPW + grp, j1 - 1);
#pragma unroll
            for (int v = 0; v < S::VPL; ++v) kr[r][v] = ku[(int64_t)j * S::VPR + lv + v * S::LPR];
        }
        __builtin_amdgcn_sched_barrier(0);
        float zs[SEL_UNROLL][G];
#pragma unroll
        for (int r = 0; r < SEL_UNROLL; ++r) {
            float acc[G];
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                acc[hh] = 0.f;
#pragma unroll
                for (int v = 0; v < S::VPL; ++v) acc[hh] = SliceDot<T>::run(qs[hh][v], kr[r][v], acc[hh]);
            }
#pragma unroll
            for (int o = 1; o < S::LPR; o <<= 1)
#pragma unroll
                for (int hh = 0; hh < G; ++hh) acc[hh] += __shfl_xor(acc[hh], o, 64);
            const bool live = w0 + r * GPW + grp < j1;
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                zs[r][hh] = scale * acc[hh];
                if (live) mx[hh] = fmaxf(mx[hh], zs[r][hh]);
            }
        }
        if constexpr (WROWS <= 64) {
            // lane L stores row w0 + L of every head (whole pieces of 4 * WROWS
            // bytes): that value sits in lane group L % GPW, unroll slot L / GPW
            const int jw = w0 + lane;
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                float v = 0.f;
#pragma unroll
                for (int r = 0; r < SEL_UNROLL; ++r) {
                    const float t = __shfl(zs[r][hh], (lane % GPW) * S::LPR, 64);
                    v = lane / GPW == r ? t : v;
                }
                if (lane < WROWS && jw < j1) zu[(int64_t)hh * ldz + jw] = v;
            }
        } else {
            // one or two lanes per row: the lane groups of a step already hold
            // consecutive rows
#pragma unroll
            for (int r = 0; r < SEL_UNROLL; ++r) {
                const int j = w0 + r * GPW + grp;
#pragma unroll
                for (int hh = 0; hh < G; ++hh)
                    if (hh % S::LPR == lv && j < j1) zu[(int64_t)hh * ldz + j] = zs[r][hh];
            }
        }
    }
    // the chunk's maximum of every head (exact: a maximum of the stored values)
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        const float m = wave_max(mx[hh]);
        if (threadIdx.x % 64 == 0) wmax[wave][hh] = m;
    }
    __syncthreads();
    if (threadIdx.x < G) {
        float m = -INFINITY;
#pragma unroll
        for (int w = 0; w < SEL_THREADS / 64; ++w) m = fmaxf(m, wmax[w][threadIdx.x]);
        zmax[(u * nchunk + chunk) * G + threadIdx.x] = m;
    }
}

template <int ITEMS>
__global__ __launch_bounds__(TOPK_THREADS) void select_thresh_kernel(int B, int L, int Hkv, int G,
                                                                       const int32_t *__restrict__ cu_seqlens,
                                                                       int64_t T_, int ldz, int nchunk,
                                                                       const float *__restrict__ z,
                                                                       const float *__restrict__ zmax, float alpha,
                                                                       const int32_t *__restrict__ cu_cap,
                                                                       int64_t K_cap, int32_t *__restrict__ idx,
                                                                       int32_t *__restrict__ n_sel) {
    __shared__ SelectSmem sm;
    __shared__ float gmax[1][SEL_MAX_G];
    const int64_t u = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
    const SelUnit g = sel_unit(u, B, Hkv, cu_seqlens, T_);
    const int64_t lh = u / B;
    int32_t *ns = n_sel + (int64_t)g.b * L * Hkv + lh;
    const int64_t c0 = cu_cap[g.b], c1 = cu_cap[g.b + 1];
    if (c0 < 0 || c1 < c0 || c1 > K_cap) {   // no writable segment
        if (tid == 0) *ns = 0;
        return;
    }
    int32_t *out = idx + lh * K_cap + c0;
    const int64_t cap = c1 - c0;
    const int N = (int)g.N;
    if (cap == 0 || N == 0 || N > ldz || N > ITEMS * TOPK_THREADS) {
        for (int64_t i = tid; i < cap; i += TOPK_THREADS) out[i] = -1;
        if (tid == 0) *ns = 0;
        return;
    }
    const float *zu = z + u * G * (int64_t)ldz;
    const int first = tid * ITEMS;
    const int nv = max(0, min(ITEMS, N - first));
    // each head's maximum over the unit's keys, from the logits pass's chunk maxima
    const int nc = (int)ceil_div(N, SEL_CHUNK);
    if (wave == 0) {
        for (int hh = 0; hh < G; ++hh) {
            float m = -INFINITY;
            for (int c = lane; c < nc; c += 64) m = fmaxf(m, zmax[(u * nchunk + c) * G + hh]);
            m = wave_max(m);
            if (lane == 0) gmax[0][hh] = m;
        }
    }
    __syncthreads();
    float mg[SEL_MAX_G];
#pragma unroll
    for (int hh = 0; hh < SEL_MAX_G; ++hh) mg[hh] = hh < G ? gmax[0][hh] : -INFINITY;
    // r_j = the best margin over the group's heads; the rule's count
    uint32_t key[ITEMS];
    float rr[ITEMS];
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) rr[i] = -INFINITY;
    const bool vec = ITEMS % 4 == 0 && nv == ITEMS && ldz % 4 == 0;    // whole, 16-byte aligned pieces
#pragma unroll
    for (int hh = 0; hh < SEL_MAX_G; ++hh) {
        if (hh < G) {
            const float *zr = zu + (int64_t)hh * ldz + first;
            if (vec) {
#pragma unroll
                for (int i = 0; i < ITEMS; i += 4) {
                    const float4 x = *reinterpret_cast<const float4 *>(zr + i);
                    rr[i] = fmaxf(rr[i], x.x - mg[hh]);
                    rr[i + 1] = fmaxf(rr[i + 1], x.y - mg[hh]);
                    rr[i + 2] = fmaxf(rr[i + 2], x.z - mg[hh]);
                    rr[i + 3] = fmaxf(rr[i + 3], x.w - mg[hh]);
                }
            } else {
#pragma unroll
                for (int i = 0; i < ITEMS; ++i)
                    if (i < nv) rr[i] = fmaxf(rr[i], zr[i] - mg[hh]);
            }
        }
    }
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
        key[i] = i < nv ? order_key(rr[i]) : 0u;
        cnt += (i < nv && rr[i] >= -alpha) ? 1 : 0;
    }
    int total;
    block_scan_incl(cnt, sm.wsum, total);
    const int kk = (int)min<int64_t>(total, cap);
    if (kk > 0) select_top<ITEMS>(key, nv, first, kk, out, sm);
    for (int64_t i = kk + tid; i < cap; i += TOPK_THREADS) out[i] = -1;
    if (tid == 0) *ns = kk;
}

struct LogitsArgs {
    int B, L, Hq, Hkv;
    const int32_t *cu_seqlens;
    int64_t T;
    int max_seqlen;
    const void *q, *k;
    int64_t k_layer_rows;
    float scale;
    float *z, *zmax;
};

template <typename E, int D, int G>
static void launch_logits(hipStream_t s, const LogitsArgs &a) {
    const int nchunk = (int)ceil_div(a.max_seqlen, SEL_CHUNK);
    const int64_t grid = (int64_t)a.B * a.L * a.Hkv * nchunk;
    select_logits_kernel<E, D, G><<<(unsigned)grid, SEL_THREADS, 0, s>>>(
        a.B, a.L, a.Hq, a.Hkv, a.cu_seqlens, a.T, reinterpret_cast<const E *>(a.q), reinterpret_cast<const E *>(a.k),
        a.k_layer_rows, a.scale, nchunk, a.max_seqlen, a.z, a.zmax);
}

template <typename E, int D>
static void launch_logits_g(hipStream_t s, int G, const LogitsArgs &a) {
    switch (G) {
        case 1: launch_logits<E, D, 1>(s, a); break;
        case 2: launch_logits<E, D, 2>(s, a); break;
        case 4: launch_logits<E, D, 4>(s, a); break;
        default: launch_logits<E, D, 8>(s, a); break;
    }
}

template <typename E>
static void launch_logits_d(hipStream_t s, int d, int G, const LogitsArgs &a) {
    switch (d) {
        case 32: launch_logits_g<E, 32>(s, G, a); break;
        case 40: launch_logits_g<E, 40>(s, G, a); break;
        case 48: launch_logits_g<E, 48>(s, G, a); break;
        case 64: launch_logits_g<E, 64>(s, G, a); break;
        default: launch_logits_g<E, 128>(s, G, a); break;
    }
}

}  // namespace sg

using namespace sg;

// Workspace: the logits z [units][G][max_seqlen], then the chunk maxima
// [units][nchunk][G] (units * G = B * L * Hq).
extern "C" size_t sg_decode_select_workspace_size(int B, int L, int Hq, int max_seqlen) {
    if (B <= 0 || L <= 0 || Hq <= 0 || max_seqlen <= 0) return 0;
    return (size_t)B * L * Hq * ((size_t)max_seqlen + ceil_div(max_seqlen, SEL_CHUNK)) * sizeof(float);
}

extern "C" int sg_decode_select(void *stream, sg_dtype dt, int B, int L, int Hq, int Hkv, int d, const void *q,
                                const int32_t *cu_seqlens, int64_t T, int max_seqlen, const void *k,
                                int64_t k_layer_rows, float scale, float alpha, const int32_t *cu_cap,
                                int64_t K_cap, int32_t *idx, int32_t *n_sel, void *ws, size_t ws_bytes) {
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "sg_decode_select: unknown dtype %d", (int)dt);
    SG_REQUIRE(B >= 1 && L >= 1 && Hq >= 1 && Hkv >= 1 && Hq % Hkv == 0, SG_EINVAL,
               "sg_decode_select: need B, L, Hq, Hkv >= 1 and Hq %% Hkv == 0");
    const int G = Hq / Hkv;
    SG_REQUIRE(G == 1 || G == 2 || G == 4 || G == 8, SG_EUNSUPPORTED, "sg_decode_select: group size %d (1, 2, 4, 8)",
               G);
    SG_REQUIRE(d == 32 || d == 40 || d == 48 || d == 64 || d == 128, SG_EUNSUPPORTED,
               "sg_decode_select: row width %d not supported (32, 40, 48, 64, 128)", d);
    SG_REQUIRE(scale >= 0.f && scale < INFINITY, SG_EINVAL, "sg_decode_select: scale must be finite and >= 0");
    if (scale == 0.f) scale = 1.0f / sqrtf((float)d);
    SG_REQUIRE(alpha >= 0.f && alpha < INFINITY, SG_EINVAL, "sg_decode_select: alpha must be finite and >= 0");
    SG_REQUIRE(T >= 0 && max_seqlen >= 0 && k_layer_rows >= 0 && K_cap >= 0, SG_EINVAL,
               "sg_decode_select: negative size");
    SG_REQUIRE(max_seqlen <= 32 * TOPK_THREADS, SG_EUNSUPPORTED, "sg_decode_select: max_seqlen %d above %d",
               max_seqlen, 32 * TOPK_THREADS);
    SG_REQUIRE(cu_seqlens && cu_cap && n_sel && (K_cap == 0 || idx), SG_EINVAL, "sg_decode_select: null pointer");
    const int64_t units = (int64_t)B * L * Hkv;
    SG_REQUIRE(units * std::max<int64_t>(1, ceil_div(max_seqlen, SEL_CHUNK)) <= 0x7fffffff, SG_EINVAL,
               "sg_decode_select: grid too large");
    const int ldz = std::max(max_seqlen, 1);
    hipStream_t s = as_stream(stream);
    if (max_seqlen > 0 && T > 0) {
        SG_REQUIRE(q && k, SG_EINVAL, "sg_decode_select: null pointer");
        SG_REQUIRE(aligned16(q) && aligned16(k), SG_EINVAL, "sg_decode_select: q and k must be 16-byte aligned");
        const size_t need = sg_decode_select_workspace_size(B, L, Hq, max_seqlen);
        SG_REQUIRE(ws && ws_bytes >= need, SG_EWORKSPACE, "sg_decode_select: workspace %zu < %zu", ws_bytes, need);
        float *z = reinterpret_cast<float *>(ws);
        float *zm = z + (int64_t)B * L * Hq * max_seqlen;
        const LogitsArgs a{B, L, Hq, Hkv, cu_seqlens, T, max_seqlen, q, k, k_layer_rows, scale, z, zm};
        if (dt == SG_BF16) launch_logits_d<uint16_t>(s, d, G, a);
        else launch_logits_d<float>(s, d, G, a);
    }
    const float *z = reinterpret_cast<const float *>(ws);
    const float *zm = z + (int64_t)B * L * Hq * std::max(max_seqlen, 0);
    const int nchunk = (int)std::max<int64_t>(1, ceil_div(max_seqlen, SEL_CHUNK));
    const unsigned grid = (unsigned)units;
    if (max_seqlen <= 2 * TOPK_THREADS)
        select_thresh_kernel<2><<<grid, TOPK_THREADS, 0, s>>>(B, L, Hkv, G, cu_seqlens, T, ldz, nchunk, z, zm, alpha, cu_cap, K_cap, idx, n_sel);
    else if (max_seqlen <= 8 * TOPK_THREADS)
        select_thresh_kernel<8><<<grid, TOPK_THREADS, 0, s>>>(B, L, Hkv, G, cu_seqlens, T, ldz, nchunk, z, zm, alpha, cu_cap, K_cap, idx, n_sel);
    else
        select_thresh_kernel<32><<<grid, TOPK_THREADS, 0, s>>>(B, L, Hkv, G, cu_seqlens, T, ldz, nchunk, z, zm, alpha, cu_cap, K_cap, idx, n_sel);
    return launch_status("sg_decode_select");
}
