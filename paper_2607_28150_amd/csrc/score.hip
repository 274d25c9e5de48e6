// sg_score: per-token importance from a window of prefill attention.
//
// For one unit the window queries form an R x d matrix (R = G * W rows: the G
// q heads of the KV group times the W window positions) and the unit's keys an
// N x d matrix.  score_j = sum over rows of softmax_row(Q K^T / sqrt(d))_j with
// the causal limit j <= position(row).  The row normaliser (log-sum-exp) is
// needed before any column can be summed, so the contraction runs twice:
//
//   A  stats  : per (unit, 512-key chunk) the per-row (max, sum exp) of the
//               chunk's logits;
//   B  merge  : per unit, merge the chunk statistics into each row's LSE;
//   C  colsum : recompute the logits, p = exp(z - LSE), and sum p over the R
//               rows for every key of the chunk.
//
// When the caller passes the LSE (a prefill flash attention produces it) only
// C runs.  A and C share one tile engine: a workgroup of ceil(R/64)
// wavefronts keeps its 64 query rows per wavefront in registers as MFMA A
// fragments; 64-key tiles of K are staged through LDS (rows padded by 16
// bytes so the 16 lanes reading one fragment column hit distinct banks) and
// every wavefront multiplies its rows against the tile with
// v_mfma_f32_16x16x32_bf16 (bf16) or v_mfma_f32_16x16x4_f32 (fp32), fp32
// accumulation.  Exponentials use exp2 with log2(e)/sqrt(d) folded into one
// multiply.  All reductions run in a fixed order: results are deterministic.
#include "score_common.h"

namespace sg {

// ---------------------------------------------------------------- pass A: row statistics per chunk
template <typename T, int D>
__global__ __launch_bounds__(512) void score_stats_kernel(int B, int L, int Hq, int Hkv, int W,
                                                           const int32_t *__restrict__ cu_seqlens, int64_t T_,
                                                           const T *__restrict__ q_win, const T *__restrict__ k,
                                                           int64_t k_layer_rows, float c2, int nchunk,
                                                           float2 *__restrict__ part) {
    __shared__ __attribute__((aligned(16))) char tile[SC_TK * Frag<T, D>::ROWB];
    const int64_t u = blockIdx.x;
    const int chunk = blockIdx.y;
    const UnitGeom g = unit_geom(u, B, Hkv, cu_seqlens, T_);
    const int G = Hq / Hkv, R = G * W;
    const int64_t key_begin = (int64_t)chunk * SC_CHUNK;
    if (g.N < W || key_begin >= g.N) return;
    const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
    const T *qunit = q_win + (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * W * D;
    const T *kunit = k + ((int64_t)g.l * k_layer_rows + (int64_t)g.h * T_ + g.s0) * D;
    typename Frag<T, D>::A qa[4][Frag<T, D>::KSTEPS];
    load_q<T, D>(qunit, R, wave, lane, qa);

    // this lane's 16 rows: rb * 16 + 4 * (lane / 16) + i
    float m[4][4], s[4][4];
    int64_t pos[4][4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = wave * 64 + rb * 16 + 4 * (lane / 16) + i;
            m[rb][i] = -INFINITY;
            s[rb][i] = 0.f;
            pos[rb][i] = r < R ? g.N - W + (r % W) : -1;  // causal limit of the row
        }
    const int64_t key_end = min<int64_t>(g.N, key_begin + SC_CHUNK);
    for (int64_t key0 = key_begin; key0 < key_end; key0 += SC_TK) {
        __syncthreads();
        stage_tile<T, D>(tile, kunit, key0, g.N);
        __syncthreads();
        f32x4 acc[4][4];
        tile_mma<T, D>(qa, tile, lane, acc);
        const bool full = key0 + SC_TK - 1 <= g.N - W;  // every row sees every key of the tile
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float z[4];
                float mx = -INFINITY;
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    const int64_t key = key0 + kb * 16 + lane % 16;
                    const bool ok = full || key <= pos[rb][i];
                    z[kb] = ok ? acc[rb][kb][i] * c2 : -INFINITY;
                    mx = fmaxf(mx, z[kb]);
                }
                if (mx > -INFINITY) {
                    const float mn = fmaxf(m[rb][i], mx);
                    float add = 0.f;
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb) add += __builtin_amdgcn_exp2f(z[kb] - mn);
                    s[rb][i] = s[rb][i] * __builtin_amdgcn_exp2f(m[rb][i] - mn) + add;
                    m[rb][i] = mn;
                }
            }
    }
    // combine the 16 lanes that share rows (lane % 16 varies the key column)
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float mm = m[rb][i], ss = s[rb][i];
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) {
                const float mo = __shfl_xor(mm, off, 64), so = __shfl_xor(ss, off, 64);
                const float mn = fmaxf(mm, mo);
                if (mn > -INFINITY) {
                    ss = ss * __builtin_amdgcn_exp2f(mm - mn) + so * __builtin_amdgcn_exp2f(mo - mn);
                    mm = mn;
                }
            }
            const int r = wave * 64 + rb * 16 + 4 * (lane / 16) + i;
            if (lane % 16 == 0 && r < R) part[(u * nchunk + chunk) * (int64_t)R + r] = make_float2(mm, ss);
        }
}

// ---------------------------------------------------------------- pass B: merge chunks into the LSE
__global__ __launch_bounds__(512) void score_lse_kernel(int B, int L, int Hq, int Hkv, int W,
                                                         const int32_t *__restrict__ cu_seqlens, int64_t T_,
                                                         int nchunk, const float2 *__restrict__ part,
                                                         float *__restrict__ lse) {
    const int64_t u = blockIdx.x;
    const UnitGeom g = unit_geom(u, B, Hkv, cu_seqlens, T_);
    const int G = Hq / Hkv, R = G * W;
    const int r = threadIdx.x;
    if (r >= R) return;
    const int64_t out = (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * W + r;
    if (g.N < W) { lse[out] = INFINITY; return; }
    const int nc = (int)min<int64_t>(ceil_div(g.N, SC_CHUNK), nchunk);  // a prompt above max_seqlen is cut
    float M = -INFINITY;
    for (int c = 0; c < nc; ++c) M = fmaxf(M, part[(u * nchunk + c) * (int64_t)R + r].x);
    float S = 0.f;
    for (int c = 0; c < nc; ++c) {
        const float2 p = part[(u * nchunk + c) * (int64_t)R + r];
        if (p.x > -INFINITY) S += p.y * __builtin_amdgcn_exp2f(p.x - M);
    }
    lse[out] = (M + __log2f(S)) * SC_LN2;  // natural log, like a flash-attention LSE
}

// ---------------------------------------------------------------- pass C: normalised column sums
template <typename T, int D>
__global__ __launch_bounds__(512) void score_colsum_kernel(int B, int L, int Hq, int Hkv, int W,
                                                            const int32_t *__restrict__ cu_seqlens, int64_t T_,
                                                            const T *__restrict__ q_win, const T *__restrict__ k,
                                                            int64_t k_layer_rows, float c2,
                                                            const float *__restrict__ lse,
                                                            float *__restrict__ scores) {
    __shared__ __attribute__((aligned(16))) char tile[SC_TK * Frag<T, D>::ROWB];
    __shared__ float csum[SC_MAXR / 64][SC_TK];
    const int64_t u = blockIdx.x;
    const int chunk = blockIdx.y;
    const UnitGeom g = unit_geom(u, B, Hkv, cu_seqlens, T_);
    const int G = Hq / Hkv, R = G * W;
    const int64_t key_begin = (int64_t)chunk * SC_CHUNK;
    const int nwave = blockDim.x / 64;
    float *srow = scores + ((int64_t)g.l * Hkv + g.h) * T_ + g.s0;
    if (g.N < W) {  // documented fallback: zero scores
        for (int64_t j = key_begin + threadIdx.x; j < min<int64_t>(g.N, key_begin + SC_CHUNK); j += blockDim.x) srow[j] = 0.f;
        return;
    }
    if (key_begin >= g.N) return;
    const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
    const T *qunit = q_win + (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * W * D;
    const T *kunit = k + ((int64_t)g.l * k_layer_rows + (int64_t)g.h * T_ + g.s0) * D;
    const float *lunit = lse + (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * W;
    typename Frag<T, D>::A qa[4][Frag<T, D>::KSTEPS];
    load_q<T, D>(qunit, R, wave, lane, qa);
    float l2[4][4];
    int64_t pos[4][4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = wave * 64 + rb * 16 + 4 * (lane / 16) + i;
            l2[rb][i] = r < R ? lunit[r] * SC_LOG2E : INFINITY;   // padded rows contribute exp2(-inf) = 0
            pos[rb][i] = r < R ? g.N - W + (r % W) : -1;
        }
    const int64_t key_end = min<int64_t>(g.N, key_begin + SC_CHUNK);
    for (int64_t key0 = key_begin; key0 < key_end; key0 += SC_TK) {
        __syncthreads();
        stage_tile<T, D>(tile, kunit, key0, g.N);
        __syncthreads();
        f32x4 acc[4][4];
        tile_mma<T, D>(qa, tile, lane, acc);
        const bool full = key0 + SC_TK - 1 <= g.N - W;
        float cs[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    const int64_t key = key0 + kb * 16 + lane % 16;
                    const bool ok = full || key <= pos[rb][i];
                    const float p = __builtin_amdgcn_exp2f(fmaf(acc[rb][kb][i], c2, -l2[rb][i]));
                    cs[kb] += ok ? p : 0.f;
                }
        // sum over the four lane groups holding different rows of the same keys
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            cs[kb] += __shfl_xor(cs[kb], 16, 64);
            cs[kb] += __shfl_xor(cs[kb], 32, 64);
        }
        if (lane < 16) {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) csum[wave][kb * 16 + lane] = cs[kb];
        }
        __syncthreads();
        if (threadIdx.x < SC_TK) {
            float t = 0.f;
            for (int w = 0; w < nwave; ++w) t += csum[w][threadIdx.x];
            const int64_t key = key0 + threadIdx.x;
            if (key < g.N) srow[key] = t;
        }
    }
}

template <typename T, int D>
static int launch_score(hipStream_t s, int B, int L, int Hq, int Hkv, int W, const int32_t *cu_seqlens, int64_t ntok,
                        int max_seqlen, const void *q_win, const void *k, int64_t k_layer_rows,
                        const float *lse_in, float *scores, void *ws) {
    const int R = (Hq / Hkv) * W;
    const int threads = (int)ceil_div(R, 64) * 64;
    const int nchunk = (int)ceil_div(max_seqlen, SC_CHUNK);
    const int64_t units = (int64_t)L * Hkv * B;
    const float c2 = SC_LOG2E / sqrtf((float)D);
    dim3 grid((unsigned)units, (unsigned)nchunk);
    const float *lse = lse_in;
    if (!lse) {
        float2 *part = reinterpret_cast<float2 *>(ws);
        float *lse_ws = reinterpret_cast<float *>(part + units * nchunk * R);
        score_stats_kernel<T, D><<<grid, threads, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok,
                                                         reinterpret_cast<const T *>(q_win),
                                                         reinterpret_cast<const T *>(k), k_layer_rows, c2,
                                                         nchunk, part);
        score_lse_kernel<<<(unsigned)units, threads, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok, nchunk, part, lse_ws);
        lse = lse_ws;
    }
    score_colsum_kernel<T, D><<<grid, threads, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok,
                                                      reinterpret_cast<const T *>(q_win),
                                                      reinterpret_cast<const T *>(k), k_layer_rows, c2, lse,
                                                      scores);
    return launch_status("sg_score");
}

}  // namespace sg

using namespace sg;

static size_t two_pass_workspace(int B, int L, int Hq, int Hkv, int W, int max_seqlen) {
    const int64_t R = (int64_t)(Hq / Hkv) * W;
    const int64_t units = (int64_t)L * Hkv * B;
    const int64_t nchunk = ceil_div(max_seqlen, SC_CHUNK);
    return (size_t)(units * nchunk * R) * sizeof(float2) + (size_t)B * L * Hq * W * sizeof(float);
}

extern "C" size_t sg_score_workspace_size(int B, int L, int Hq, int Hkv, int d, int W, int max_seqlen) {
    if (B <= 0 || L <= 0 || Hkv <= 0 || Hq <= 0 || W <= 0 || max_seqlen <= 0 || d <= 0) return 0;
    return std::max(two_pass_workspace(B, L, Hq, Hkv, W, max_seqlen),
                    score_fused_workspace(B, L, Hq, Hkv, W, max_seqlen));
}

extern "C" int sg_score(void *stream, sg_dtype dt, int B, int L, int Hq, int Hkv, int d, int W,
                        const int32_t *cu_seqlens, int64_t T, int max_seqlen, const void *q_win, const void *k,
                        int64_t k_layer_rows, const float *lse_in, float *scores, void *ws, size_t ws_bytes) {
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "sg_score: unknown dtype %d", (int)dt);
    SG_REQUIRE(B >= 1 && L >= 1 && Hq >= 1 && Hkv >= 1 && Hq % Hkv == 0, SG_EINVAL,
               "sg_score: need B, L, Hq, Hkv >= 1 and Hq %% Hkv == 0");
    SG_REQUIRE(d == 64 || d == 128, SG_EUNSUPPORTED, "sg_score: head dimension %d not supported (64 or 128)", d);
    SG_REQUIRE(W >= 1, SG_EINVAL, "sg_score: window must be >= 1");
    SG_REQUIRE((int64_t)(Hq / Hkv) * W <= SC_MAXR, SG_EUNSUPPORTED, "sg_score: G*W = %d above %d",
               (Hq / Hkv) * W, SC_MAXR);
    SG_REQUIRE(T >= 0 && max_seqlen >= 0 && k_layer_rows >= 0, SG_EINVAL, "sg_score: negative size");
    SG_REQUIRE(max_seqlen <= (1 << 30), SG_EINVAL, "sg_score: max_seqlen too large");
    if (T == 0 || max_seqlen == 0) return SG_OK;
    SG_REQUIRE(cu_seqlens && q_win && k && scores, SG_EINVAL, "sg_score: null pointer");
    SG_REQUIRE(aligned16(q_win) && aligned16(k), SG_EINVAL, "sg_score: q_win and k must be 16-byte aligned");
    const int64_t units = (int64_t)L * Hkv * B;
    SG_REQUIRE(units <= 0x7fffffff && ceil_div(max_seqlen, SC_CHUNK) <= 65535, SG_EINVAL, "sg_score: grid too large");
    if (!lse_in) {
        const size_t need = sg_score_workspace_size(B, L, Hq, Hkv, d, W, max_seqlen);
        SG_REQUIRE(ws && ws_bytes >= need, SG_EWORKSPACE, "sg_score: workspace %zu < %zu", ws_bytes, need);
        SG_REQUIRE(aligned16(ws), SG_EINVAL, "sg_score: workspace must be 16-byte aligned");
    }
    hipStream_t s = as_stream(stream);
    if (!lse_in) {
        // single pass when the cooperative launch fits; otherwise the two-pass kernels
        const int rc = launch_score_fused(s, dt, d, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k,
                                          k_layer_rows, scores, ws, ws_bytes);
        if (rc != SG_EUNSUPPORTED) return rc;
    }
    if (dt == SG_BF16) {
        if (d == 128) return launch_score<uint16_t, 128>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, scores, ws);
        return launch_score<uint16_t, 64>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, scores, ws);
    }
    if (d == 128) return launch_score<float, 128>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, scores, ws);
    return launch_score<float, 64>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, scores, ws);
}
