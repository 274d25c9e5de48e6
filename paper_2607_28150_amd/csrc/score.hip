// sg_score: per-token importance from a window of prefill attention.
//
// For one unit the window queries form an R x d matrix (R = G * W rows: the G
// q heads of the KV group times the W window positions) and the unit's keys an
// N x d matrix.  score_j = sum over rows of softmax_row(Q K^T / sqrt(d))_j with
// the causal limit j <= position(row).  The row normaliser (log-sum-exp) is
// needed before any column can be summed, so the contraction runs twice:
//
//   A  stats  : per (unit, 1024-key chunk) the per-row (max, sum exp) of the
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

// Double-buffered staging of 64-key K tiles: the next tile's vectors are
// loaded into registers while the current tile is multiplied, then written
// to the other LDS buffer; one workgroup barrier per tile.
template <typename T, int D, int NW>
struct Stager {
    static constexpr int VPR = D * (int)sizeof(T) / 16;      // 16-byte vectors per key row
    static constexpr int NV = SC_TK * VPR;                   // vectors per tile
    static constexpr int PF = (NV + 64 * NW - 1) / (64 * NW);
    v4u r[PF];
    __device__ __forceinline__ void load(const T *kunit, int key0, int N) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int i = (int)threadIdx.x + j * 64 * NW;
            r[j] = v4u{0u, 0u, 0u, 0u};
            if (i < NV && key0 + i / VPR < N)
                r[j] = reinterpret_cast<const v4u *>(kunit + (int64_t)(key0 + i / VPR) * D)[i % VPR];
        }
    }
    __device__ __forceinline__ void store(char *tile) const {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int i = (int)threadIdx.x + j * 64 * NW;
            if (i < NV) *reinterpret_cast<v4u *>(tile + (i / VPR) * Frag<T, D>::ROWB + (i % VPR) * 16) = r[j];
        }
    }
};

// The two passes share one tile engine.  For every 64-key tile of the
// workgroup's key chunk it produces acc[rb][kb] = Q(rows of row-block rb) .
// K(keys of key-block kb) for the wavefront's 64 rows and hands it to
// `on_tile(acc, key0, full, t)`; `full` means every row may see every key of
// the tile (no causal or end-of-prompt masking needed).  After the tile's
// workgroup barrier it calls `after_barrier(key0, t)`.
template <typename T, int D, int NW, typename OnTile, typename After>
__device__ __forceinline__ void for_each_tile(const T *kunit, int N, int W, int key_begin, int key_end,
                                              char *tiles, const typename Frag<T, D>::A (&qa)[4][Frag<T, D>::KSTEPS],
                                              int lane, OnTile &&on_tile, After &&after_barrier) {
    constexpr int TB = SC_TK * Frag<T, D>::ROWB;
    Stager<T, D, NW> st;
    st.load(kunit, key_begin, N);
    st.store(tiles);
    __syncthreads();
    int buf = 0, t = 0;
    for (int key0 = key_begin; key0 < key_end; key0 += SC_TK, ++t) {
        const bool more = key0 + SC_TK < key_end;
        if (more) st.load(kunit, key0 + SC_TK, N);
        f32x4 acc[4][4];
        tile_mma<T, D>(qa, tiles + buf * TB, lane, acc);
        on_tile(acc, key0, key0 + SC_TK - 1 <= N - W, t);
        if (more) st.store(tiles + (buf ^ 1) * TB);
        __syncthreads();
        after_barrier(key0, t);
        buf ^= 1;
    }
}

// ---------------------------------------------------------------- pass A: row statistics per chunk
template <typename T, int D, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) void score_stats_kernel(int B, int L, int Hq, int Hkv, int W,
                                                               const int32_t *__restrict__ cu_seqlens, int64_t T_,
                                                               const T *__restrict__ q_win, const T *__restrict__ k,
                                                               int64_t k_layer_rows, float c2, int nchunk,
                                                               float2 *__restrict__ part) {
    __shared__ __attribute__((aligned(16))) char tiles[2 * SC_TK * Frag<T, D>::ROWB];
    int64_t u;
    int chunk;
    unit_chunk((int64_t)L * Hkv * B, nchunk, u, chunk);
    const UnitGeom g = unit_geom(u, B, Hkv, cu_seqlens, T_);
    const int G = Hq / Hkv, R = G * W;
    const int N = (int)g.N;
    const int key_begin = chunk * SC_CHUNK;
    if (N < W || key_begin >= N) return;
    const int lane = threadIdx.x % 64;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const T *qunit = q_win + (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * W * D;
    const T *kunit = k + ((int64_t)g.l * k_layer_rows + (int64_t)g.h * T_ + g.s0) * D;
    typename Frag<T, D>::A qa[4][Frag<T, D>::KSTEPS];
    load_q<T, D>(qunit, R, wave, lane, qa);

    // running (max, sum) of this lane's 16 rows (rb*16 + 4*(lane/16) + i) over its key columns, log2 units
    float m[4][4], s[4][4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) { m[rb][i] = -INFINITY; s[rb][i] = 0.f; }
    const int key_end = min(N, key_begin + SC_CHUNK);
    for_each_tile<T, D, NW>(kunit, N, W, key_begin, key_end, tiles, qa, lane,
                            [&](f32x4 (&acc)[4][4], int key0, bool full, int) {
        if (!full) {   // causal / end-of-prompt masking (the last tiles of a prompt only)
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int r = wave * 64 + rb * 16 + 4 * (lane / 16) + i;
                    const int pos = r < R ? N - W + (r % W) : -1;
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb)
                        if (key0 + kb * 16 + lane % 16 > pos) acc[rb][kb][i] = -INFINITY;
                }
        }
        // online (max, sum) update; in masked tiles a row with no usable key so
        // far keeps m = -inf and s = 0 (its reference is taken as 0 so that no
        // inf - inf appears)
        if (full) {
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float mx = fmaxf(fmaxf(acc[rb][0][i], acc[rb][1][i]), fmaxf(acc[rb][2][i], acc[rb][3][i]));
                    const float mn = fmaxf(m[rb][i], mx * c2);
                    float add = 0.f;
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb) add += __builtin_amdgcn_exp2f(fmaf(acc[rb][kb][i], c2, -mn));
                    s[rb][i] = fmaf(s[rb][i], __builtin_amdgcn_exp2f(m[rb][i] - mn), add);
                    m[rb][i] = mn;
                }
        } else {
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float mx = fmaxf(fmaxf(acc[rb][0][i], acc[rb][1][i]), fmaxf(acc[rb][2][i], acc[rb][3][i]));
                    const float mn = fmaxf(m[rb][i], mx * c2);
                    const float ref = mn == -INFINITY ? 0.f : mn;
                    float add = 0.f;
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb) add += __builtin_amdgcn_exp2f(fmaf(acc[rb][kb][i], c2, -ref));
                    s[rb][i] = fmaf(s[rb][i], __builtin_amdgcn_exp2f(m[rb][i] - ref), add);
                    m[rb][i] = mn;
                }
        }
    }, [](int, int) {});
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
template <typename T, int D, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) void score_colsum_kernel(int B, int L, int Hq, int Hkv, int W,
                                                                const int32_t *__restrict__ cu_seqlens, int64_t T_,
                                                                const T *__restrict__ q_win, const T *__restrict__ k,
                                                                int64_t k_layer_rows, float c2, int nchunk,
                                                                const float *__restrict__ lse,
                                                                float *__restrict__ scores) {
    __shared__ __attribute__((aligned(16))) char tiles[2 * SC_TK * Frag<T, D>::ROWB];
    __shared__ float csum[2][NW][SC_TK];
    int64_t u;
    int chunk;
    unit_chunk((int64_t)L * Hkv * B, nchunk, u, chunk);
    const UnitGeom g = unit_geom(u, B, Hkv, cu_seqlens, T_);
    const int G = Hq / Hkv, R = G * W;
    const int N = (int)g.N;
    const int key_begin = chunk * SC_CHUNK;
    float *srow = scores + ((int64_t)g.l * Hkv + g.h) * T_ + g.s0;
    if (N < W) {  // documented fallback: zero scores
        for (int j = key_begin + (int)threadIdx.x; j < min(N, key_begin + SC_CHUNK); j += blockDim.x) srow[j] = 0.f;
        return;
    }
    if (key_begin >= N) return;
    const int lane = threadIdx.x % 64;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const T *qunit = q_win + (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * W * D;
    const T *kunit = k + ((int64_t)g.l * k_layer_rows + (int64_t)g.h * T_ + g.s0) * D;
    const float *lunit = lse + (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * W;
    typename Frag<T, D>::A qa[4][Frag<T, D>::KSTEPS];
    load_q<T, D>(qunit, R, wave, lane, qa);
    float l2[4][4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = wave * 64 + rb * 16 + 4 * (lane / 16) + i;
            l2[rb][i] = r < R ? lunit[r] * SC_LOG2E : INFINITY;   // padded rows contribute exp2(-inf) = 0
        }
    const int key_end = min(N, key_begin + SC_CHUNK);
    const int nwave = NW;
    for_each_tile<T, D, NW>(kunit, N, W, key_begin, key_end, tiles, qa, lane,
                            [&](f32x4 (&acc)[4][4], int key0, bool full, int t) {
        float cs[4] = {0.f, 0.f, 0.f, 0.f};
        if (full) {
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb)
                        cs[kb] += __builtin_amdgcn_exp2f(fmaf(acc[rb][kb][i], c2, -l2[rb][i]));
        } else {
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int r = wave * 64 + rb * 16 + 4 * (lane / 16) + i;
                    const int pos = r < R ? N - W + (r % W) : -1;
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb) {
                        const float p = __builtin_amdgcn_exp2f(fmaf(acc[rb][kb][i], c2, -l2[rb][i]));
                        cs[kb] += (key0 + kb * 16 + lane % 16 <= pos) ? p : 0.f;
                    }
                }
        }
        // sum over the four lane groups holding different rows of the same keys
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            cs[kb] += __shfl_xor(cs[kb], 16, 64);
            cs[kb] += __shfl_xor(cs[kb], 32, 64);
        }
        if (lane < 16) {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) csum[t & 1][wave][kb * 16 + lane] = cs[kb];
        }
    }, [&](int key0, int t) {
        // sum over the wavefronts (double-buffered: the next tile writes the other half)
        if (threadIdx.x < SC_TK) {
            float v = 0.f;
            for (int w = 0; w < nwave; ++w) v += csum[t & 1][w][threadIdx.x];
            const int key = key0 + (int)threadIdx.x;
            if (key < N) srow[key] = v;
        }
    });
}

template <typename T, int D, int NW>
static void launch_two_pass(hipStream_t s, dim3 grid, int units, int B, int L, int Hq, int Hkv, int W,
                            const int32_t *cu_seqlens, int64_t ntok, const void *q_win, const void *k,
                            int64_t k_layer_rows, float c2, int nchunk, const float *lse_in, float *scores, void *ws) {
    const int R = (Hq / Hkv) * W;
    const float *lse = lse_in;
    if (!lse) {
        float2 *part = reinterpret_cast<float2 *>(ws);
        float *lse_ws = reinterpret_cast<float *>(part + (int64_t)units * nchunk * R);
        score_stats_kernel<T, D, NW><<<grid, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok,
                                                             reinterpret_cast<const T *>(q_win),
                                                             reinterpret_cast<const T *>(k), k_layer_rows, c2,
                                                             nchunk, part);
        score_lse_kernel<<<(unsigned)units, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok, nchunk, part, lse_ws);
        lse = lse_ws;
    }
    score_colsum_kernel<T, D, NW><<<grid, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok,
                                                          reinterpret_cast<const T *>(q_win),
                                                          reinterpret_cast<const T *>(k), k_layer_rows, c2, nchunk,
                                                          lse, scores);
}

template <typename T, int D>
static int launch_score(hipStream_t s, int B, int L, int Hq, int Hkv, int W, const int32_t *cu_seqlens, int64_t ntok,
                        int max_seqlen, const void *q_win, const void *k, int64_t k_layer_rows,
                        const float *lse_in, float *scores, void *ws) {
    const int R = (Hq / Hkv) * W;
    const int nw = (int)ceil_div(R, 64);
    const int nchunk = (int)ceil_div(max_seqlen, SC_CHUNK);
    const int64_t units = (int64_t)L * Hkv * B;
    const float c2 = SC_LOG2E / sqrtf((float)D);
    dim3 grid((unsigned)(units * nchunk));
    if (nw <= 1) launch_two_pass<T, D, 1>(s, grid, (int)units, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, c2, nchunk, lse_in, scores, ws);
    else if (nw <= 2) launch_two_pass<T, D, 2>(s, grid, (int)units, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, c2, nchunk, lse_in, scores, ws);
    else if (nw <= 4) launch_two_pass<T, D, 4>(s, grid, (int)units, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, c2, nchunk, lse_in, scores, ws);
    else launch_two_pass<T, D, 8>(s, grid, (int)units, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, c2, nchunk, lse_in, scores, ws);
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
    return two_pass_workspace(B, L, Hq, Hkv, W, max_seqlen);
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
    SG_REQUIRE(units * ceil_div(max_seqlen, SC_CHUNK) <= 0x7fffffff, SG_EINVAL, "sg_score: grid too large");
    if (!lse_in) {
        const size_t need = sg_score_workspace_size(B, L, Hq, Hkv, d, W, max_seqlen);
        SG_REQUIRE(ws && ws_bytes >= need, SG_EWORKSPACE, "sg_score: workspace %zu < %zu", ws_bytes, need);
        SG_REQUIRE(aligned16(ws), SG_EINVAL, "sg_score: workspace must be 16-byte aligned");
    }
    hipStream_t s = as_stream(stream);
    if (dt == SG_BF16) {
        if (d == 128) return launch_score<uint16_t, 128>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, scores, ws);
        return launch_score<uint16_t, 64>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, scores, ws);
    }
    if (d == 128) return launch_score<float, 128>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, scores, ws);
    return launch_score<float, 64>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, scores, ws);
}
