// sg_score: per-token importance from a window of prefill attention.
//
// For one unit the window queries form an R x d matrix (R = G * W rows: the G
// q heads of the KV group times the W window positions) and the unit's keys an
// N x d matrix.  score_j = sum over rows of softmax_row(Q K^T / sqrt(d))_j with
// the causal limit j <= position(row).  The row normaliser (log-sum-exp) is
// needed before any column can be summed, so the contraction runs twice:
//
//   stats  : per (unit, 2048-key chunk) the per-row (reference, sum exp) of
//            the chunk's logits;
//   colsum : merge the chunk statistics into each row's LSE, recompute the
//            logits, p = exp(z - LSE), and sum p over the R rows for every key.
//
// When the caller passes the LSE (a prefill flash attention produces it) only
// colsum runs.
//
// Both passes use one engine.  A workgroup owns one (unit, chunk) and has one
// wavefront per 64 query rows; each wavefront keeps its rows in registers as
// MFMA operand fragments.  The chunk's keys stream through LDS in tiles of 64
// keys (stats) or 128 (colsum; 64 at fp32), double buffered: direct
// global->LDS loads of the
// next tile run while every wavefront multiplies its rows against the current
// one with v_mfma_f32_32x32x16_bf16 (bf16) or v_mfma_f32_16x16x4_f32 (fp32),
// fp32 accumulation; one workgroup barrier per tile.  Within a tile the
// (key block, row block) products are software pipelined: the MFMAs of the
// next block and the LDS reads of the block after are issued next to the
// exponentials of the current one.
//
//   stats computes C = K Q^T: a lane's results of a block belong to one query
//   row, so the row's (reference, sum) stays in the lane.  Terms are summed
//   against the current reference (initially 0); only when a block's terms
//   grow past 2^64 of it, or the sum stays below 2^-60 of it (and on the
//   masked tiles at the end of the prompt), the row takes a new reference from
//   the block's exact max.
//   colsum computes C = Q K^T: a lane's results of a block belong to one key;
//   the wavefronts' partial column sums meet in LDS once per tile.
//
// Exponentials use exp2 with log2(e)/sqrt(d) folded into one multiply.  All
// reductions run in a fixed order: results are deterministic.
#include <algorithm>
#include <type_traits>

#include "score_tiles.h"

namespace sg {

// Keys per LDS tile.  The stats pass takes 64-key tiles (32 KB double
// buffered at bf16 d = 128), so three workgroups fit a CU and the pass runs at
// three wavefronts per SIMD (168 VGPRs), where 128-key tiles allowed two.  The
// colsum pass needs about 200 VGPRs and stays at two wavefronts per SIMD (at
// three the compiler spills 50 or more registers, even with the row
// normalisers read from LDS, and the pass slows by half); it keeps 128-key
// tiles, which measured 2-3% faster for it than 64 at the 64-request shape.
// Same box, alternating builds: 64 requests, two passes 43.8 against 44.0 ms
// and the request pairs 40.9 against 41.2 ms; 8K workload 325 against 331 us.
constexpr int SC_STATS_TILE_KEYS = 64;
template <typename T>
constexpr int colsum_tile_keys() { return sizeof(T) == 2 ? 128 : 64; }

// Wavefronts per SIMD the stats kernel is compiled for: three for the bf16
// probability pass (168 VGPRs, 2 spilled); the count mode's max-only pass and
// the fp32 passes would spill far more at three and keep two.
template <typename T>
constexpr int stats_waves(bool maxonly) {
    return sizeof(T) == 2 && !maxonly ? 3 : 2;
}

// ---------------------------------------------------------------- stats pass

// Exact update of the blocks whose bit (kb * NRB + rb) is set in `sel`.  The
// state (m, s) of a row means: the sum of 2^x over the keys seen so far is
// s * 2^m, with any reference m.  The new reference is the larger of the
// state's magnitude m + log2(s) and the block's max over its visible keys
// (all keys unless MASK), so neither the state nor the block's terms can
// overflow or lose precision.
template <typename T, int D, bool MASK>
struct StatsExact {
    static constexpr int NRB = QFrags<T, D>::NRB;
    float (&m)[NRB];
    float (&s)[NRB];
    unsigned sel;
    int lane, wave, key0, N, W, R;
    float c2;
    __device__ __forceinline__ void operator()(TC<T, D> &acc, int kb, int rb) const {
        using M = MT<T, D>;
        if (MASK) {
            const int row = wave * 64 + rb * M::BM + lane % M::BM;
            const int pos = row < R ? N - W + row % W : -1;
#pragma unroll
            for (int v = 0; v < M::NV; ++v) acc[v] = key0 + kb * M::BM + M::crow(v, lane) <= pos ? acc[v] : -INFINITY;
        }
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < M::NV; ++v) mx = fmaxf(mx, acc[v]);
        const float eff = s[rb] > 0.f ? m[rb] + __log2f(s[rb]) : -INFINITY;
        const float mn = fmaxf(eff, mx * c2);
        const float ref = mn == -INFINITY ? 0.f : mn;
        float t = 0.f;
#pragma unroll
        for (int v = 0; v < M::NV; ++v) t += __builtin_amdgcn_exp2f(fmaf(acc[v], c2, -ref));
        const float sn = fmaf(s[rb], __builtin_amdgcn_exp2f(m[rb] - ref), t);
        const bool take = (sel >> (kb * NRB + rb)) & 1u;
        s[rb] = take ? sn : s[rb];
        m[rb] = take ? ref : m[rb];
    }
};

// Fast update against the current reference.  A block whose terms sum past
// 2^64 of it, or after which the row's sum is still below 2^-60 of it, is left
// untouched and reported in `need` (then the exact update takes it).
template <typename T, int D>
struct StatsFast {
    static constexpr int NRB = QFrags<T, D>::NRB;
    const float (&m)[NRB];
    float (&s)[NRB];
    unsigned &need;
    float c2;
    __device__ __forceinline__ void operator()(TC<T, D> &acc, int kb, int rb) const {
        using M = MT<T, D>;
        const float nm = -m[rb];
        float t[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int v = 0; v < M::NV; ++v) t[v % 4] += __builtin_amdgcn_exp2f(fmaf(acc[v], c2, nm));
        const float tt = (t[0] + t[1]) + (t[2] + t[3]);
        const float sn = s[rb] + tt;
        const bool bad = !(tt <= 0x1p64f) || !(sn >= 0x1p-60f);     // also inf and NaN
        need |= (unsigned)bad << (kb * NRB + rb);
        s[rb] = bad ? s[rb] : sn;
    }
};

// Count mode: only each row's exact maximum of the raw products q . k over
// its visible keys (all keys unless MASK).
template <typename T, int D, bool MASK>
struct StatsMax {
    static constexpr int NRB = QFrags<T, D>::NRB;
    float (&m)[NRB];
    int lane, wave, key0, N, W, R;
    __device__ __forceinline__ void operator()(TC<T, D> &acc, int kb, int rb) const {
        using M = MT<T, D>;
        int pos = N;
        if (MASK) {
            const int row = wave * 64 + rb * M::BM + lane % M::BM;
            pos = row < R ? N - W + row % W : -1;
        }
        float mx = m[rb];
#pragma unroll
        for (int v = 0; v < M::NV; ++v)
            mx = fmaxf(mx, (!MASK || key0 + kb * M::BM + M::crow(v, lane) <= pos) ? acc[v] : -INFINITY);
        m[rb] = mx;
    }
};

template <typename T, int D, int NW, bool MAXONLY>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(stats_waves<T>(MAXONLY)))) void score_stats_kernel(
    int B, int L, int Hq, int Hkv, int W, const int32_t *__restrict__ cu_seqlens, int64_t T_,
    const T *__restrict__ q_win, const T *__restrict__ k, int64_t k_layer_rows, float c2, int nchunk, int chunk_keys,
    float2 *__restrict__ part) {
    using M = MT<T, D>;
    using KT = KTile<T, D, SC_STATS_TILE_KEYS>;
    constexpr int NRB = QFrags<T, D>::NRB;
    // two tile buffers as separate objects: the compiler can then tell that the
    // direct loads into one never alias the fragment reads from the other
    __shared__ __attribute__((aligned(16))) char kbA[KT::BYTES];
    __shared__ __attribute__((aligned(16))) char kbB[KT::BYTES];
    int64_t u;
    int chunk;
    unit_chunk((int64_t)L * Hkv * B, nchunk, u, chunk);
    const UnitGeom g = unit_geom(u, B, Hkv, cu_seqlens, T_);
    const int G = Hq / Hkv, R = G * W;
    const int N = (int)g.N;
    const int key_begin = chunk * chunk_keys;
    if (N < W || key_begin >= N) return;
    const int lane = threadIdx.x % 64;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const T *qunit = q_win + (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * W * D;
    const T *kunit = k + ((int64_t)g.l * k_layer_rows + (int64_t)g.h * T_ + g.s0) * D;
    const int key_end = min(N, key_begin + chunk_keys);
    const int ntile = (int)ceil_div(key_end - key_begin, KT::TK);
    KT::template load<NW>(kbA, kunit, key_begin, N, wave, lane);
    QFrags<T, D> q;
    q.load(qunit, R, wave, lane);

    TC<T, D> zero[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) zero[rb] = M::zero();
    // (reference, sum) of row wave * 64 + rb * BM + lane % BM over this lane's keys, log2 units
    // (count mode: the row's maximum raw product, and no sum)
    float m[NRB], s[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) { m[rb] = MAXONLY ? -INFINITY : 0.f; s[rb] = 0.f; }
    // one tile (in kbA when t is even, kbB when odd): wait for it, release the
    // other buffer, load the next tile, then `work`
    auto step = [&](int t, char *cur, char *nxt, auto &&work) {
        barrier_after_loads();      // tile t landed; every wavefront is done with tile t - 1
        const int key0 = key_begin + t * KT::TK;
        if (t + 1 < ntile) KT::template load<NW>(nxt, kunit, key0 + KT::TK, N, wave, lane);
        work(cur, key0);
    };
    auto full = [&](const char *buf, int key0) {       // every row sees every key of the tile
        if constexpr (MAXONLY) {
            tile_sweep<T, D, true, SC_STATS_TILE_KEYS>(buf, q, zero, lane, StatsMax<T, D, false>{m, lane, wave, key0, N, W, R});
        } else {
            unsigned need = 0u;
            tile_sweep<T, D, true, SC_STATS_TILE_KEYS>(buf, q, zero, lane, StatsFast<T, D>{m, s, need, c2});
            if (__any(need != 0u))             // rare: those blocks again, exactly
                tile_sweep<T, D, true, SC_STATS_TILE_KEYS>(buf, q, zero, lane,
                                       StatsExact<T, D, false>{m, s, need, lane, wave, key0, N, W, R, c2});
        }
    };
    auto masked = [&](const char *buf, int key0) {     // causal limit and prompt end (or a leftover full tile)
        if constexpr (MAXONLY)
            tile_sweep_plain<T, D, true, SC_STATS_TILE_KEYS>(buf, q, zero, lane, StatsMax<T, D, true>{m, lane, wave, key0, N, W, R});
        else
            tile_sweep_plain<T, D, true, SC_STATS_TILE_KEYS>(buf, q, zero, lane,
                                         StatsExact<T, D, true>{m, s, ~0u, lane, wave, key0, N, W, R, c2});
    };
    const int nfull = full_tiles(key_begin, ntile, KT::TK, N, W);
    int t = 0;
    for (; t + 1 < nfull; t += 2) {
        step(t, kbA, kbB, full);
        step(t + 1, kbB, kbA, full);
    }
    for (; t < ntile; ++t) {
        if (t & 1) step(t, kbB, kbA, masked);
        else step(t, kbA, kbB, masked);
    }
    barrier_after_loads();      // no load in flight when the workgroup ends
    // combine the lane groups that hold the same row (different keys); the
    // wavefront owns its rows, so the result is the chunk's
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
#pragma unroll
        for (int off = M::BM; off < 64; off <<= 1) {
            const float mo = __shfl_xor(m[rb], off, 64), so = __shfl_xor(s[rb], off, 64);
            const float mn = fmaxf(m[rb], mo);
            if constexpr (!MAXONLY)
                s[rb] = s[rb] * __builtin_amdgcn_exp2f(m[rb] - mn) + so * __builtin_amdgcn_exp2f(mo - mn);
            m[rb] = mn;
        }
        const int row = wave * 64 + rb * M::BM + lane;
        if (lane < M::BM && row < R) part[(u * nchunk + chunk) * (int64_t)R + row] = make_float2(m[rb], s[rb]);
    }
}

// ---------------------------------------------------------------- colsum pass

// Column sums of one block: cs[kb] += sum over the lane's rows of exp(z - LSE).
// Column sums of one block: cs[kb] += sum over the lane's rows of
// exp2(c2 * acc), where the products were accumulated onto minus each row's
// normaliser (divided by c2), so acc * c2 = z * c2 - LSE_row in log2 units.
// Count mode (COUNT): the accumulators start at minus the row's threshold in
// raw product units, and a key adds 1 where the row picks it (acc >= 0).
template <typename T, int D, bool MASK, bool COUNT>
struct ColsumStep {
    float (&cs)[KTile<T, D, colsum_tile_keys<T>()>::NKB];
    const int *poss;    // window position of every row of the unit (-1 for padded rows), LDS
    int lane, wave, key0;
    float c2;
    __device__ __forceinline__ void operator()(TC<T, D> &acc, int kb, int rb) const {
        using M = MT<T, D>;
        const int key = key0 + kb * M::BM + lane % M::BM;
        // four independent partial sums (one long chain of dependent adds
        // would stall the wavefront), combined in a fixed order
        float t[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int g4 = 0; g4 < M::NV / 4; ++g4) {
            int4 pos = make_int4(0, 0, 0, 0);
            if (MASK) pos = *reinterpret_cast<const int4 *>(poss + wave * 64 + rb * M::BM + M::crow(4 * g4, lane));
            const int ps[4] = {pos.x, pos.y, pos.z, pos.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float p = COUNT ? (acc[4 * g4 + i] >= 0.f ? 1.f : 0.f)
                                      : __builtin_amdgcn_exp2f(acc[4 * g4 + i] * c2);
                t[i] += (!MASK || key <= ps[i]) ? p : 0.f;
            }
        }
        cs[kb] += (t[0] + t[1]) + (t[2] + t[3]);
    }
};

template <typename T, int D, int NW, bool COUNT>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) void score_colsum_kernel(
    int B, int L, int Hq, int Hkv, int W, const int32_t *__restrict__ cu_seqlens, int64_t T_,
    const T *__restrict__ q_win, const T *__restrict__ k, int64_t k_layer_rows, float c2, int nchunk, int chunk_keys,
    const float2 *__restrict__ part, const float *__restrict__ lse_in, float thr_off, float *__restrict__ scores) {
    using M = MT<T, D>;
    using KT = KTile<T, D, colsum_tile_keys<T>()>;
    constexpr int NRB = QFrags<T, D>::NRB, NKB = KT::NKB;
    __shared__ __attribute__((aligned(16))) char kbA[KT::BYTES];   // separate objects, see the stats kernel
    __shared__ __attribute__((aligned(16))) char kbB[KT::BYTES];
    __shared__ float csum[2][NW][KT::TK];
    __shared__ __attribute__((aligned(16))) float nl2s[NW * 64];
    __shared__ __attribute__((aligned(16))) int poss[NW * 64];
    int64_t u;
    int chunk;
    unit_chunk((int64_t)L * Hkv * B, nchunk, u, chunk);
    const UnitGeom g = unit_geom(u, B, Hkv, cu_seqlens, T_);
    const int G = Hq / Hkv, R = G * W;
    const int N = (int)g.N;
    const int key_begin = chunk * chunk_keys;
    const int key_end = min(N, key_begin + chunk_keys);
    float *srow = scores + ((int64_t)g.l * Hkv + g.h) * T_ + g.s0;
    if (N < W) {  // documented fallback: zero scores
        for (int j = key_begin + (int)threadIdx.x; j < key_end; j += blockDim.x) srow[j] = 0.f;
        return;
    }
    if (key_begin >= N) return;
    const int lane = threadIdx.x % 64;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const int64_t rbase = (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * W;   // first window row of the unit
    const T *kunit = k + ((int64_t)g.l * k_layer_rows + (int64_t)g.h * T_ + g.s0) * D;
    const int ntile = (int)ceil_div(key_end - key_begin, KT::TK);
    KT::template load<NW>(kbA, kunit, key_begin, N, wave, lane);
    QFrags<T, D> q;
    q.load(q_win + rbase * D, R, wave, lane);
    // row normalisers in log2 units: the caller's LSE, or the merge of the chunk statistics
    for (int r = threadIdx.x; r < NW * 64; r += 64 * NW) {
        if constexpr (COUNT) {
            // the row picks key j when q . k_j >= max - alpha sqrt(d) (raw units)
            float start = -INFINITY;             // padded rows pick nothing
            if (r < R) {
                const int nc = (int)min<int64_t>(ceil_div(N, chunk_keys), nchunk);
                const float2 *pr = part + u * nchunk * (int64_t)R + r;
                float Mx = -INFINITY;
                for (int c = 0; c < nc; ++c) Mx = fmaxf(Mx, pr[(int64_t)c * R].x);
                start = -(Mx - thr_off);
            }
            nl2s[r] = start;
            poss[r] = r < R ? N - W + r % W : -1;
            continue;
        }
        float l2 = INFINITY;                     // padded rows contribute exp2(-inf) = 0
        if (r < R) {
            if (lse_in) {
                l2 = lse_in[rbase + r] * SC_LOG2E;
            } else {
                const int nc = (int)min<int64_t>(ceil_div(N, chunk_keys), nchunk);  // a prompt above max_seqlen is cut
                const float2 *pr = part + u * nchunk * (int64_t)R + r;
                float Mx = -INFINITY;
                for (int c = 0; c < nc; ++c) Mx = fmaxf(Mx, pr[(int64_t)c * R].x);
                const float ref = Mx == -INFINITY ? 0.f : Mx;
                float S = 0.f;
                for (int c = 0; c < nc; ++c) {
                    const float2 p = pr[(int64_t)c * R];
                    S += p.y * __builtin_amdgcn_exp2f(p.x - ref);
                }
                l2 = S > 0.f ? ref + __log2f(S) : INFINITY;
            }
        }
        nl2s[r] = -l2 / c2;
        poss[r] = r < R ? N - W + r % W : -1;
    }
    __syncthreads();
    // accumulator start of every row block: minus the lane's rows' normalisers
    TC<T, D> c0[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int v = 0; v < M::NV; ++v) c0[rb][v] = nl2s[wave * 64 + rb * M::BM + M::crow(v, lane)];

    // per tile: the wavefronts' partial column sums go to csum[t & 1]; they are
    // added and stored after the next barrier
    auto flush = [&](int t) {
        const int key0 = key_begin + t * KT::TK;
        for (int j = threadIdx.x; j < KT::TK; j += 64 * NW) {
            float v = 0.f;
            for (int w = 0; w < NW; ++w) v += csum[t & 1][w][j];
            if (key0 + j < N) srow[key0 + j] = v;
        }
    };
    // one tile (in kbA when t is even, kbB when odd): wait for it, release the
    // other buffer, load the next tile, multiply
    auto step = [&](int t, char *cur, char *nxt, auto mask) {
        constexpr bool MASK = decltype(mask)::value;
        barrier_after_loads();      // tile t landed; tile t - 1 finished everywhere
        if (t > 0) flush(t - 1);
        const int key0 = key_begin + t * KT::TK;
        if (t + 1 < ntile) KT::template load<NW>(nxt, kunit, key0 + KT::TK, N, wave, lane);
        float cs[NKB];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) cs[kb] = 0.f;
        if (MASK)
            tile_sweep_plain<T, D, false, colsum_tile_keys<T>()>(cur, q, c0, lane, ColsumStep<T, D, true, COUNT>{cs, poss, lane, wave, key0, c2});
        else
            tile_sweep<T, D, false, colsum_tile_keys<T>()>(cur, q, c0, lane, ColsumStep<T, D, false, COUNT>{cs, poss, lane, wave, key0, c2});
        // lanes holding the same key (different rows) add up; every such lane
        // then holds the total and stores it (same value, same address: no
        // branch, so the exponentials are not moved behind one)
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
#pragma unroll
            for (int off = M::BM; off < 64; off <<= 1) cs[kb] += __shfl_xor(cs[kb], off, 64);
            csum[t & 1][wave][kb * M::BM + lane % M::BM] = cs[kb];
        }
    };
    const int nfull = full_tiles(key_begin, ntile, KT::TK, N, W);
    int t = 0;
    for (; t + 1 < nfull; t += 2) {
        step(t, kbA, kbB, std::false_type{});
        step(t + 1, kbB, kbA, std::false_type{});
    }
    for (; t < ntile; ++t) {                   // the prompt's last keys (and a leftover full tile)
        if (t & 1) step(t, kbB, kbA, std::true_type{});
        else step(t, kbA, kbB, std::true_type{});
    }
    __syncthreads();
    flush(ntile - 1);
}

// thr_off < 0: probabilities; thr_off >= 0: count mode with the threshold
// max - thr_off in raw product units (thr_off = alpha * sqrt(d)).
template <typename T, int D, int NW>
static void launch_passes(hipStream_t s, const ScorePlan &p, int B, int L, int Hq, int Hkv, int W,
                          const int32_t *cu_seqlens, int64_t ntok, const void *q_win, const void *k,
                          int64_t k_layer_rows, float c2, const float *lse_in, float thr_off, float *scores,
                          void *ws) {
    float2 *part = reinterpret_cast<float2 *>(ws);
    const T *q = reinterpret_cast<const T *>(q_win);
    const T *kk = reinterpret_cast<const T *>(k);
    const dim3 grid((unsigned)((int64_t)L * Hkv * B * p.nchunk));
    if (thr_off >= 0.f) {
        score_stats_kernel<T, D, NW, true><<<grid, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok, q, kk,
                                                                   k_layer_rows, c2, p.nchunk, p.chunk_keys, part);
        score_colsum_kernel<T, D, NW, true><<<grid, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok, q, kk,
                                                                    k_layer_rows, c2, p.nchunk, p.chunk_keys, part,
                                                                    nullptr, thr_off, scores);
        return;
    }
    if (!lse_in)
        score_stats_kernel<T, D, NW, false><<<grid, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok, q, kk,
                                                                    k_layer_rows, c2, p.nchunk, p.chunk_keys, part);
    score_colsum_kernel<T, D, NW, false><<<grid, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok, q, kk,
                                                                 k_layer_rows, c2, p.nchunk, p.chunk_keys, part,
                                                                 lse_in, thr_off, scores);
}

template <typename T, int D>
static int launch_score(const char *name, hipStream_t s, int B, int L, int Hq, int Hkv, int W,
                        const int32_t *cu_seqlens, int64_t ntok, int max_seqlen, const void *q_win, const void *k,
                        int64_t k_layer_rows, const float *lse_in, float thr_off, float *scores, void *ws) {
    const int R = (Hq / Hkv) * W;
    const int nw = (int)ceil_div(R, 64);
    const ScorePlan p = score_plan(B, L, Hkv, max_seqlen);
    const float c2 = SC_LOG2E / sqrtf((float)D);
    if (nw <= 1) launch_passes<T, D, 1>(s, p, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, c2, lse_in, thr_off, scores, ws);
    else if (nw <= 2) launch_passes<T, D, 2>(s, p, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, c2, lse_in, thr_off, scores, ws);
    else if (nw <= 4) launch_passes<T, D, 4>(s, p, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, c2, lse_in, thr_off, scores, ws);
    else launch_passes<T, D, 8>(s, p, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, c2, lse_in, thr_off, scores, ws);
    return launch_status(name);
}

}  // namespace sg

using namespace sg;

extern "C" size_t sg_score_workspace_size(int B, int L, int Hq, int Hkv, int d, int W, int max_seqlen) {
    if (B <= 0 || L <= 0 || Hkv <= 0 || Hq <= 0 || W <= 0 || max_seqlen <= 0 || d <= 0) return 0;
    const int64_t R = (int64_t)(Hq / Hkv) * W;
    const ScorePlan p = score_plan(B, L, Hkv, max_seqlen);
    return (size_t)((int64_t)L * Hkv * B * p.nchunk * R) * sizeof(float2);
}

static int score_entry(const char *name, void *stream, sg_dtype dt, int B, int L, int Hq, int Hkv, int d, int W,
                       const int32_t *cu_seqlens, int64_t T, int max_seqlen, const void *q_win, const void *k,
                       int64_t k_layer_rows, const float *lse_in, float thr_off, float *scores, void *ws,
                       size_t ws_bytes) {
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "%s: unknown dtype %d", name, (int)dt);
    SG_REQUIRE(B >= 1 && L >= 1 && Hq >= 1 && Hkv >= 1 && Hq % Hkv == 0, SG_EINVAL,
               "%s: need B, L, Hq, Hkv >= 1 and Hq %% Hkv == 0", name);
    SG_REQUIRE(d == 64 || d == 128, SG_EUNSUPPORTED, "%s: head dimension %d not supported (64 or 128)", name, d);
    SG_REQUIRE(W >= 1, SG_EINVAL, "%s: window must be >= 1", name);
    SG_REQUIRE((int64_t)(Hq / Hkv) * W <= SC_MAXR, SG_EUNSUPPORTED, "%s: G*W = %d above %d", name, (Hq / Hkv) * W,
               SC_MAXR);
    SG_REQUIRE(T >= 0 && max_seqlen >= 0 && k_layer_rows >= 0, SG_EINVAL, "%s: negative size", name);
    SG_REQUIRE(max_seqlen <= (1 << 30), SG_EINVAL, "%s: max_seqlen too large", name);
    if (T == 0 || max_seqlen == 0) return SG_OK;
    SG_REQUIRE(cu_seqlens && q_win && k && scores, SG_EINVAL, "%s: null pointer", name);
    SG_REQUIRE(aligned16(q_win) && aligned16(k), SG_EINVAL, "%s: q_win and k must be 16-byte aligned", name);
    const int64_t units = (int64_t)L * Hkv * B;
    SG_REQUIRE(units * ceil_div(max_seqlen, 128) <= 0x7fffffff, SG_EINVAL, "%s: grid too large", name);
    if (!lse_in) {
        const size_t need = sg_score_workspace_size(B, L, Hq, Hkv, d, W, max_seqlen);
        SG_REQUIRE(ws && ws_bytes >= need, SG_EWORKSPACE, "%s: workspace %zu < %zu", name, ws_bytes, need);
        SG_REQUIRE(aligned16(ws), SG_EINVAL, "%s: workspace must be 16-byte aligned", name);
    }
    hipStream_t s = as_stream(stream);
    if (dt == SG_BF16) {
        if (d == 128) return launch_score<uint16_t, 128>(name, s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, thr_off, scores, ws);
        return launch_score<uint16_t, 64>(name, s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, thr_off, scores, ws);
    }
    if (d == 128) return launch_score<float, 128>(name, s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, thr_off, scores, ws);
    return launch_score<float, 64>(name, s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, lse_in, thr_off, scores, ws);
}

extern "C" int sg_score(void *stream, sg_dtype dt, int B, int L, int Hq, int Hkv, int d, int W,
                        const int32_t *cu_seqlens, int64_t T, int max_seqlen, const void *q_win, const void *k,
                        int64_t k_layer_rows, const float *lse_in, float *scores, void *ws, size_t ws_bytes) {
    return score_entry("sg_score", stream, dt, B, L, Hq, Hkv, d, W, cu_seqlens, T, max_seqlen, q_win, k,
                       k_layer_rows, lse_in, -1.f, scores, ws, ws_bytes);
}

extern "C" int sg_score_count(void *stream, sg_dtype dt, int B, int L, int Hq, int Hkv, int d, int W,
                              const int32_t *cu_seqlens, int64_t T, int max_seqlen, const void *q_win, const void *k,
                              int64_t k_layer_rows, float alpha, float *counts, void *ws, size_t ws_bytes) {
    SG_REQUIRE(alpha >= 0.f && alpha < INFINITY, SG_EINVAL, "sg_score_count: alpha must be finite and >= 0");
    return score_entry("sg_score_count", stream, dt, B, L, Hq, Hkv, d, W, cu_seqlens, T, max_seqlen, q_win, k,
                       k_layer_rows, nullptr, (float)((double)alpha * sqrt((double)d)), counts, ws, ws_bytes);
}
