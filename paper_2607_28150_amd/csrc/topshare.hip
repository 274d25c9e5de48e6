// sg_score_topshare: selection-frequency importance when every window row
// picks a fixed share of the keys it sees.
//
// Row w of q head g (prompt position p = N - W + w) sees the n = p + 1 keys
// j <= p and picks those whose logit z_j = q . k_j / sqrt(d) is at or above
// its k-th largest, k = floor(n * ratio_bp / 10000) clamped to [1, n]; keys
// tied with the k-th largest are all picked.  counts[j] is the number of
// (q head, window row) pairs of the unit that pick key j.
//
// The k-th largest logit of every row is found exactly by a radix select,
// most significant digit first, over the logits' bit patterns.  A float maps
// to an unsigned key of the same order (sign bit set for non-negative values,
// every bit flipped for negative ones); each pass resolves one digit of DB
// bits of every row's threshold key:
//
//   hist  : recompute the logits with the MFMA engine of sg_score in the
//           C = K Q^T layout (a lane's values of a block belong to one row)
//           and, for each value whose key matches its row's resolved prefix,
//           add one to the row's bin of the next digit (LDS atomics, bins x
//           rows); the chunk's nonzero bins go into the unit's global
//           histogram with global atomics (integer adds: the result does not
//           depend on their order);
//   digit : per row, walk the bins from the top until the remaining rank is
//           reached: that bin's digit extends the prefix, the rank drops by
//           the keys above the bin, and the bins are cleared for the next
//           pass.
//
// After 32 bits the prefix is the key of the row's k-th largest value.  Two
// shortcuts end most rows much earlier:
//   settle : a row whose chosen bin holds exactly the keys it still needs is
//            done (every key at or above the bin's lower edge is picked and
//            nothing below it);
//   gather : once 18 bits are resolved a row's bin holds only a few keys
//            (with real-valued logits); a row whose bin holds at most TS_CMAX
//            keys gathers their values (one more logit pass appends each to
//            the row's list, in LDS, then in the workspace) and a small kernel
//            picks the exact k-th largest among them.  Rows with larger bins
//            (many ties) keep the radix passes.
// A unit with no row left to resolve returns at the start of the remaining
// passes.  The count pass recomputes the logits in the same layout, so each
// row compares exactly the values its threshold came from (the same MFMA
// operands in the same order), and counts each key's picks with one wavefront
// ballot per value (one bit per row) and population counts.
//
// The passes work on the raw products q . k_j: the positive scale 1/sqrt(d)
// keeps their order.  The picks compare floats against the threshold: the
// row's k-th largest value, or a settled bin's lower edge (the float of the
// smallest key in the bin's range, -inf below the keys of -inf), which picks
// exactly the keys at or above the edge.  -0 sorts just below +0 as a key; as
// floats they are equal and picked together, as for any other tie, so a bin
// whose lower edge is +0 does not settle early (-0 would tie it).
#include <algorithm>

#include "score_tiles.h"

namespace sg {

constexpr int TS_MAXBINS = 64;     // bins per row of the global histogram (digits of at most 6 bits)
constexpr int TS_MAXPASS = 8;      // per-unit flag words per call (7 passes at most)
constexpr int TS_CMAX = 32;        // keys a row may gather
constexpr int TS_GATHER_BITS = 18; // resolved bits before a row may gather
constexpr uint32_t TS_GATHER = 0x80000000u;   // need flag: the row gathers its bin

// Digit width: 6 bits (at most 6 histogram passes) while the bins of up to
// 256 rows fit in LDS beside the two K tiles; 5 bits (at most 7) for 512 rows.
template <int NW>
struct TsDigits {
    static constexpr int DB = NW == 8 ? 5 : 6;
    static constexpr int NB = 1 << DB;
};

__device__ __forceinline__ uint32_t order_key(float f) {
    const uint32_t x = __float_as_uint(f);
    return x ^ ((uint32_t)((int32_t)x >> 31) | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t key) {
    return __uint_as_float((key & 0x80000000u) ? (key & 0x7fffffffu) : ~key);
}

// The float threshold of a row whose picks are the keys >= key.
__device__ __forceinline__ float threshold_value(uint32_t key) {
    constexpr uint32_t NEG_INF_KEY = 0x007fffffu;         // order_key(-inf); keys below it are NaN patterns
    return key < NEG_INF_KEY ? -INFINITY : key_value(key);
}

// One block of the histogram pass.  FIRST: the first digit, every value
// counts.  Later passes: c = prefix ^ (the sign flip of the prefix's sign), so
// for a value x of the prefix's sign, x ^ c = key(x) ^ prefix, whose bits
// above the digit are zero exactly when the key matches the prefix; a value of
// the other sign sets the top bit (the prefix always covers the sign bit).
template <typename T, int D, int NW, bool FIRST, bool MASK>
struct HistStep {
    static constexpr int NRB = QFrags<T, D>::NRB;
    uint32_t *hist;                 // LDS [bins][64 * NW]
    const uint32_t (&c)[NRB];
    const int (&pos)[NRB];          // window position of the lane's row (-1: padded row)
    int lane, wave, key0, sh;
    uint32_t lim;                   // bins of this pass (bin lim takes the values that do not count)
    __device__ __forceinline__ void operator()(TC<T, D> &acc, int kb, int rb) const {
        using M = MT<T, D>;
        uint32_t *h = hist + wave * 64 + rb * M::BM + lane % M::BM;      // bin 0 of the lane's row
        // no branch per value (it would split the block and undo the MFMA /
        // vector interleave): a value that does not count goes to bin lim,
        // which is never read
#pragma unroll
        for (int v = 0; v < M::NV; ++v) {
            uint32_t t = FIRST ? order_key(acc[v]) >> sh : min((__float_as_uint(acc[v]) ^ c[rb]) >> sh, lim);
            if (MASK) t = key0 + kb * M::BM + M::crow(v, lane) <= pos[rb] ? t : lim;
            __hip_atomic_fetch_add(h + t * (64 * NW), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
    }
};

template <typename T, int D, int NW, bool FIRST>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) void ts_hist_kernel(
    int B, int L, int Hq, int Hkv, int W, const int32_t *__restrict__ cu_seqlens, int64_t T_,
    const T *__restrict__ q_win, const T *__restrict__ k, int64_t k_layer_rows, int nchunk, int chunk_keys,
    int sh, int width, const uint32_t *__restrict__ busy, const uint32_t *__restrict__ pre,
    uint32_t *__restrict__ ghist) {
    using M = MT<T, D>;
    using KT = KTile<T, D>;
    constexpr int NRB = QFrags<T, D>::NRB, ROWS = 64 * NW, NB = TsDigits<NW>::NB;
    __shared__ __attribute__((aligned(16))) char kbA[KT::BYTES];
    __shared__ __attribute__((aligned(16))) char kbB[KT::BYTES];
    __shared__ __attribute__((aligned(16))) uint32_t hist[(NB + 1) * ROWS];
    int64_t u;
    int chunk;
    unit_chunk((int64_t)L * Hkv * B, nchunk, u, chunk);
    if (!FIRST && busy[u] == 0u) return;        // every row of the unit has settled
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
    const int nbins = 1 << width;
    for (int i = threadIdx.x; i < nbins * ROWS / 4; i += 64 * NW)
        reinterpret_cast<uint4 *>(hist)[i] = make_uint4(0u, 0u, 0u, 0u);
    uint32_t c[NRB];
    int pos[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
        const int row = wave * 64 + rb * M::BM + lane % M::BM;
        pos[rb] = row < R ? N - W + row % W : -1;
        const uint32_t p = (!FIRST && row < R) ? pre[u * R + row] : 0u;
        c[rb] = p ^ ((p & 0x80000000u) ? 0x80000000u : 0xffffffffu);
    }
    TC<T, D> zero[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) zero[rb] = M::zero();
    auto step = [&](int t, char *cur, char *nxt, auto mask) {
        constexpr bool MASK = decltype(mask)::value;
        barrier_after_loads();      // tile t landed (and the bins are clear); tile t - 1 done everywhere
        const int key0 = key_begin + t * KT::TK;
        if (t + 1 < ntile) KT::template load<NW>(nxt, kunit, key0 + KT::TK, N, wave, lane);
        const HistStep<T, D, NW, FIRST, MASK> f{hist, c, pos, lane, wave, key0, sh, (uint32_t)nbins};
        if (MASK) tile_sweep_plain<T, D, true>(cur, q, zero, lane, f);
        else tile_sweep<T, D, true>(cur, q, zero, lane, f);
    };
    const int nfull = full_tiles(key_begin, ntile, KT::TK, N, W);
    int t = 0;
    for (; t + 1 < nfull; t += 2) {
        step(t, kbA, kbB, std::false_type{});
        step(t + 1, kbB, kbA, std::false_type{});
    }
    for (; t < ntile; ++t) {
        if (t & 1) step(t, kbB, kbA, std::true_type{});
        else step(t, kbA, kbB, std::true_type{});
    }
    barrier_after_loads();      // every bin final, no load in flight
    uint32_t *gh = ghist + u * NB * (int64_t)R;
    for (int i = threadIdx.x; i < nbins * ROWS; i += 64 * NW) {
        const int row = i % ROWS;
        const uint32_t v = hist[i];
        if (row < R && v != 0u)
            __hip_atomic_fetch_add(gh + (int64_t)(i / ROWS) * R + row, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// One thread per (unit, row): the start of the select.  need = k, the rank
// (from the top) of the wanted key; prefix = 0; the unit's bins and its
// per-pass flags cleared.
__global__ __launch_bounds__(256) void ts_init_kernel(int64_t nrows, int R, int W, int B, int Hkv,
                                                      const int32_t *__restrict__ cu_seqlens, int64_t T_,
                                                      int ratio_bp, uint32_t *__restrict__ pre,
                                                      uint32_t *__restrict__ need, uint32_t *__restrict__ ghist,
                                                      int nb, uint32_t *__restrict__ busy, int64_t units,
                                                      uint32_t *__restrict__ gcount, uint32_t *__restrict__ gflag) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= nrows) return;
    const int64_t u = i / R;
    const int r = (int)(i % R);
    const UnitGeom g = unit_geom(u, B, Hkv, cu_seqlens, T_);
    const int64_t n = g.N - W + r % W + 1;                 // keys the row sees
    const int64_t kk = std::min<int64_t>(std::max<int64_t>(n, 1), std::max<int64_t>(1, n * ratio_bp / 10000));
    pre[i] = 0u;
    need[i] = (uint32_t)kk;
    uint32_t *h = ghist + u * nb * (int64_t)R + r;
    for (int b = 0; b < nb; ++b) h[(int64_t)b * R] = 0u;
    gcount[i] = 0u;
    if (r == 0) {
        for (int k = 0; k < TS_MAXPASS; ++k) busy[k * units + u] = 0u;
        gflag[u] = 0u;
    }
}

// One thread per (unit, row): pick this pass's digit of the threshold key.
// The bins of a row are R words apart, so a wavefront's 64 rows read each bin
// as one contiguous run; eight bins are read before any is used.  need = 0
// marks a settled row (its bins are only cleared).  busy_in: the flags the
// previous pass set (a unit without one did not run this pass); busy_out: set
// for the unit of every row that has not settled (NULL after the last digit).
// gflag (the digit after which rows may gather, else NULL): a row whose bin
// holds at most TS_CMAX keys is flagged to gather them (need | TS_GATHER) and
// sets gflag of its unit instead of busy_out.
__global__ __launch_bounds__(256) void ts_digit_kernel(int64_t nrows, int R, int nb, int sh, int width,
                                                       const uint32_t *__restrict__ busy_in,
                                                       uint32_t *__restrict__ busy_out, uint32_t *__restrict__ pre,
                                                       uint32_t *__restrict__ need, uint32_t *__restrict__ ghist,
                                                       uint32_t *__restrict__ gflag) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= nrows) return;
    const int64_t u = i / R;
    const int r = (int)(i % R);
    if (busy_in && busy_in[u] == 0u) return;        // settled unit: its pass did not run, the bins are clear
    uint32_t *h = ghist + u * nb * (int64_t)R + r;
    const uint32_t nd = need[i];
    uint32_t above = 0u, digit = 0u, rest = nd, in_bin = 0u;
    bool found = false;
    for (int b0 = (1 << width) - 1; b0 >= 0; b0 -= 8) {          // bins come in fours: 4, 32 or 64
        uint32_t c[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) c[j] = b0 - j >= 0 ? h[(int64_t)(b0 - j) * R] : 0u;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (b0 - j >= 0) h[(int64_t)(b0 - j) * R] = 0u;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (!found && b0 - j >= 0 && above + c[j] >= nd) {
                found = true;
                digit = (uint32_t)(b0 - j);
                rest = nd - above;
                in_bin = c[j];
            }
            above += c[j];
        }
    }
    if (nd == 0u) return;
    const uint32_t p = pre[i] | (digit << sh);
    pre[i] = p;
    const bool settled = rest == in_bin && p != 0x80000000u;      // +0 edge: -0 would tie it
    const bool gather = !settled && gflag && in_bin <= (uint32_t)TS_CMAX;
    need[i] = settled ? 0u : gather ? (rest | TS_GATHER) : rest;
    // every writer of a flag stores the same value
    if (gather) gflag[u] = 1u;
    else if (!settled && busy_out) busy_out[u] = 1u;
}

// One block of the gather pass: the values of gathering rows whose key
// matches the row's prefix (all bits above sh) are appended to the row's list
// in LDS.  A value matches when (bits ^ c) < lim, where lim is 2^sh for a
// gathering row and 0 otherwise: one compare per value, whose wavefront mask
// (one bit per lane) is kept.  Matches are rare (a few per row over the whole
// prompt), so they are handled behind one wavefront-uniform test per block.
// The lanes holding one row (lane % BM) keep the row's count in step: a
// value's mask gives every lane its slot (the count plus the set bits of its
// row's lanes below it) and the count's increase, so no atomics are needed.
template <typename T, int D, int NW, bool MASK>
struct GatherStep {
    static constexpr int NRB = QFrags<T, D>::NRB;
    uint32_t *lcand;                // LDS [64 * NW][TS_CMAX]
    uint32_t (&cnt)[NRB];           // values gathered so far for the lane's row
    const uint32_t (&c)[NRB];       // as in HistStep
    const uint32_t (&lim)[NRB];
    const int (&pos)[NRB];
    uint64_t rowmask, below;        // the lanes of the lane's row; those of them below the lane
    int lane, wave, key0;
    __device__ __forceinline__ void operator()(TC<T, D> &acc, int kb, int rb) const {
        using M = MT<T, D>;
        uint64_t m[M::NV], any = 0u;
#pragma unroll
        for (int v = 0; v < M::NV; ++v) {
            bool h = (__float_as_uint(acc[v]) ^ c[rb]) < lim[rb];
            if (MASK) h = h && key0 + kb * M::BM + M::crow(v, lane) <= pos[rb];
            m[v] = __ballot(h);
            any |= m[v];
        }
        if (__builtin_expect(any != 0u, 0)) {
            const int row = wave * 64 + rb * M::BM + lane % M::BM;
#pragma unroll
            for (int v = 0; v < M::NV; ++v) {
                if (m[v] == 0u) continue;           // wavefront-uniform
                const uint32_t slot = cnt[rb] + (uint32_t)__popcll(m[v] & below);
                if (((m[v] >> lane) & 1u) && slot < (uint32_t)TS_CMAX)
                    lcand[row * TS_CMAX + slot] = __float_as_uint(acc[v]);
                cnt[rb] += (uint32_t)__popcll(m[v] & rowmask);
            }
        }
    }
};

template <typename T, int D, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) void ts_gather_kernel(
    int B, int L, int Hq, int Hkv, int W, const int32_t *__restrict__ cu_seqlens, int64_t T_,
    const T *__restrict__ q_win, const T *__restrict__ k, int64_t k_layer_rows, int nchunk, int chunk_keys,
    int sh, const uint32_t *__restrict__ gflag, const uint32_t *__restrict__ pre, const uint32_t *__restrict__ need,
    uint32_t *__restrict__ gcount, uint32_t *__restrict__ gcand) {
    using M = MT<T, D>;
    using KT = KTile<T, D>;
    constexpr int NRB = QFrags<T, D>::NRB, ROWS = 64 * NW;
    __shared__ __attribute__((aligned(16))) char kbA[KT::BYTES];
    __shared__ __attribute__((aligned(16))) char kbB[KT::BYTES];
    __shared__ uint32_t lcand[ROWS * TS_CMAX];
    int64_t u;
    int chunk;
    unit_chunk((int64_t)L * Hkv * B, nchunk, u, chunk);
    if (gflag[u] == 0u) return;                 // no row of the unit gathers
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
    uint32_t c[NRB], cnt[NRB], lim[NRB];
    int pos[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
        const int row = wave * 64 + rb * M::BM + lane % M::BM;
        pos[rb] = row < R ? N - W + row % W : -1;
        const uint32_t p = row < R ? pre[u * R + row] : 0u;
        const bool on = row < R && (need[u * R + row] & TS_GATHER) != 0u;
        lim[rb] = on ? 1u << sh : 0u;
        c[rb] = p ^ ((p & 0x80000000u) ? 0x80000000u : 0xffffffffu);
        cnt[rb] = 0u;
    }
    // lanes holding the same row: lane % BM, one per lane group
    uint64_t rowmask = 0u;
#pragma unroll
    for (int gi = 0; gi < 64 / M::BM; ++gi) rowmask |= 1ull << (gi * M::BM + lane % M::BM);
    const uint64_t below = rowmask & ((1ull << lane) - 1u);
    TC<T, D> zero[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) zero[rb] = M::zero();
    auto step = [&](int t, char *cur, char *nxt, auto mask) {
        constexpr bool MASK = decltype(mask)::value;
        barrier_after_loads();      // tile t landed; tile t - 1 done everywhere
        const int key0 = key_begin + t * KT::TK;
        if (t + 1 < ntile) KT::template load<NW>(nxt, kunit, key0 + KT::TK, N, wave, lane);
        const GatherStep<T, D, NW, MASK> f{lcand, cnt, c, lim, pos, rowmask, below, lane, wave, key0};
        if (MASK) tile_sweep_plain<T, D, true>(cur, q, zero, lane, f);
        else tile_sweep<T, D, true>(cur, q, zero, lane, f);
    };
    const int nfull = full_tiles(key_begin, ntile, KT::TK, N, W);
    int t = 0;
    for (; t + 1 < nfull; t += 2) {
        step(t, kbA, kbB, std::false_type{});
        step(t + 1, kbB, kbA, std::false_type{});
    }
    for (; t < ntile; ++t) {
        if (t & 1) step(t, kbB, kbA, std::true_type{});
        else step(t, kbA, kbB, std::true_type{});
    }
    barrier_after_loads();      // every list final, no load in flight
    // the chunk's values go after those of the unit's other chunks (their order
    // does not matter: the pick below ranks them); the first lane group of each
    // row block writes its rows' lists
    if (lane < M::BM) {
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
            const int row = wave * 64 + rb * M::BM + lane;
            const uint32_t n = min(cnt[rb], (uint32_t)TS_CMAX);
            if (row >= R || n == 0u) continue;
            const int64_t i = u * R + row;
            const uint32_t base = __hip_atomic_fetch_add(gcount + i, n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            for (uint32_t j = 0; j < n && base + j < (uint32_t)TS_CMAX; ++j)
                gcand[i * TS_CMAX + base + j] = lcand[row * TS_CMAX + j];
        }
    }
}

// One thread per gathering row: the exact key of rank `need` (from the top)
// among the gathered values; the row then settles on it.  The values wait in
// LDS, so the loops run over the row's own count.
__global__ __launch_bounds__(256) void ts_pick_kernel(int64_t nrows, const uint32_t *__restrict__ gcount,
                                                      const uint32_t *__restrict__ gcand, uint32_t *__restrict__ pre,
                                                      uint32_t *__restrict__ need) {
    __shared__ uint32_t keys[TS_CMAX][256];
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= nrows) return;
    const uint32_t nd = need[i];
    if ((nd & TS_GATHER) == 0u) return;
    const uint32_t rank = nd & ~TS_GATHER;
    const int n = (int)min(gcount[i], (uint32_t)TS_CMAX);
    uint32_t *kk = &keys[0][threadIdx.x];             // this thread's column: entries 256 words apart
    for (int a = 0; a < n; ++a) {
        const uint32_t x = gcand[i * TS_CMAX + a];
        kk[a * 256] = x ^ ((uint32_t)((int32_t)x >> 31) | 0x80000000u);
    }
    uint32_t best = pre[i];          // kept only if the values disagreed with the counts
    for (int a = 0; a < n; ++a) {
        const uint32_t ka = kk[a * 256];
        uint32_t above = 0u, atleast = 0u;
        for (int b = 0; b < n; ++b) {
            const uint32_t kb = kk[b * 256];
            above += kb > ka ? 1u : 0u;
            atleast += kb >= ka ? 1u : 0u;
        }
        if (above < rank && rank <= atleast) best = ka;
    }
    pre[i] = best;
    need[i] = 0u;
}

// One block of the count pass: a ballot per value (bit = lane = row), whose
// lane groups hold different keys; a key's picks in the block are the
// population count of its lane group.  Four consecutive keys' counts go to
// LDS in one write (lane 0), one slot per row block.
template <typename T, int D, bool MASK>
struct TsCountStep {
    static constexpr int NRB = QFrags<T, D>::NRB, GR = 64 / MT<T, D>::BM;
    uint32_t *cs;                          // LDS [NRB][tile keys]: this wavefront's picks
    const float (&thr)[NRB];               // the lane's row's threshold (+inf: padded row)
    const int (&pos)[NRB];
    int lane, key0;
    __device__ __forceinline__ void operator()(TC<T, D> &acc, int kb, int rb) const {
        using M = MT<T, D>;
        constexpr uint32_t GMASK = (uint32_t)((1ull << M::BM) - 1);
#pragma unroll
        for (int v4 = 0; v4 < M::NV / 4; ++v4) {
            uint32_t n[GR][4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int v = 4 * v4 + i;
                bool pick = acc[v] >= thr[rb];
                if (MASK) pick = pick && key0 + kb * M::BM + M::crow(v, lane) <= pos[rb];
                const uint64_t m = __ballot(pick);
#pragma unroll
                for (int gi = 0; gi < GR; ++gi) n[gi][i] = (uint32_t)__popc((uint32_t)(m >> (gi * M::BM)) & GMASK);
            }
            // keys crow(4 v4 + i, gi * BM), i = 0..3, are consecutive
            if (lane == 0) {
#pragma unroll
                for (int gi = 0; gi < GR; ++gi)
                    *reinterpret_cast<uint4 *>(cs + rb * KTile<T, D>::TK + kb * M::BM + M::crow(4 * v4, gi * M::BM)) =
                        make_uint4(n[gi][0], n[gi][1], n[gi][2], n[gi][3]);
            }
        }
    }
};

template <typename T, int D, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) void ts_count_kernel(
    int B, int L, int Hq, int Hkv, int W, const int32_t *__restrict__ cu_seqlens, int64_t T_,
    const T *__restrict__ q_win, const T *__restrict__ k, int64_t k_layer_rows, int nchunk, int chunk_keys,
    const uint32_t *__restrict__ pre, float *__restrict__ counts) {
    using M = MT<T, D>;
    using KT = KTile<T, D>;
    constexpr int NRB = QFrags<T, D>::NRB;
    __shared__ __attribute__((aligned(16))) char kbA[KT::BYTES];
    __shared__ __attribute__((aligned(16))) char kbB[KT::BYTES];
    __shared__ __attribute__((aligned(16))) uint32_t csum[2][NW][NRB][KT::TK];
    int64_t u;
    int chunk;
    unit_chunk((int64_t)L * Hkv * B, nchunk, u, chunk);
    const UnitGeom g = unit_geom(u, B, Hkv, cu_seqlens, T_);
    const int G = Hq / Hkv, R = G * W;
    const int N = (int)g.N;
    const int key_begin = chunk * chunk_keys;
    const int key_end = min(N, key_begin + chunk_keys);
    float *orow = counts + ((int64_t)g.l * Hkv + g.h) * T_ + g.s0;
    if (N < W) {  // documented fallback: zero counts
        for (int j = key_begin + (int)threadIdx.x; j < key_end; j += blockDim.x) orow[j] = 0.f;
        return;
    }
    if (key_begin >= N) return;
    const int lane = threadIdx.x % 64;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const T *qunit = q_win + (((int64_t)g.b * L + g.l) * Hq + (int64_t)g.h * G) * W * D;
    const T *kunit = k + ((int64_t)g.l * k_layer_rows + (int64_t)g.h * T_ + g.s0) * D;
    const int ntile = (int)ceil_div(key_end - key_begin, KT::TK);
    KT::template load<NW>(kbA, kunit, key_begin, N, wave, lane);
    QFrags<T, D> q;
    q.load(qunit, R, wave, lane);
    float thr[NRB];
    int pos[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
        const int row = wave * 64 + rb * M::BM + lane % M::BM;
        pos[rb] = row < R ? N - W + row % W : -1;
        thr[rb] = row < R ? threshold_value(pre[u * R + row]) : INFINITY;
    }
    TC<T, D> zero[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) zero[rb] = M::zero();
    // the wavefronts' picks of tile t sit in csum[t & 1]; they are added and
    // stored after the next barrier
    auto flush = [&](int t) {
        const int key0 = key_begin + t * KT::TK;
        for (int j = threadIdx.x; j < KT::TK; j += 64 * NW) {
            uint32_t v = 0u;
            for (int w = 0; w < NW; ++w)
                for (int rb = 0; rb < NRB; ++rb) v += csum[t & 1][w][rb][j];
            if (key0 + j < N) orow[key0 + j] = (float)v;
        }
    };
    auto step = [&](int t, char *cur, char *nxt, auto mask) {
        constexpr bool MASK = decltype(mask)::value;
        barrier_after_loads();      // tile t landed; tile t - 1 finished everywhere
        if (t > 0) flush(t - 1);
        const int key0 = key_begin + t * KT::TK;
        if (t + 1 < ntile) KT::template load<NW>(nxt, kunit, key0 + KT::TK, N, wave, lane);
        const TsCountStep<T, D, MASK> f{&csum[t & 1][wave][0][0], thr, pos, lane, key0};
        if (MASK) tile_sweep_plain<T, D, true>(cur, q, zero, lane, f);
        else tile_sweep<T, D, true>(cur, q, zero, lane, f);
    };
    const int nfull = full_tiles(key_begin, ntile, KT::TK, N, W);
    int t = 0;
    for (; t + 1 < nfull; t += 2) {
        step(t, kbA, kbB, std::false_type{});
        step(t + 1, kbB, kbA, std::false_type{});
    }
    for (; t < ntile; ++t) {
        if (t & 1) step(t, kbB, kbA, std::true_type{});
        else step(t, kbA, kbB, std::true_type{});
    }
    barrier_after_loads();
    flush(ntile - 1);
}

template <typename T, int D, int NW>
static void launch_topshare(hipStream_t s, const ScorePlan &p, int B, int L, int Hq, int Hkv, int W,
                            const int32_t *cu_seqlens, int64_t ntok, const void *q_win, const void *k,
                            int64_t k_layer_rows, int ratio_bp, float *counts, void *ws) {
    constexpr int DB = TsDigits<NW>::DB, NB = TsDigits<NW>::NB;
    const int R = (Hq / Hkv) * W;
    const int64_t units = (int64_t)L * Hkv * B, nrows = units * R;
    uint32_t *pre = reinterpret_cast<uint32_t *>(ws);
    uint32_t *need = pre + nrows;
    uint32_t *gh = need + nrows;
    uint32_t *busy = gh + nrows * TS_MAXBINS;               // [TS_MAXPASS][units]
    uint32_t *gflag = busy + TS_MAXPASS * units;            // [units]
    uint32_t *gcount = gflag + units;                       // [rows]
    uint32_t *gcand = gcount + nrows;                       // [rows][TS_CMAX]
    const T *q = reinterpret_cast<const T *>(q_win);
    const T *kk = reinterpret_cast<const T *>(k);
    const dim3 rgrid((unsigned)ceil_div(nrows, 256));
    const dim3 grid((unsigned)(units * p.nchunk));
    static_assert((32 + DB - 1) / DB <= TS_MAXPASS, "flag words");
    ts_init_kernel<<<rgrid, 256, 0, s>>>(nrows, R, W, B, Hkv, cu_seqlens, ntok, ratio_bp, pre, need, gh, NB, busy,
                                         units, gcount, gflag);
    for (int pass = 0, hi = 32; hi > 0; ++pass) {
        const int sh = std::max(0, hi - DB), width = hi - sh;
        const uint32_t *busy_in = pass > 0 ? busy + (pass - 1) * units : nullptr;
        uint32_t *busy_out = sh > 0 ? busy + pass * units : nullptr;
        if (pass == 0)
            ts_hist_kernel<T, D, NW, true><<<grid, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok, q, kk,
                                                                  k_layer_rows, p.nchunk, p.chunk_keys, sh, width,
                                                                  busy_in, pre, gh);
        else
            ts_hist_kernel<T, D, NW, false><<<grid, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok, q, kk,
                                                                   k_layer_rows, p.nchunk, p.chunk_keys, sh, width,
                                                                   busy_in, pre, gh);
        const bool gather = 32 - sh >= TS_GATHER_BITS && 32 - hi < TS_GATHER_BITS;   // first digit past 18 bits
        ts_digit_kernel<<<rgrid, 256, 0, s>>>(nrows, R, NB, sh, width, busy_in, busy_out, pre, need, gh,
                                              gather ? gflag : nullptr);
        if (gather) {
            ts_gather_kernel<T, D, NW><<<grid, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok, q, kk,
                                                               k_layer_rows, p.nchunk, p.chunk_keys, sh, gflag, pre,
                                                               need, gcount, gcand);
            ts_pick_kernel<<<rgrid, 256, 0, s>>>(nrows, gcount, gcand, pre, need);
        }
        hi = sh;
    }
    ts_count_kernel<T, D, NW><<<grid, 64 * NW, 0, s>>>(B, L, Hq, Hkv, W, cu_seqlens, ntok, q, kk, k_layer_rows,
                                                      p.nchunk, p.chunk_keys, pre, counts);
}

template <typename T, int D>
static int topshare_dispatch(hipStream_t s, int B, int L, int Hq, int Hkv, int W, const int32_t *cu_seqlens,
                             int64_t ntok, int max_seqlen, const void *q_win, const void *k, int64_t k_layer_rows,
                             int ratio_bp, float *counts, void *ws) {
    const int R = (Hq / Hkv) * W;
    const int nw = (int)ceil_div(R, 64);
    const ScorePlan p = score_plan(B, L, Hkv, max_seqlen);
    if (nw <= 1) launch_topshare<T, D, 1>(s, p, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, ratio_bp, counts, ws);
    else if (nw <= 2) launch_topshare<T, D, 2>(s, p, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, ratio_bp, counts, ws);
    else if (nw <= 4) launch_topshare<T, D, 4>(s, p, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, ratio_bp, counts, ws);
    else launch_topshare<T, D, 8>(s, p, B, L, Hq, Hkv, W, cu_seqlens, ntok, q_win, k, k_layer_rows, ratio_bp, counts, ws);
    return launch_status("sg_score_topshare");
}

}  // namespace sg

using namespace sg;

extern "C" size_t sg_score_topshare_workspace_size(int B, int L, int Hq, int Hkv, int d, int W, int max_seqlen) {
    if (B <= 0 || L <= 0 || Hkv <= 0 || Hq <= 0 || W <= 0 || max_seqlen <= 0 || d <= 0) return 0;
    const int64_t units = (int64_t)L * Hkv * B, rows = units * (Hq / Hkv) * W;
    return (size_t)(rows * (3 + TS_MAXBINS + TS_CMAX) + units * (TS_MAXPASS + 1)) * sizeof(uint32_t);
}

extern "C" int sg_score_topshare(void *stream, sg_dtype dt, int B, int L, int Hq, int Hkv, int d, int W,
                                 const int32_t *cu_seqlens, int64_t T, int max_seqlen, const void *q_win,
                                 const void *k, int64_t k_layer_rows, int ratio_bp, float *counts, void *ws,
                                 size_t ws_bytes) {
    const char *name = "sg_score_topshare";
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "%s: unknown dtype %d", name, (int)dt);
    SG_REQUIRE(B >= 1 && L >= 1 && Hq >= 1 && Hkv >= 1 && Hq % Hkv == 0, SG_EINVAL,
               "%s: need B, L, Hq, Hkv >= 1 and Hq %% Hkv == 0", name);
    SG_REQUIRE(d == 64 || d == 128, SG_EUNSUPPORTED, "%s: head dimension %d not supported (64 or 128)", name, d);
    SG_REQUIRE(W >= 1, SG_EINVAL, "%s: window must be >= 1", name);
    SG_REQUIRE((int64_t)(Hq / Hkv) * W <= SC_MAXR, SG_EUNSUPPORTED, "%s: G*W = %d above %d", name, (Hq / Hkv) * W,
               SC_MAXR);
    SG_REQUIRE(ratio_bp >= 1 && ratio_bp <= 10000, SG_EINVAL, "%s: ratio_bp %d outside [1, 10000]", name, ratio_bp);
    SG_REQUIRE(T >= 0 && max_seqlen >= 0 && k_layer_rows >= 0, SG_EINVAL, "%s: negative size", name);
    SG_REQUIRE(max_seqlen <= (1 << 30), SG_EINVAL, "%s: max_seqlen too large", name);
    if (T == 0 || max_seqlen == 0) return SG_OK;
    SG_REQUIRE(cu_seqlens && q_win && k && counts, SG_EINVAL, "%s: null pointer", name);
    SG_REQUIRE(aligned16(q_win) && aligned16(k), SG_EINVAL, "%s: q_win and k must be 16-byte aligned", name);
    const int64_t units = (int64_t)L * Hkv * B;
    SG_REQUIRE(units * ceil_div(max_seqlen, 128) <= 0x7fffffff, SG_EINVAL, "%s: grid too large", name);
    SG_REQUIRE(units * (Hq / Hkv) * W <= (int64_t)0x7fffffff, SG_EINVAL, "%s: too many rows", name);
    const size_t need = sg_score_topshare_workspace_size(B, L, Hq, Hkv, d, W, max_seqlen);
    SG_REQUIRE(ws && ws_bytes >= need, SG_EWORKSPACE, "%s: workspace %zu < %zu", name, ws_bytes, need);
    SG_REQUIRE(aligned16(ws), SG_EINVAL, "%s: workspace must be 16-byte aligned", name);
    hipStream_t s = as_stream(stream);
    if (dt == SG_BF16) {
        if (d == 128) return topshare_dispatch<uint16_t, 128>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, ratio_bp, counts, ws);
        return topshare_dispatch<uint16_t, 64>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, ratio_bp, counts, ws);
    }
    if (d == 128) return topshare_dispatch<float, 128>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, ratio_bp, counts, ws);
    return topshare_dispatch<float, 64>(s, B, L, Hq, Hkv, W, cu_seqlens, T, max_seqlen, q_win, k, k_layer_rows, ratio_bp, counts, ws);
}
