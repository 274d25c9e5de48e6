// The MFMA engine of the score kernels (gfx950): a wavefront's 64 query rows
// as operand fragments, the (key block, row block) products of one LDS K tile
// with the vector work of each block handed to a functor, and the split of a
// chunk into tiles every row sees whole and tiles under the causal limit.
#pragma once

#include <algorithm>

#include "score_common.h"

namespace sg {

template <typename T, int D>
using TA = typename MT<T, D>::A;
template <typename T, int D>
using TC = typename MT<T, D>::C;

// The wavefront's 64 query rows (rows >= R are zero) as operand fragments.
template <typename T, int D>
struct QFrags {
    static constexpr int NRB = 64 / MT<T, D>::BM;     // row blocks per wavefront
    TA<T, D> f[NRB][MT<T, D>::KS];
    __device__ __forceinline__ void load(const T *qunit, int R, int wave, int lane) {
        using M = MT<T, D>;
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
            const int row = wave * 64 + rb * M::BM + lane % M::BM;
            const T *p = qunit + (int64_t)min(row, R - 1) * D;
#pragma unroll
            for (int ks = 0; ks < M::KS; ++ks) {
                const TA<T, D> x = M::load_global(p, ks, lane);
                f[rb][ks] = row < R ? x : TA<T, D>{};
            }
        }
    }
};

// One (key block, row block) product over the whole contraction.  KEY_ROWS:
// C[key][row] (stats), else C[row][key] (colsum).
template <typename T, int D, bool KEY_ROWS>
__device__ __forceinline__ TC<T, D> block_mma(const TA<T, D> (&kf)[MT<T, D>::KS], const TA<T, D> (&qf)[MT<T, D>::KS]) {
    using M = MT<T, D>;
    TC<T, D> acc = KEY_ROWS ? M::mma(kf[0], qf[0], M::zero()) : M::mma(qf[0], kf[0], M::zero());
#pragma unroll
    for (int ks = 1; ks < M::KS; ++ks) acc = KEY_ROWS ? M::mma(kf[ks], qf[ks], acc) : M::mma(qf[ks], kf[ks], acc);
    return acc;
}

template <typename T, int D>
__device__ __forceinline__ void load_kf(const char *buf, int kb, int lane, TA<T, D> (&kf)[MT<T, D>::KS]) {
#pragma unroll
    for (int ks = 0; ks < MT<T, D>::KS; ++ks) kf[ks] = KTile<T, D>::frag(buf, kb, ks, lane);
}

// One block product, accumulated onto c0, whose key fragments are refilled,
// right behind each MFMA that reads them, with key block `next` of the tile
// (when next >= 0).
template <typename T, int D, bool KEY_ROWS>
__device__ __forceinline__ TC<T, D> block_mma_refill(const char *buf, int next, int lane, const TC<T, D> &c0,
                                                     TA<T, D> (&kf)[MT<T, D>::KS],
                                                     const TA<T, D> (&qf)[MT<T, D>::KS]) {
    using M = MT<T, D>;
    TC<T, D> acc = c0;
#pragma unroll
    for (int ks = 0; ks < M::KS; ++ks) {
        acc = KEY_ROWS ? M::mma(kf[ks], qf[ks], acc) : M::mma(qf[ks], kf[ks], acc);
        if (next >= 0) kf[ks] = KTile<T, D>::frag(buf, next, ks, lane);
    }
    return acc;
}

// All (key block, row block) products of the tile in `buf`, key block major.
// Software pipelined: step b issues the MFMAs of block b + 1 and then hands
// block b to valu(acc, kb, rb).  One set of key fragments: the last block of
// a key block refills them with the next key block's behind its own MFMAs.
// Scheduling barriers keep the compiler from hoisting later loads, and group
// barriers interleave each MFMA with a share of the vector work.
template <typename T, int D, bool KEY_ROWS, int TKEYS = KTile<T, D>::TK, typename F>
__device__ __forceinline__ void tile_sweep(const char *buf, const QFrags<T, D> &q,
                                           const TC<T, D> (&c0)[QFrags<T, D>::NRB], int lane, F &&valu) {
    constexpr int NKB = KTile<T, D, TKEYS>::NKB, NRB = QFrags<T, D>::NRB, NB = NKB * NRB;
    // a block's vector work is about 3 instructions per output value
    constexpr int VALU_PER_MFMA = (3 * MT<T, D>::NV + MT<T, D>::KS - 1) / MT<T, D>::KS;
    TA<T, D> kf[MT<T, D>::KS];
    load_kf<T, D>(buf, 0, lane, kf);
    TC<T, D> acc = block_mma_refill<T, D, KEY_ROWS>(buf, NRB == 1 && NKB > 1 ? 1 : -1, lane, c0[0], kf, q.f[0]), nacc;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        __builtin_amdgcn_sched_barrier(0);
        if (b + 1 < NB) {
            const int nkb = (b + 1) / NRB, nrb = (b + 1) % NRB;
            const int refill = nrb == NRB - 1 && nkb + 1 < NKB ? nkb + 1 : -1;
            nacc = block_mma_refill<T, D, KEY_ROWS>(buf, refill, lane, c0[nrb], kf, q.f[nrb]);
        }
        valu(acc, b / NRB, b % NRB);
        // issue order of the step: each MFMA of block b + 1 followed by a share
        // of block b's vector work, so the two overlap
        if (b + 1 < NB) {
#pragma unroll
            for (int i = 0; i < MT<T, D>::KS; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                // MFMA
                __builtin_amdgcn_sched_group_barrier(0x002, VALU_PER_MFMA, 0);    // VALU
            }
        }
        acc = nacc;
    }
    __builtin_amdgcn_sched_barrier(0);
}

// The same products without pipelining, for the few tiles at the end of a
// prompt (keeps their masking work from raising the register needs of the
// main loop).
template <typename T, int D, bool KEY_ROWS, int TKEYS = KTile<T, D>::TK, typename F>
__device__ __forceinline__ void tile_sweep_plain(const char *buf, const QFrags<T, D> &q,
                                                 const TC<T, D> (&c0)[QFrags<T, D>::NRB], int lane, F &&valu) {
    constexpr int NKB = KTile<T, D, TKEYS>::NKB, NRB = QFrags<T, D>::NRB;
#pragma unroll 1
    for (int kb = 0; kb < NKB; ++kb) {
        TA<T, D> kf[MT<T, D>::KS];
        load_kf<T, D>(buf, kb, lane, kf);
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
            TC<T, D> acc = block_mma_refill<T, D, KEY_ROWS>(buf, -1, lane, c0[rb], kf, q.f[rb]);
            valu(acc, kb, rb);
        }
    }
}

// Tiles [0, nfull) of a chunk lie wholly before the first window position, so
// every row sees every key of them; the rest need the causal mask.
__device__ __forceinline__ int full_tiles(int key_begin, int ntile, int tk, int N, int W) {
    const int span = N - W + 1 - key_begin;            // keys key_begin .. N - W are seen by every row
    return max(0, min(ntile, span >= 0 ? span / tk : 0));
}

// Launch plan: each unit's keys split into chunks of chunk_keys (a multiple
// of the LDS tile), one workgroup per (unit, chunk).  Long chunks keep the
// per-workgroup set-up (query fragments, row normalisers) small against the
// streaming work; short prompts or few units take shorter chunks so that the
// launch still has enough workgroups to fill the chip.
struct ScorePlan {
    int chunk_keys, nchunk;
};

inline ScorePlan score_plan(int B, int L, int Hkv, int max_seqlen) {
    constexpr int64_t MIN_WG = 1024;                      // two rounds of two workgroups per CU
    constexpr int TILE = 128;                             // chunk granularity (keys)
    const int64_t units = (int64_t)B * L * Hkv;
    ScorePlan p;
    if (units * ceil_div(max_seqlen, SC_CHUNK) >= MIN_WG) {
        // full-length chunks already fill the chip: keep them, so that the
        // chunk boundaries (and the rounding of every score) do not depend on
        // how many requests one call covers
        p.chunk_keys = SC_CHUNK;
    } else {
        const int64_t want = std::max<int64_t>(1, ceil_div(MIN_WG, units));   // chunks per unit
        p.chunk_keys = (int)std::min<int64_t>(
            SC_CHUNK, std::max<int64_t>(TILE, ceil_div(ceil_div(max_seqlen, want), TILE) * TILE));
    }
    p.nchunk = (int)ceil_div(max_seqlen, p.chunk_keys);
    return p;
}

}  // namespace sg
