// Exact top-k of a row held in registers by one workgroup of NT threads (1024
// by default): wavefront-level radix select, shared by sg_topk and the
// decode-time selection.
//
// Scores are mapped to order-preserving 32-bit keys (NaN -> 0, the lowest key;
// -0 -> +0).  Four 8-bit digit passes, most significant first, narrow down the
// exact k-th largest key T and how many entries equal to T must be taken
// ("need").  Histograms are built per wavefront with LDS atomics: the lanes
// sharing the digit of the wavefront's first candidate (every lane when keys
// tie) add their count in one atomic, every other lane adds its own (measured
// on gfx950: 2.1 us per pass over 32K random keys against 15.7 us for finding
// each digit's lane group with ballots; plain per-lane atomics on 32K equal
// keys take 27 us).  The output pass keeps every key > T and the first
// `need` keys == T in index order, written at positions given by one
// block-wide scan, so the ids come out ascending with ties resolved to the
// lower index.
#pragma once

#include "sg_internal.h"

namespace sg {

constexpr int TOPK_THREADS = 1024;
constexpr int TOPK_WAVES = TOPK_THREADS / 64;

__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;  // NaN: below every number
    if (u == 0x80000000u) u = 0u;                     // -0 ranks as +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// inclusive scan over the NT threads of the block; `tot` receives the block total
template <int NT = TOPK_THREADS>
__device__ __forceinline__ int block_scan_incl(int x, int *wsum, int &tot) {
    constexpr int NWV = NT / 64;
    const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int before = 0;
    tot = 0;
#pragma unroll
    for (int w = 0; w < NWV; ++w) {
        const int v = wsum[w];
        before += (w < wave) ? v : 0;
        tot += v;
    }
    __syncthreads();
    return x + before;
}

template <int NT>
struct SelectSmemT {
    uint32_t hist[NT / 64][256];
    int wsum[NT / 64];
    int wsum2[NT / 64];
    uint32_t digit;
    int rem;
};
using SelectSmem = SelectSmemT<TOPK_THREADS>;

// Thread t holds keys key[0 .. nv) of row entries first + i.  Writes the ids
// of the kk largest keys (ties: lower id), ascending, to out[0 .. kk).
// 0 < kk <= number of valid keys.  Every thread of the block must call it.
template <int ITEMS, int NT = TOPK_THREADS>
__device__ __forceinline__ void select_top(const uint32_t (&key)[ITEMS], int nv, int first, int kk, int32_t *out,
                                           SelectSmemT<NT> &sm) {
    constexpr int NWV = NT / 64;
    const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
    uint32_t prefix = 0, pmask = 0;
    int rem = kk;
#pragma unroll 1
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        for (int i = tid; i < NWV * 256; i += NT) (&sm.hist[0][0])[i] = 0;
        __syncthreads();
#pragma unroll
        for (int i = 0; i < ITEMS; ++i) {
            const bool cand = i < nv && (key[i] & pmask) == prefix;
            const uint64_t act = __ballot(cand);
            if (act == 0) continue;  // uniform across the wavefront
            const uint32_t dg = (key[i] >> shift) & 255u;
            // the lanes sharing the first candidate's digit (all of them when
            // the keys tie) add their count with one atomic; every other lane
            // adds its own one (few of them share a bin)
            const int lead = __ffsll((unsigned long long)act) - 1;
            const uint32_t d0 = (uint32_t)__builtin_amdgcn_readlane((int)dg, lead);
            const uint64_t same = __ballot(cand && dg == d0);
            if (cand) {
                if (dg != d0) atomicAdd(&sm.hist[wave][dg], 1u);
                else if (lane == lead) atomicAdd(&sm.hist[wave][d0], (uint32_t)__popcll(same));
            }
        }
        __syncthreads();
        // threads 0..255 own one digit each, in descending digit order
        int cnt = 0;
        if (tid < 256) {
            const int dg = 255 - tid;
#pragma unroll
            for (int w = 0; w < NWV; ++w) cnt += sm.hist[w][dg];
        }
        int tot;
        const int incl = block_scan_incl<NT>(tid < 256 ? cnt : 0, sm.wsum, tot);
        const int excl = incl - cnt;
        if (tid < 256 && cnt > 0 && excl < rem && rem <= incl) {
            sm.digit = 255 - tid;
            sm.rem = rem - excl;
        }
        __syncthreads();
        prefix |= sm.digit << shift;
        pmask |= 255u << shift;
        rem = sm.rem;
        __syncthreads();
    }
    const uint32_t thr = prefix;
    const int need = rem;  // entries equal to thr that are taken, lowest index first

    int gt = 0, eq = 0;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
        gt += (i < nv && key[i] > thr) ? 1 : 0;
        eq += (i < nv && key[i] == thr) ? 1 : 0;
    }
    int tot_gt, tot_eq;
    const int gt_pre = block_scan_incl<NT>(gt, sm.wsum, tot_gt) - gt;
    const int eq_pre = block_scan_incl<NT>(eq, sm.wsum2, tot_eq) - eq;
    int pos = gt_pre + min(eq_pre, need);
    int eq_seen = eq_pre;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
        if (i < nv) {
            if (key[i] > thr) {
                out[pos++] = first + i;
            } else if (key[i] == thr) {
                if (eq_seen < need) out[pos++] = first + i;
                ++eq_seen;
            }
        }
    }
}

}  // namespace sg
