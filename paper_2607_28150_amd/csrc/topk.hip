// sg_topk: exact budgeted top-k per unit row by wavefront-level radix select.
//
// One 1024-thread workgroup owns one (request, layer, KV head) row (or, for
// block selection, one request's row of L * M block importances).  The row is
// held in registers, ITEMS consecutive keys per thread (up to 80).  Scores
// are mapped to order-preserving 32-bit keys (NaN -> 0, the lowest key;
// -0 -> +0).  Four 8-bit digit passes, most significant first, narrow down the exact k-th
// largest key T and how many entries equal to T must be taken ("need").
// Histograms are built per wavefront: the lanes holding the same digit are
// found with eight ballots (one per digit bit), and one lane per distinct
// digit adds the group's popcount, so LDS atomics never collide inside a
// wavefront.  The output pass keeps every key > T and the first `need` keys
// == T in index order, written at positions given by one block-wide scan, so
// the ids come out ascending with ties resolved to the lower index.
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

// inclusive scan over the 1024 threads of the block; `tot` receives the block total
__device__ __forceinline__ int block_scan_incl(int x, int *wsum, int &tot) {
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
    for (int w = 0; w < TOPK_WAVES; ++w) {
        const int v = wsum[w];
        before += (w < wave) ? v : 0;
        tot += v;
    }
    __syncthreads();
    return x + before;
}

template <int ITEMS>
__global__ __launch_bounds__(TOPK_THREADS) void topk_kernel(int B, const int32_t *__restrict__ cu_seqlens,
                                                            int64_t T, const int32_t *__restrict__ cu_k,
                                                            int64_t K_total, const float *__restrict__ scores,
                                                            int32_t *__restrict__ idx) {
    __shared__ uint32_t hist[TOPK_WAVES][256];
    __shared__ int wsum[TOPK_WAVES];
    __shared__ int wsum2[TOPK_WAVES];
    __shared__ uint32_t s_digit;
    __shared__ int s_rem;

    const int b = blockIdx.x % B;
    const int64_t lh = blockIdx.x / B;
    const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
    const int64_t c0 = cu_k[b], c1 = cu_k[b + 1];
    const int64_t s0 = cu_seqlens[b], s1 = cu_seqlens[b + 1];
    if (c0 < 0 || c1 < c0 || c1 > K_total) return;  // no writable segment
    int32_t *out = idx + lh * K_total + c0;
    const int64_t kk = c1 - c0;
    const int64_t N = s1 - s0;
    if (s0 < 0 || s1 < s0 || s1 > T || kk > N || N > (int64_t)ITEMS * TOPK_THREADS) {
        for (int64_t i = tid; i < kk; i += TOPK_THREADS) out[i] = -1;
        return;
    }
    if (kk == 0) return;
    if (kk == N) {  // everything is selected
        for (int64_t i = tid; i < kk; i += TOPK_THREADS) out[i] = (int32_t)i;
        return;
    }
    const float *row = scores + lh * T + s0;
    const int first = tid * ITEMS;
    const int nv = (int)max<int64_t>(0, min<int64_t>(ITEMS, N - first));
    uint32_t key[ITEMS];
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) key[i] = i < nv ? order_key(row[first + i]) : 0u;

    uint32_t prefix = 0, pmask = 0;
    int rem = (int)kk;
#pragma unroll 1
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        for (int i = tid; i < TOPK_WAVES * 256; i += TOPK_THREADS) (&hist[0][0])[i] = 0;
        __syncthreads();
#pragma unroll
        for (int i = 0; i < ITEMS; ++i) {
            const bool cand = i < nv && (key[i] & pmask) == prefix;
            const uint64_t act = __ballot(cand);
            if (act == 0) continue;  // uniform across the wavefront
            const uint32_t dg = (key[i] >> shift) & 255u;
            uint64_t peers = act;
#pragma unroll
            for (int bit = 0; bit < 8; ++bit) {
                const uint64_t bm = __ballot((dg >> bit) & 1u);
                peers &= ((dg >> bit) & 1u) ? bm : ~bm;
            }
            if (cand && lane == __ffsll((unsigned long long)peers) - 1)
                atomicAdd(&hist[wave][dg], (uint32_t)__popcll(peers));
        }
        __syncthreads();
        // threads 0..255 own one digit each, in descending digit order
        int cnt = 0;
        if (tid < 256) {
            const int dg = 255 - tid;
#pragma unroll
            for (int w = 0; w < TOPK_WAVES; ++w) cnt += hist[w][dg];
        }
        int tot;
        const int incl = block_scan_incl(tid < 256 ? cnt : 0, wsum, tot);
        const int excl = incl - cnt;
        if (tid < 256 && cnt > 0 && excl < rem && rem <= incl) {
            s_digit = 255 - tid;
            s_rem = rem - excl;
        }
        __syncthreads();
        prefix |= s_digit << shift;
        pmask |= 255u << shift;
        rem = s_rem;
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
    const int gt_pre = block_scan_incl(gt, wsum, tot_gt) - gt;
    const int eq_pre = block_scan_incl(eq, wsum2, tot_eq) - eq;
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

using namespace sg;

extern "C" int sg_topk(void *stream, int B, int L, int Hkv, const int32_t *cu_seqlens, int64_t T, int max_seqlen,
                       const int32_t *cu_k, int64_t K_total, const float *scores, int32_t *idx) {
    SG_REQUIRE(B >= 1 && L >= 1 && Hkv >= 1, SG_EINVAL, "sg_topk: B, L, Hkv must be >= 1");
    SG_REQUIRE(T >= 0 && K_total >= 0 && max_seqlen >= 0, SG_EINVAL, "sg_topk: negative size");
    SG_REQUIRE(max_seqlen <= 80 * TOPK_THREADS, SG_EUNSUPPORTED, "sg_topk: max_seqlen %d above %d", max_seqlen,
               80 * TOPK_THREADS);
    if (K_total == 0) return SG_OK;
    SG_REQUIRE(cu_seqlens && cu_k && scores && idx, SG_EINVAL, "sg_topk: null pointer");
    const int64_t blocks = (int64_t)B * L * Hkv;
    SG_REQUIRE(blocks <= 0x7fffffff, SG_EINVAL, "sg_topk: too many rows");
    hipStream_t s = as_stream(stream);
    if (max_seqlen <= 2 * TOPK_THREADS)
        topk_kernel<2><<<(unsigned)blocks, TOPK_THREADS, 0, s>>>(B, cu_seqlens, T, cu_k, K_total, scores, idx);
    else if (max_seqlen <= 8 * TOPK_THREADS)
        topk_kernel<8><<<(unsigned)blocks, TOPK_THREADS, 0, s>>>(B, cu_seqlens, T, cu_k, K_total, scores, idx);
    else if (max_seqlen <= 32 * TOPK_THREADS)
        topk_kernel<32><<<(unsigned)blocks, TOPK_THREADS, 0, s>>>(B, cu_seqlens, T, cu_k, K_total, scores, idx);
    else if (max_seqlen <= 64 * TOPK_THREADS)
        topk_kernel<64><<<(unsigned)blocks, TOPK_THREADS, 0, s>>>(B, cu_seqlens, T, cu_k, K_total, scores, idx);
    else    // block rows of up to 80 layers x 1024 blocks
        topk_kernel<80><<<(unsigned)blocks, TOPK_THREADS, 0, s>>>(B, cu_seqlens, T, cu_k, K_total, scores, idx);
    return launch_status("sg_topk");
}
