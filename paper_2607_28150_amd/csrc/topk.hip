// sg_topk: exact budgeted top-k per unit row by wavefront-level radix select
// (select_common.h).
//
// One workgroup owns one (request, layer, KV head) row (or, for block
// selection, one request's row of L * M block importances).  The row is held
// in registers, ITEMS consecutive keys per thread (up to 80).  Rows of 8K to
// 32K keys take 512 threads with 64 keys each (104 VGPRs, 8 KB of LDS) when
// the call has at least two rows per CU: two workgroups then share a CU, and
// one fits beside a score workgroup when the select region runs a request
// pair's top-k beside the next pair's score, where 1024 threads with 32 keys
// each (110 VGPRs, 84 KB of LDS for the staged row) held a whole CU.  64
// requests (16,384 rows of 2.6K-32.6K keys): 2.04 against 2.75 ms alone, the
// select region 46.1 against 46.7 ms.  With fewer rows the 1024-thread form
// finishes each row sooner (256 rows of 32K keys: 0.050-0.058 against
// 0.062 ms).
#include "select_common.h"

namespace sg {

template <int ITEMS, int NT = TOPK_THREADS>
__global__ __launch_bounds__(NT) void topk_kernel(int B, const int32_t *__restrict__ cu_seqlens,
                                                            int64_t T, const int32_t *__restrict__ cu_k,
                                                            int64_t K_total, const float *__restrict__ scores,
                                                            int32_t *__restrict__ idx) {
    __shared__ SelectSmemT<NT> sm;
    // long rows pass through LDS in chunks: coalesced loads, then each thread
    // reads its consecutive keys (one pad word per 32 keeps the reads free of
    // bank conflicts); reading them straight from memory would touch a new
    // cache line per lane and instruction
    constexpr bool STAGE = ITEMS >= 16 && ITEMS <= 32;   // wider rows: no registers to spare
    constexpr int CH = 16384;
    __shared__ float stage[STAGE ? CH + CH / 32 : 1];

    const int b = blockIdx.x % B;
    const int64_t lh = blockIdx.x / B;
    const int tid = threadIdx.x;
    const int64_t c0 = cu_k[b], c1 = cu_k[b + 1];
    const int64_t s0 = cu_seqlens[b], s1 = cu_seqlens[b + 1];
    if (c0 < 0 || c1 < c0 || c1 > K_total) return;  // no writable segment
    int32_t *out = idx + lh * K_total + c0;
    const int64_t kk = c1 - c0;
    const int64_t N = s1 - s0;
    if (s0 < 0 || s1 < s0 || s1 > T || kk > N || N > (int64_t)ITEMS * NT) {
        for (int64_t i = tid; i < kk; i += NT) out[i] = -1;
        return;
    }
    if (kk == 0) return;
    if (kk == N) {  // everything is selected
        for (int64_t i = tid; i < kk; i += NT) out[i] = (int32_t)i;
        return;
    }
    const float *row = scores + lh * T + s0;
    const int first = tid * ITEMS;
    const int nv = (int)max<int64_t>(0, min<int64_t>(ITEMS, N - first));
    uint32_t key[ITEMS];
    if constexpr (STAGE) {
#pragma unroll
        for (int i = 0; i < ITEMS; ++i) key[i] = 0u;
        for (int c0 = 0; c0 < (int)N; c0 += CH) {       // uniform
            const int cn = min<int64_t>(CH, N - c0);
#pragma unroll 4
            for (int j = tid; j < cn; j += NT) stage[j + (j >> 5)] = row[c0 + j];
            __syncthreads();
#pragma unroll
            for (int i = 0; i < ITEMS; ++i) {
                const int x = first + i - c0;
                if (i < nv && x >= 0 && x < cn) key[i] = order_key(stage[x + (x >> 5)]);
            }
            __syncthreads();
        }
    } else if (ITEMS % 4 == 0 && nv == ITEMS && (reinterpret_cast<uintptr_t>(row + first) & 15u) == 0) {
        // a thread's keys whole and 16-byte aligned: vector loads
#pragma unroll
        for (int i = 0; i < ITEMS; i += 4) {
            const float4 x = *reinterpret_cast<const float4 *>(row + first + i);
            key[i] = order_key(x.x);
            key[i + 1] = order_key(x.y);
            key[i + 2] = order_key(x.z);
            key[i + 3] = order_key(x.w);
        }
    } else {
#pragma unroll
        for (int i = 0; i < ITEMS; ++i) key[i] = i < nv ? order_key(row[first + i]) : 0u;
    }

    select_top<ITEMS, NT>(key, nv, first, (int)kk, out, sm);
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
    else if (max_seqlen <= 32 * TOPK_THREADS && blocks >= 2 * (int64_t)device_cus())
        topk_kernel<64, 512><<<(unsigned)blocks, 512, 0, s>>>(B, cu_seqlens, T, cu_k, K_total, scores, idx);
    else if (max_seqlen <= 32 * TOPK_THREADS)
        topk_kernel<32><<<(unsigned)blocks, TOPK_THREADS, 0, s>>>(B, cu_seqlens, T, cu_k, K_total, scores, idx);
    else if (max_seqlen <= 64 * TOPK_THREADS)
        topk_kernel<64><<<(unsigned)blocks, TOPK_THREADS, 0, s>>>(B, cu_seqlens, T, cu_k, K_total, scores, idx);
    else    // block rows of up to 80 layers x 1024 blocks
        topk_kernel<80><<<(unsigned)blocks, TOPK_THREADS, 0, s>>>(B, cu_seqlens, T, cu_k, K_total, scores, idx);
    return launch_status("sg_topk");
}
