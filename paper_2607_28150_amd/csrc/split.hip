// sg_split: Algorithm 1 (KV index splitting and reordering), one wavefront
// per row of the KV index.
//
// The row is walked in 64-entry chunks.  Each lane gathers the mask value of
// its entry (operator 1); three ballots give, for every lane, how many earlier
// lanes carry each mask value, so the stable partitions (operators 2, 3) and
// the stable descending sort by mask value (operators 4, 5) are all prefix
// popcounts plus a running per-value count.  For a reordered row a first pass
// counts the remote and local entries, which fixes where the local and pad
// blocks start; without reordering the row is read once (the 64-request
// decode step's split: 37.3 M entries, 0.34 ms with both passes).  Each pass
// takes four chunks at a time, issuing all their loads together.
#include "sg_internal.h"

namespace sg {

constexpr int SPLIT_WAVES = 4;
constexpr int SPLIT_GROUP = 4;     // 64-entry chunks whose loads are issued together

__global__ __launch_bounds__(64 * SPLIT_WAVES) void split_kernel(
    int rows, const int32_t *__restrict__ row_off, int64_t total, const int32_t *__restrict__ kv_index,
    const int8_t *__restrict__ mask, int64_t mask_bytes, const int64_t *__restrict__ mask_off,
    const int32_t *__restrict__ mask_len, int reorder, int32_t *__restrict__ out_index,
    int32_t *__restrict__ local, int32_t *__restrict__ remote, int32_t *__restrict__ n_local,
    int32_t *__restrict__ n_remote, int32_t *__restrict__ n_kept) {
    const int r = blockIdx.x * SPLIT_WAVES + threadIdx.x / 64;
    if (r >= rows) return;
    const int lane = threadIdx.x % 64;
    int64_t o = row_off[r], e = row_off[r + 1];
    if (o < 0 || e < o || e > total) {  // bad device metadata: empty row
        if (lane == 0) {
            n_local[r] = 0;
            n_remote[r] = 0;
            if (n_kept) n_kept[r] = 0;
        }
        return;
    }
    const int64_t n = e - o;
    const int64_t moff = mask_off[r];
    const int32_t mlen = moff >= 0 ? mask_len[r] : 0;   // a negative offset makes every entry a pad
    const uint64_t lt = lanemask_lt();

    // The loads of SPLIT_GROUP chunks are issued together (indices, then mask
    // values at clamped addresses), so a group costs two memory round trips.
    const bool has_mask = mask_bytes > 0;
    auto load_group = [&](int64_t c, int32_t (&t)[SPLIT_GROUP], int (&m)[SPLIT_GROUP]) {
#pragma unroll
        for (int u = 0; u < SPLIT_GROUP; ++u) t[u] = kv_index[o + min<int64_t>(c + u * 64 + lane, n - 1)];
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < SPLIT_GROUP; ++u) {
            const bool ok = has_mask && t[u] >= 0 && t[u] < mlen && moff + t[u] < mask_bytes;
            const int x = has_mask ? mask[ok ? moff + t[u] : 0] : 0;
            m[u] = ok && (x == 1 || x == 2) ? x : 0;
        }
    };
    // pass 1 (reordered rows only): count remote and local entries, which fix
    // where the local and pad blocks start in the reordered row
    int64_t n2 = 0, n1 = 0;
    for (int64_t c = 0; reorder && c < n; c += 64 * SPLIT_GROUP) {
        int32_t t[SPLIT_GROUP];
        int m[SPLIT_GROUP];
        load_group(c, t, m);
#pragma unroll
        for (int u = 0; u < SPLIT_GROUP; ++u) {
            const bool in = c + u * 64 + lane < n;
            n2 += __popcll(__ballot(in && m[u] == 2));
            n1 += __popcll(__ballot(in && m[u] == 1));
        }
    }
    // pass 2: write the partitions
    int64_t c2 = 0, c1 = 0, c0 = 0;
    for (int64_t c = 0; c < n; c += 64 * SPLIT_GROUP) {
        int32_t tt[SPLIT_GROUP];
        int mm[SPLIT_GROUP];
        load_group(c, tt, mm);
#pragma unroll
        for (int u = 0; u < SPLIT_GROUP; ++u) {
            const int64_t i = c + u * 64 + lane;
            const int32_t t = tt[u];
            const int m = mm[u];
            const uint64_t b2 = __ballot(i < n && m == 2);
            const uint64_t b1 = __ballot(i < n && m == 1);
            const uint64_t b0 = __ballot(i < n && m == 0);
            if (i < n) {
                if (m == 2) {
                    const int64_t p = c2 + __popcll(b2 & lt);
                    remote[o + p] = t;
                    if (reorder) out_index[o + p] = t;
                } else if (m == 1) {
                    const int64_t p = c1 + __popcll(b1 & lt);
                    local[o + p] = t;
                    if (reorder) out_index[o + n2 + p] = t;
                } else if (reorder) {
                    out_index[o + n2 + n1 + c0 + __popcll(b0 & lt)] = t;
                }
            }
            c2 += __popcll(b2);
            c1 += __popcll(b1);
            c0 += __popcll(b0);
        }
    }
    // the running counts are the totals (equal to pass 1's when it ran)
    n1 = c1;
    n2 = c2;
    // unused tails of the compacted outputs
    for (int64_t i = n1 + lane; i < n; i += 64) local[o + i] = -1;
    for (int64_t i = n2 + lane; i < n; i += 64) remote[o + i] = -1;
    if (lane == 0) {
        n_local[r] = (int32_t)n1;
        n_remote[r] = (int32_t)n2;
        if (n_kept) n_kept[r] = (int32_t)(n1 + n2);
    }
}

}  // namespace sg

using namespace sg;

extern "C" int sg_split(void *stream, int rows, const int32_t *row_off, int64_t total,
                        const int32_t *kv_index, const int8_t *mask, int64_t mask_bytes,
                        const int64_t *mask_off, const int32_t *mask_len, int reorder, int32_t *out_index, int32_t *local,
                        int32_t *remote, int32_t *n_local, int32_t *n_remote, int32_t *n_kept) {
    SG_REQUIRE(rows >= 0 && total >= 0 && mask_bytes >= 0, SG_EINVAL, "sg_split: negative size");
    if (rows == 0) return SG_OK;
    SG_REQUIRE(row_off && n_local && n_remote && mask_off && mask_len, SG_EINVAL, "sg_split: null pointer");
    SG_REQUIRE(total == 0 || (kv_index && mask && local && remote), SG_EINVAL, "sg_split: null pointer");
    SG_REQUIRE(!reorder || total == 0 || out_index, SG_EINVAL, "sg_split: reorder needs out_index");
    const int blocks = (int)ceil_div(rows, SPLIT_WAVES);
    split_kernel<<<blocks, 64 * SPLIT_WAVES, 0, as_stream(stream)>>>(
        rows, row_off, total, kv_index, mask, mask_bytes, mask_off, mask_len, reorder ? 1 : 0, out_index, local, remote,
        n_local, n_remote, n_kept);
    return launch_status("sg_split");
}
