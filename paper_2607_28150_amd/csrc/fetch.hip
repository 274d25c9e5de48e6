// sg_fetch: indexed copy of K/V rows into paged destination slots.
// sg_fetch_keep: the same copy, where each fetched row is also kept at its own
// position in the decode side's KV store and its mask entry turns local, so
// later steps find it on the local lane (reuse of fetched entries).
//
// Used for the remote lane of on-demand transfer (source rows in pinned host
// memory read over the host link) and for the local lane and the placement of
// received rows into the decode-side page pool (device source).  A workgroup
// of 256 threads walks one row of the index: CPR lanes move one 16-byte vector
// each of a K/V row, so 256/CPR entries are in flight per step, UNROLL steps
// deep.  Eight steps (64 KB of a bf16 d = 128 row set per workgroup): scattered
// single-row reads over the host link wait on its latency, and at four steps
// the 16 host-source workgroups moved 47 GB/s where eight reach 55.  Pool
// pages are written with non-temporal stores (nothing reads them before the
// whole call has landed): the 64-request receive of 31.8 GB into randomly
// placed 16-row pages took 6.33 against 6.49 ms with plain stores.
#include "sg_internal.h"

namespace sg {

constexpr int FETCH_THREADS = 256;
constexpr int FETCH_UNROLL = 8;

struct KeepArgs {
    const int64_t *row_base;   // store row of token 0 of each index row
    v4u *k, *v;
    int64_t rows;
    int8_t *mask;              // NULL: no mask update
    int64_t mask_bytes;
    const int64_t *mask_off;
    const int32_t *mask_len;
};

template <int CPR, bool KEEP>
__device__ __forceinline__ void fetch_row(
    int r, const int32_t *__restrict__ row_off, int64_t total, const int32_t *__restrict__ index,
    const int32_t *__restrict__ n_valid, const int64_t *__restrict__ src_row_base, int64_t src_rows,
    const v4u *__restrict__ k_src, const v4u *__restrict__ v_src, const int32_t *__restrict__ page_table,
    int page_size, int max_pages, const int32_t *__restrict__ dst_start, v4u *__restrict__ k_pool,
    v4u *__restrict__ v_pool, int64_t pool_rows, const KeepArgs &keep) {
    constexpr int EPI = FETCH_THREADS / CPR;   // entries per step
    constexpr int EPB = EPI * FETCH_UNROLL;    // entries per block pass
    const int64_t o = row_off[r], e = row_off[r + 1];
    if (o < 0 || e < o || e > total) return;
    int64_t n = e - o;
    if (n_valid) n = min<int64_t>(n, max<int32_t>(n_valid[r], 0));
    const int64_t sbase = src_row_base[r];
    const bool to_pool = !KEEP || page_table != nullptr;
    const int64_t lbase = to_pool ? dst_start[r] : 0;
    const int32_t *pt = to_pool ? page_table + (int64_t)r * max_pages : nullptr;
    int64_t kbase = 0, moff = 0;
    int32_t mlen = 0;
    if (KEEP) {
        kbase = keep.row_base[r];
        if (keep.mask) {
            moff = keep.mask_off[r];
            mlen = keep.mask_len[r];
        }
    }
    const int lane = threadIdx.x % CPR;
    const int esub = threadIdx.x / CPR;

    if (src_rows <= 0) return;
    for (int64_t base = (int64_t)blockIdx.y * EPB; base < n; base += (int64_t)gridDim.y * EPB) {
        // all index loads of the pass, then all row loads (an entry that is not
        // copied reads source row 0), then the stores: every load is in flight
        // before the first use
        int64_t tok[FETCH_UNROLL];
#pragma unroll
        for (int j = 0; j < FETCH_UNROLL; ++j) {
            const int64_t i = min(base + esub + j * EPI, n - 1);
            tok[j] = index ? (int64_t)index[o + i] : i;
        }
        __builtin_amdgcn_sched_barrier(0);
        v4u kr[FETCH_UNROLL], vr[FETCH_UNROLL];
        int64_t dst[FETCH_UNROLL], kdst[FETCH_UNROLL], mpos[FETCH_UNROLL];
#pragma unroll
        for (int j = 0; j < FETCH_UNROLL; ++j) {
            const int64_t i = base + esub + j * EPI;
            const int64_t t = tok[j];
            const int64_t src = sbase + t;
            const bool live = i < n && src >= 0 && src < src_rows;
            dst[j] = -1;
            kdst[j] = -1;
            mpos[j] = -1;
            if (to_pool) {
                const int64_t lr = lbase + i;
                if (live && lr >= 0 && lr / page_size < max_pages) {
                    const int64_t pr = (int64_t)pt[lr / page_size] + lr % page_size;
                    if (pr >= 0 && pr < pool_rows) dst[j] = pr;
                }
            }
            if (KEEP) {
                const int64_t kr_row = kbase + t;
                if (live && kr_row >= 0 && kr_row < keep.rows) {
                    kdst[j] = kr_row;
                    if (keep.mask && lane == 0 && t >= 0 && t < mlen && moff + t >= 0 && moff + t < keep.mask_bytes)
                        mpos[j] = moff + t;
                }
            }
            const int64_t s_row = live ? src : 0;    // independent of the page-table loads
            kr[j] = __builtin_nontemporal_load(k_src + s_row * CPR + lane);
            vr[j] = __builtin_nontemporal_load(v_src + s_row * CPR + lane);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < FETCH_UNROLL; ++j) {
            if (dst[j] >= 0) {
                __builtin_nontemporal_store(kr[j], k_pool + dst[j] * CPR + lane);
                __builtin_nontemporal_store(vr[j], v_pool + dst[j] * CPR + lane);
            }
            if (KEEP) {
                if (kdst[j] >= 0) {
                    keep.k[kdst[j] * CPR + lane] = kr[j];
                    keep.v[kdst[j] * CPR + lane] = vr[j];
                }
                if (mpos[j] >= 0) keep.mask[mpos[j]] = 1;
            }
        }
    }
}

template <int CPR, bool KEEP>
__global__ __launch_bounds__(FETCH_THREADS) void fetch_kernel(
    int rows, const int32_t *__restrict__ row_off, int64_t total, const int32_t *__restrict__ index,
    const int32_t *__restrict__ n_valid, const int64_t *__restrict__ src_row_base, int64_t src_rows,
    const v4u *__restrict__ k_src, const v4u *__restrict__ v_src, const int32_t *__restrict__ page_table,
    int page_size, int max_pages, const int32_t *__restrict__ dst_start, v4u *__restrict__ k_pool,
    v4u *__restrict__ v_pool, int64_t pool_rows, KeepArgs keep) {
    for (int r = blockIdx.x; r < rows; r += gridDim.x)
        fetch_row<CPR, KEEP>(r, row_off, total, index, n_valid, src_row_base, src_rows, k_src, v_src, page_table,
                             page_size, max_pages, dst_start, k_pool, v_pool, pool_rows, keep);
}

template <bool KEEP>
int launch_fetch(const char *name, hipStream_t s, int cpr, int rows, const int32_t *row_off, int64_t total,
                 const int32_t *index, const int32_t *n_valid, const int64_t *src_row_base, int64_t src_rows,
                 const void *k_src, const void *v_src, const int32_t *page_table, int page_size, int max_pages,
                 const int32_t *dst_start, void *k_pool, void *v_pool, int64_t pool_rows, const KeepArgs &keep) {
    // four workgroups per row keep HBM busy; from a host source the rows are
    // shared out over HOST_LINK_WORKGROUPS workgroups.  Rows longer than one
    // pass are covered by the grid-stride loops.
    dim3 grid((unsigned)rows, 4);
    if (host_memory(k_src) || host_memory(v_src)) {
        grid.x = (unsigned)std::min(rows, HOST_LINK_WORKGROUPS);
        grid.y = (unsigned)std::max(1, HOST_LINK_WORKGROUPS / (int)grid.x);
    }
    auto ks = reinterpret_cast<const v4u *>(k_src);
    auto vs = reinterpret_cast<const v4u *>(v_src);
    auto kp = reinterpret_cast<v4u *>(k_pool);
    auto vp = reinterpret_cast<v4u *>(v_pool);
    switch (cpr) {
        case 8: fetch_kernel<8, KEEP><<<grid, FETCH_THREADS, 0, s>>>(rows, row_off, total, index, n_valid, src_row_base, src_rows, ks, vs, page_table, page_size, max_pages, dst_start, kp, vp, pool_rows, keep); break;
        case 16: fetch_kernel<16, KEEP><<<grid, FETCH_THREADS, 0, s>>>(rows, row_off, total, index, n_valid, src_row_base, src_rows, ks, vs, page_table, page_size, max_pages, dst_start, kp, vp, pool_rows, keep); break;
        case 32: fetch_kernel<32, KEEP><<<grid, FETCH_THREADS, 0, s>>>(rows, row_off, total, index, n_valid, src_row_base, src_rows, ks, vs, page_table, page_size, max_pages, dst_start, kp, vp, pool_rows, keep); break;
        default: set_error("%s: internal row size", name); return SG_EINTERNAL;
    }
    return launch_status(name);
}

}  // namespace sg

using namespace sg;

extern "C" int sg_fetch(void *stream, sg_dtype dt, int d, int rows, const int32_t *row_off, int64_t total,
                        const int32_t *index, const int32_t *n_valid, const int64_t *src_row_base,
                        int64_t src_rows, const void *k_src, const void *v_src, const int32_t *page_table,
                        int page_size, int max_pages, const int32_t *dst_start, void *k_pool, void *v_pool,
                        int64_t pool_rows) {
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "sg_fetch: unknown dtype %d", (int)dt);
    SG_REQUIRE(d == 64 || d == 128, SG_EUNSUPPORTED, "sg_fetch: head dimension %d not supported (64 or 128)", d);
    SG_REQUIRE(rows >= 0 && total >= 0 && src_rows >= 0 && pool_rows >= 0, SG_EINVAL, "sg_fetch: negative size");
    SG_REQUIRE(page_size >= 1 && max_pages >= 1, SG_EINVAL, "sg_fetch: page_size and max_pages must be >= 1");
    if (rows == 0 || total == 0) return SG_OK;
    SG_REQUIRE(row_off && src_row_base && k_src && v_src && page_table && dst_start && k_pool && v_pool,
               SG_EINVAL, "sg_fetch: null pointer");
    SG_REQUIRE(aligned16(k_src) && aligned16(v_src) && aligned16(k_pool) && aligned16(v_pool), SG_EINVAL,
               "sg_fetch: row arrays must be 16-byte aligned");
    return launch_fetch<false>("sg_fetch", as_stream(stream), d * esize_of(dt) / 16, rows, row_off, total, index,
                               n_valid, src_row_base, src_rows, k_src, v_src, page_table, page_size, max_pages,
                               dst_start, k_pool, v_pool, pool_rows, KeepArgs{});
}

extern "C" int sg_fetch_keep(void *stream, sg_dtype dt, int d, int rows, const int32_t *row_off, int64_t total,
                             const int32_t *index, const int32_t *n_valid, const int64_t *src_row_base,
                             int64_t src_rows, const void *k_src, const void *v_src, const int32_t *page_table,
                             int page_size, int max_pages, const int32_t *dst_start, void *k_pool, void *v_pool,
                             int64_t pool_rows, const int64_t *keep_row_base, void *k_keep, void *v_keep,
                             int64_t keep_rows, int8_t *mask, int64_t mask_bytes, const int64_t *mask_off,
                             const int32_t *mask_len) {
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "sg_fetch_keep: unknown dtype %d", (int)dt);
    SG_REQUIRE(d == 64 || d == 128, SG_EUNSUPPORTED, "sg_fetch_keep: head dimension %d not supported (64 or 128)",
               d);
    SG_REQUIRE(rows >= 0 && total >= 0 && src_rows >= 0 && keep_rows >= 0 && mask_bytes >= 0, SG_EINVAL,
               "sg_fetch_keep: negative size");
    if (page_table) {
        SG_REQUIRE(page_size >= 1 && max_pages >= 1 && pool_rows >= 0, SG_EINVAL,
                   "sg_fetch_keep: page_size and max_pages must be >= 1");
    }
    if (rows == 0 || total == 0) return SG_OK;
    SG_REQUIRE(row_off && index && src_row_base && k_src && v_src && keep_row_base && k_keep && v_keep, SG_EINVAL,
               "sg_fetch_keep: null pointer");
    SG_REQUIRE(!page_table || (dst_start && k_pool && v_pool), SG_EINVAL,
               "sg_fetch_keep: a page table needs dst_start and the pools");
    SG_REQUIRE(!mask || (mask_off && mask_len), SG_EINVAL, "sg_fetch_keep: a mask needs mask_off and mask_len");
    SG_REQUIRE(aligned16(k_src) && aligned16(v_src) && aligned16(k_keep) && aligned16(v_keep) &&
                   (!page_table || (aligned16(k_pool) && aligned16(v_pool))),
               SG_EINVAL, "sg_fetch_keep: row arrays must be 16-byte aligned");
    KeepArgs keep{keep_row_base, reinterpret_cast<v4u *>(k_keep), reinterpret_cast<v4u *>(v_keep), keep_rows,
                  mask, mask_bytes, mask_off, mask_len};
    return launch_fetch<true>("sg_fetch_keep", as_stream(stream), d * esize_of(dt) / 16, rows, row_off, total,
                              index, n_valid, src_row_base, src_rows, k_src, v_src, page_table,
                              page_table ? page_size : 1, page_table ? max_pages : 1, dst_start, k_pool, v_pool,
                              page_table ? pool_rows : 0, keep);
}
