// sg_fetch: indexed copy of K/V rows into paged destination slots.
//
// Used for the remote lane of on-demand transfer (source rows in pinned host
// memory read over the host link) and for placing received rows into the
// decode-side page pool (device source).  A workgroup of 256 threads walks one
// row of the index: CPR lanes move one 16-byte vector each of a K/V row, so
// 256/CPR entries are in flight per step, UNROLL steps deep.
#include "sg_internal.h"

namespace sg {

constexpr int FETCH_THREADS = 256;
constexpr int FETCH_UNROLL = 4;

template <int CPR>
__global__ __launch_bounds__(FETCH_THREADS) void fetch_kernel(
    int rows, const int32_t *__restrict__ row_off, int64_t total, const int32_t *__restrict__ index,
    const int32_t *__restrict__ n_valid, const int64_t *__restrict__ src_row_base, int64_t src_rows,
    const v4u *__restrict__ k_src, const v4u *__restrict__ v_src, const int32_t *__restrict__ page_table,
    int page_size, int max_pages, const int32_t *__restrict__ dst_start, v4u *__restrict__ k_pool,
    v4u *__restrict__ v_pool, int64_t pool_rows) {
    constexpr int EPI = FETCH_THREADS / CPR;   // entries per step
    constexpr int EPB = EPI * FETCH_UNROLL;    // entries per block pass
    const int r = blockIdx.x;
    const int64_t o = row_off[r], e = row_off[r + 1];
    if (o < 0 || e < o || e > total) return;
    int64_t n = e - o;
    if (n_valid) n = min<int64_t>(n, max<int32_t>(n_valid[r], 0));
    const int64_t sbase = src_row_base[r];
    const int64_t lbase = dst_start[r];
    const int32_t *pt = page_table + (int64_t)r * max_pages;
    const int lane = threadIdx.x % CPR;
    const int esub = threadIdx.x / CPR;

    for (int64_t base = (int64_t)blockIdx.y * EPB; base < n; base += (int64_t)gridDim.y * EPB) {
        v4u kr[FETCH_UNROLL], vr[FETCH_UNROLL];
        int64_t dst[FETCH_UNROLL];
#pragma unroll
        for (int j = 0; j < FETCH_UNROLL; ++j) {
            const int64_t i = base + esub + j * EPI;
            dst[j] = -1;
            if (i < n) {
                const int64_t src = sbase + (index ? (int64_t)index[o + i] : i);
                const int64_t lr = lbase + i;
                if (src >= 0 && src < src_rows && lr >= 0 && lr / page_size < max_pages) {
                    const int64_t pr = (int64_t)pt[lr / page_size] + lr % page_size;
                    if (pr >= 0 && pr < pool_rows) {
                        dst[j] = pr;
                        kr[j] = __builtin_nontemporal_load(k_src + src * CPR + lane);
                        vr[j] = __builtin_nontemporal_load(v_src + src * CPR + lane);
                    }
                }
            }
        }
#pragma unroll
        for (int j = 0; j < FETCH_UNROLL; ++j) {
            if (dst[j] >= 0) {
                k_pool[dst[j] * CPR + lane] = kr[j];
                v_pool[dst[j] * CPR + lane] = vr[j];
            }
        }
    }
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
    const int cpr = d * esize_of(dt) / 16;
    // enough blocks per row to keep the host link or HBM busy; rows longer than
    // one pass are covered by the grid-stride loop
    const int ysplit = 4;
    dim3 grid((unsigned)rows, ysplit);
    hipStream_t s = as_stream(stream);
    auto ks = reinterpret_cast<const v4u *>(k_src);
    auto vs = reinterpret_cast<const v4u *>(v_src);
    auto kp = reinterpret_cast<v4u *>(k_pool);
    auto vp = reinterpret_cast<v4u *>(v_pool);
    switch (cpr) {
        case 8: fetch_kernel<8><<<grid, FETCH_THREADS, 0, s>>>(rows, row_off, total, index, n_valid, src_row_base, src_rows, ks, vs, page_table, page_size, max_pages, dst_start, kp, vp, pool_rows); break;
        case 16: fetch_kernel<16><<<grid, FETCH_THREADS, 0, s>>>(rows, row_off, total, index, n_valid, src_row_base, src_rows, ks, vs, page_table, page_size, max_pages, dst_start, kp, vp, pool_rows); break;
        case 32: fetch_kernel<32><<<grid, FETCH_THREADS, 0, s>>>(rows, row_off, total, index, n_valid, src_row_base, src_rows, ks, vs, page_table, page_size, max_pages, dst_start, kp, vp, pool_rows); break;
        default: set_error("sg_fetch: internal row size"); return SG_EINTERNAL;
    }
    return launch_status("sg_fetch");
}
