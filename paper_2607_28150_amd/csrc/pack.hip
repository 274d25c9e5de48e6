// sg_pack: gather of the selected K/V rows into one transfer buffer.
//
// One workgroup covers ROWS rows of one (unit, request) segment; CPR lanes
// (16 bytes each) cover one row, so a wavefront moves 64/CPR whole rows per
// instruction and every global access is a fully used 16-byte vector.  The
// index, K and V loads of all rows a thread owns are issued before any result
// is used, so several vectors are in flight per lane; loads and stores are
// non-temporal (the source is read once, the transfer buffer is written once
// and read by a later phase or by the host link).
#include "sg_internal.h"

namespace sg {

constexpr int PACK_THREADS = 256;
constexpr int PACK_UNROLL = 2;

template <int CPR>
__global__ __launch_bounds__(PACK_THREADS) void pack_kernel(
    int B, int Hkv, const int32_t *__restrict__ cu_seqlens, int64_t T,
    const int32_t *__restrict__ cu_k, int64_t K_total, const v4u *__restrict__ k,
    const v4u *__restrict__ v, int64_t kv_layer_rows, const int32_t *__restrict__ idx,
    v4u *__restrict__ dk, v4u *__restrict__ dv, int32_t *__restrict__ didx, int nchunk) {
    constexpr int RPI = PACK_THREADS / CPR;          // rows per iteration of the block
    constexpr int ROWS = RPI * PACK_UNROLL;           // rows per block pass
    // one-dimensional grid, segment-major: consecutive workgroups take
    // consecutive chunks of one (unit, request) segment, so the rows in flight
    // at a time stay close together (measured faster than chunk-major order)
    const int y = (int)(blockIdx.x / (unsigned)nchunk);
    const int chunk = (int)(blockIdx.x % (unsigned)nchunk);
    const int b = y % B;
    const int u = y / B;                              // l * Hkv + h
    const int l = u / Hkv, h = u % Hkv;
    const int64_t c0 = cu_k[b], c1 = cu_k[b + 1];
    const int64_t s0 = cu_seqlens[b], s1 = cu_seqlens[b + 1];
    // device metadata is clamped to the host-checked sizes
    const int64_t kb = (c0 >= 0 && c1 >= c0 && c1 <= K_total) ? c1 - c0 : 0;
    const int64_t nb = (s0 >= 0 && s1 >= s0 && s1 <= T) ? s1 - s0 : 0;
    const int64_t slot0 = (int64_t)u * K_total + c0;
    const int64_t src0 = (int64_t)l * kv_layer_rows + (int64_t)h * T + s0;
    const int lane = threadIdx.x % CPR;
    const int rsub = threadIdx.x / CPR;

    if (nb == 0) {      // a request without tokens: every index is invalid, so zero rows
        for (int64_t base = (int64_t)chunk * ROWS; base < kb; base += (int64_t)nchunk * ROWS) {
#pragma unroll
            for (int j = 0; j < PACK_UNROLL; ++j) {
                const int64_t i = base + rsub + j * RPI;
                if (i < kb) {
                    const int64_t dst = (slot0 + i) * CPR + lane;
                    __builtin_nontemporal_store(v4u{0u, 0u, 0u, 0u}, dk + dst);
                    __builtin_nontemporal_store(v4u{0u, 0u, 0u, 0u}, dv + dst);
                }
            }
            if (threadIdx.x < ROWS) {
                const int64_t i = base + threadIdx.x;
                if (i < kb) didx[slot0 + i] = idx[slot0 + i];
            }
        }
        return;
    }
    // Every load of a pass is issued before any result is used: the indices
    // first (rows past the segment read its last index), then the K and V
    // rows (an invalid index reads row 0 of the request and is zeroed
    // afterwards).  Loads behind branches would make each wait for all the
    // loads before it.
    for (int64_t base = (int64_t)chunk * ROWS; base < kb; base += (int64_t)nchunk * ROWS) {
        int32_t t[PACK_UNROLL];
#pragma unroll
        for (int j = 0; j < PACK_UNROLL; ++j) t[j] = idx[slot0 + min<int64_t>(base + rsub + j * RPI, kb - 1)];
        __builtin_amdgcn_sched_barrier(0);      // every index load ahead of the row loads
        v4u kr[PACK_UNROLL], vr[PACK_UNROLL];
        bool ok[PACK_UNROLL];
#pragma unroll
        for (int j = 0; j < PACK_UNROLL; ++j) {
            ok[j] = t[j] >= 0 && t[j] < nb;
            const int64_t src = (src0 + (ok[j] ? t[j] : 0)) * CPR + lane;
            kr[j] = __builtin_nontemporal_load(k + src);
            vr[j] = __builtin_nontemporal_load(v + src);
        }
        __builtin_amdgcn_sched_barrier(0);      // every row load ahead of the stores
#pragma unroll
        for (int j = 0; j < PACK_UNROLL; ++j) {
            const int64_t i = base + rsub + j * RPI;
            if (i < kb) {
                const int64_t dst = (slot0 + i) * CPR + lane;
                __builtin_nontemporal_store(ok[j] ? kr[j] : v4u{0u, 0u, 0u, 0u}, dk + dst);
                __builtin_nontemporal_store(ok[j] ? vr[j] : v4u{0u, 0u, 0u, 0u}, dv + dst);
            }
        }
        // the index table from the values already loaded (one lane per row);
        // no second load, so nothing waits for the stores above to complete
#pragma unroll
        for (int j = 0; j < PACK_UNROLL; ++j) {
            const int64_t i = base + rsub + j * RPI;
            if (lane == 0 && i < kb) didx[slot0 + i] = t[j];
        }
    }
}

}  // namespace sg

using namespace sg;

extern "C" size_t sg_pack_bytes(sg_dtype dt, int L, int Hkv, int d, int64_t K_total) {
    if (L <= 0 || Hkv <= 0 || d <= 0 || K_total < 0) return 0;
    const size_t S = (size_t)L * Hkv * (size_t)K_total;
    return 2 * S * (size_t)d * esize_of(dt) + 4 * S;
}

extern "C" int sg_pack(void *stream, sg_dtype dt, int B, int L, int Hkv, int d,
                       const int32_t *cu_seqlens, int64_t T, const int32_t *cu_k, int64_t K_total,
                       int max_k, const void *k, const void *v, int64_t kv_layer_rows,
                       const int32_t *idx, void *dst, size_t dst_bytes) {
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "sg_pack: unknown dtype %d", (int)dt);
    SG_REQUIRE(B >= 1 && L >= 1 && Hkv >= 1, SG_EINVAL, "sg_pack: B, L, Hkv must be >= 1 (got %d, %d, %d)", B, L, Hkv);
    SG_REQUIRE(d == 64 || d == 128, SG_EUNSUPPORTED, "sg_pack: head dimension %d not supported (64 or 128)", d);
    SG_REQUIRE(T >= 0 && K_total >= 0 && max_k >= 0, SG_EINVAL, "sg_pack: negative size");
    SG_REQUIRE(kv_layer_rows >= 0, SG_EINVAL, "sg_pack: negative layer stride");
    const size_t need = sg_pack_bytes(dt, L, Hkv, d, K_total);
    SG_REQUIRE(dst_bytes >= need, SG_EWORKSPACE, "sg_pack: destination holds %zu bytes, needs %zu", dst_bytes, need);
    if (K_total == 0) return SG_OK;
    SG_REQUIRE(cu_seqlens && cu_k && k && v && idx && dst, SG_EINVAL, "sg_pack: null pointer");
    SG_REQUIRE(aligned16(k) && aligned16(v) && aligned16(dst), SG_EINVAL, "sg_pack: k, v and dst must be 16-byte aligned");
    const int rowb = d * esize_of(dt);
    const int cpr = rowb / 16;
    const int64_t S = (int64_t)L * Hkv * K_total;
    v4u *dk = reinterpret_cast<v4u *>(dst);
    v4u *dv = dk + S * cpr;
    int32_t *di = reinterpret_cast<int32_t *>(dv + S * cpr);
    const int rows_per_block = (PACK_THREADS / cpr) * PACK_UNROLL;
    const int64_t units = (int64_t)L * Hkv * B;
    // the kernel's chunks stride over every k_b, so a bound of 0 still covers them
    const int64_t nchunk = std::min<int64_t>(std::max<int64_t>(1, ceil_div(max_k, rows_per_block)), 65535);
    SG_REQUIRE(units * nchunk <= 0x7fffffff, SG_EINVAL, "sg_pack: too many units");
    const dim3 grid((unsigned)(units * nchunk));
    hipStream_t s = as_stream(stream);
    const v4u *kk = reinterpret_cast<const v4u *>(k);
    const v4u *vv = reinterpret_cast<const v4u *>(v);
    switch (cpr) {
        case 8: pack_kernel<8><<<grid, PACK_THREADS, 0, s>>>(B, Hkv, cu_seqlens, T, cu_k, K_total, kk, vv, kv_layer_rows, idx, dk, dv, di, (int)nchunk); break;
        case 16: pack_kernel<16><<<grid, PACK_THREADS, 0, s>>>(B, Hkv, cu_seqlens, T, cu_k, K_total, kk, vv, kv_layer_rows, idx, dk, dv, di, (int)nchunk); break;
        case 32: pack_kernel<32><<<grid, PACK_THREADS, 0, s>>>(B, Hkv, cu_seqlens, T, cu_k, K_total, kk, vv, kv_layer_rows, idx, dk, dv, di, (int)nchunk); break;
        default: set_error("sg_pack: internal row size %d", rowb); return SG_EINTERNAL;
    }
    return launch_status("sg_pack");
}
