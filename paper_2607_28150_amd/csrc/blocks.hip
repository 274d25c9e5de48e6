// Block-granular proactive selection (Section 4.1): block importance (eq. 1),
// the block budget (eq. 2) and the block pack; speculative transfer of the
// remaining blocks (Section 4.3).  The global top-K_r of the
// blocks is sg_topk over one row of L * M block importances per request.
//
// sg_block_importance: 8 lanes per block, one KV head each (more heads
//   loop), 32 blocks per workgroup; fp32 sums in a fixed order (eight token
//   partials per head, then the lanes by xor shuffles).  Layers 0 and 1 get
//   +inf, empty blocks -inf.
// sg_pack_blocks: a selected block moves Hkv * Nb contiguous source rows per
//   tensor; the grid is flat over 16-byte vectors of the output, each thread
//   issues the loads of all its vectors before any store (non-temporal), so
//   the copy runs like a plain strided memcpy.
// sg_spec_push (speculative transfer, Section 4.3): the same flat copy, with
//   each row stored at its own position in the decode side's store, its mask
//   entry turned local and the block marked in the remaining importances
//   (or, without a mask, the rows alone; sg_spec_commit then does the marking
//   on the consumer's stream once the rows have landed).
#include <math.h>

#include "sg_internal.h"

namespace sg {

constexpr int BLK_THREADS = 256;

// Importance: a workgroup covers BI_BLOCKS blocks of one (request, layer);
// the 8 lanes of a block take KV heads j, j + 8, ... and sum their tokens
// (every load of a head issued before its adds), then add up in a fixed
// order with xor shuffles.
constexpr int BI_LANES = 8;
constexpr int BI_BLOCKS = BLK_THREADS / BI_LANES;

__global__ __launch_bounds__(BLK_THREADS) void block_importance_kernel(int B, int L, int Hkv,
                                                                         const int32_t *__restrict__ cu_seqlens,
                                                                         int64_t T, int M, int nchunk,
                                                                         const float *__restrict__ scores,
                                                                         float *__restrict__ imp) {
    const int chunk = blockIdx.x % nchunk;
    const int bl = blockIdx.x / nchunk;
    const int b = bl % B, l = bl / B;
    const int64_t s0 = cu_seqlens[b], s1 = cu_seqlens[b + 1];
    // device metadata is clamped to the host-checked sizes
    const int64_t N = (s0 >= 0 && s1 >= s0 && s1 <= T) ? s1 - s0 : 0;
    const int64_t Nb = (N + M - 1) / M;
    const int j = threadIdx.x % BI_LANES;
    const int m = chunk * BI_BLOCKS + threadIdx.x / BI_LANES;
    const int64_t t0 = (int64_t)m * Nb, t1 = min(t0 + Nb, N);
    float sum = 0.f;
    if (l >= 2 && m < M) {
        for (int h = j; h < Hkv; h += BI_LANES) {
            const float *row = scores + ((int64_t)l * Hkv + h) * T + s0;
            float part[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
            int64_t t = t0;
            for (; t + 8 <= t1; t += 8) {
                float x[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) x[u] = row[t + u];
#pragma unroll
                for (int u = 0; u < 8; ++u) part[u] += x[u];
            }
            for (int u = 0; t < t1; ++t, ++u) part[u] += row[t];
            sum += ((part[0] + part[1]) + (part[2] + part[3])) + ((part[4] + part[5]) + (part[6] + part[7]));
        }
    }
#pragma unroll
    for (int off = 1; off < BI_LANES; off <<= 1) sum += __shfl_xor(sum, off, 64);
    if (j == 0 && m < M) {
        float *out = imp + ((int64_t)b * L + l) * M;
        out[m] = l < 2 ? INFINITY : (t1 <= t0 ? -INFINITY : sum / (float)((t1 - t0) * Hkv));
    }
}

constexpr int PB_UNROLL = 4;

// Output vector i of the K (or V) region: slot row r_all = i / CPR, vector
// c = i % CPR; slot row r_all = (s * Hkv + h) * Nb + r.
template <int CPR>
__global__ __launch_bounds__(BLK_THREADS) void pack_blocks_kernel(int L, int Hkv, int64_t T, int64_t s0, int64_t N,
                                                                    int M, int64_t Nb, const v4u *__restrict__ k,
                                                                    const v4u *__restrict__ v, int64_t kv_layer_rows,
                                                                    int nblk, const int32_t *__restrict__ ids,
                                                                    v4u *__restrict__ dk, v4u *__restrict__ dv,
                                                                    int32_t *__restrict__ did) {
    const int64_t total = (int64_t)nblk * Hkv * Nb * CPR;
    const int64_t stride = (int64_t)gridDim.x * BLK_THREADS * PB_UNROLL;
    for (int64_t base = (int64_t)blockIdx.x * BLK_THREADS * PB_UNROLL + threadIdx.x; base < total; base += stride) {
        v4u kr[PB_UNROLL], vr[PB_UNROLL];
        bool ok[PB_UNROLL];
        // every load of the pass first (a row past the prompt or of an invalid
        // id reads the request's first row and is zeroed)
#pragma unroll
        for (int u = 0; u < PB_UNROLL; ++u) {
            const int64_t i = min(base + (int64_t)u * BLK_THREADS, total - 1);
            const int64_t row = i / CPR, c = i % CPR;
            const int64_t r = row % Nb, sh = row / Nb;
            const int h = (int)(sh % Hkv), s = (int)(sh / Hkv);
            const int32_t id = ids[s];
            const bool valid = id >= 0 && (int64_t)id < (int64_t)L * M;
            const int l = valid ? id / M : 0, m = valid ? id % M : 0;
            const int64_t t = (int64_t)m * Nb + r;
            ok[u] = valid && t < N;
            const int64_t src = ((int64_t)l * kv_layer_rows + (int64_t)h * T + s0 + (ok[u] ? t : 0)) * CPR + c;
            kr[u] = __builtin_nontemporal_load(k + src);
            vr[u] = __builtin_nontemporal_load(v + src);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < PB_UNROLL; ++u) {
            const int64_t i = base + (int64_t)u * BLK_THREADS;
            if (i < total) {
                __builtin_nontemporal_store(ok[u] ? kr[u] : v4u{0u, 0u, 0u, 0u}, dk + i);
                __builtin_nontemporal_store(ok[u] ? vr[u] : v4u{0u, 0u, 0u, 0u}, dv + i);
            }
        }
    }
    for (int64_t s = (int64_t)blockIdx.x * BLK_THREADS + threadIdx.x; s < nblk; s += (int64_t)gridDim.x * BLK_THREADS)
        did[s] = ids[s];
}

// Speculative push: the grid is flat over 16-byte vectors of the pushed rows
// like the block pack, but every row goes back to its own position in the
// decode side's store; with MARK the lane holding vector 0 of a row turns its
// mask entry local, and the first lane of a block takes the block out of the
// remaining importances.
template <int CPR, bool MARK>
__global__ __launch_bounds__(BLK_THREADS) void spec_push_kernel(int L, int Hkv, int64_t T, int64_t s0, int64_t N,
                                                                  int M, int64_t Nb, const v4u *__restrict__ k,
                                                                  const v4u *__restrict__ v, int64_t src_layer_rows,
                                                                  v4u *__restrict__ kd, v4u *__restrict__ vd,
                                                                  int64_t dst_layer_rows, int nblk,
                                                                  const int32_t *__restrict__ ids,
                                                                  int8_t *__restrict__ mask, float *__restrict__ rem) {
    const int64_t total = (int64_t)nblk * Hkv * Nb * CPR;
    const int64_t stride = (int64_t)gridDim.x * BLK_THREADS * PB_UNROLL;
    for (int64_t base = (int64_t)blockIdx.x * BLK_THREADS * PB_UNROLL + threadIdx.x; base < total; base += stride) {
        v4u kr[PB_UNROLL], vr[PB_UNROLL];
        int64_t row_dst[PB_UNROLL], mpos[PB_UNROLL];
        int32_t lead[PB_UNROLL];
        // every load of the pass first (a row that is not pushed reads the
        // request's first row of layer 0 and is not stored)
#pragma unroll
        for (int u = 0; u < PB_UNROLL; ++u) {
            const int64_t iu = base + (int64_t)u * BLK_THREADS;
            const int64_t i = min(iu, total - 1);
            const int64_t row = i / CPR, c = i % CPR;
            const int64_t r = row % Nb, sh = row / Nb;
            const int h = (int)(sh % Hkv), s = (int)(sh / Hkv);
            const int32_t id = ids[s];
            const bool valid = iu < total && id >= 0 && (int64_t)id < (int64_t)L * M;
            const int l = valid ? id / M : 0, m = valid ? id % M : 0;
            const int64_t t = (int64_t)m * Nb + r;
            const bool ok = valid && t < N;
            const int64_t off = (int64_t)h * T + s0 + (ok ? t : 0);
            kr[u] = __builtin_nontemporal_load(k + ((int64_t)l * src_layer_rows + off) * CPR + c);
            vr[u] = __builtin_nontemporal_load(v + ((int64_t)l * src_layer_rows + off) * CPR + c);
            row_dst[u] = ok ? ((int64_t)l * dst_layer_rows + off) * CPR + c : -1;
            mpos[u] = ok && c == 0 ? ((int64_t)l * Hkv + h) * T + s0 + t : -1;
            lead[u] = valid && c == 0 && h == 0 && r == 0 ? id : -1;
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < PB_UNROLL; ++u) {
            if (row_dst[u] >= 0) {
                __builtin_nontemporal_store(kr[u], kd + row_dst[u]);
                __builtin_nontemporal_store(vr[u], vd + row_dst[u]);
            }
            if constexpr (MARK) {
                if (mpos[u] >= 0) mask[mpos[u]] = 1;
                if (rem && lead[u] >= 0) rem[lead[u]] = __builtin_nanf("");
            }
        }
    }
}

// Commit of delivered blocks: one thread per (block, KV head, block token)
// turns the mask entry local; the block's first thread takes it out of the
// remaining importances.
__global__ __launch_bounds__(BLK_THREADS) void spec_commit_kernel(int L, int Hkv, int64_t T, int64_t s0, int64_t N,
                                                                    int M, int64_t Nb, int nblk,
                                                                    const int32_t *__restrict__ ids,
                                                                    int8_t *__restrict__ mask,
                                                                    float *__restrict__ rem) {
    const int64_t total = (int64_t)nblk * Hkv * Nb;
    for (int64_t i = (int64_t)blockIdx.x * BLK_THREADS + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * BLK_THREADS) {
        const int64_t r = i % Nb, sh = i / Nb;
        const int h = (int)(sh % Hkv), s = (int)(sh / Hkv);
        const int32_t id = ids[s];
        if (id < 0 || (int64_t)id >= (int64_t)L * M) continue;
        const int l = id / M, m = id % M;
        const int64_t t = (int64_t)m * Nb + r;
        if (t < N) mask[((int64_t)l * Hkv + h) * T + s0 + t] = 1;
        if (rem && h == 0 && r == 0) rem[id] = __builtin_nanf("");
    }
}

}  // namespace sg

using namespace sg;

extern "C" int sg_block_importance(void *stream, int B, int L, int Hkv, const int32_t *cu_seqlens, int64_t T,
                                   int M, const float *scores, float *imp) {
    SG_REQUIRE(B >= 1 && L >= 1 && Hkv >= 1, SG_EINVAL, "sg_block_importance: B, L, Hkv must be >= 1");
    SG_REQUIRE(M >= 1 && T >= 0, SG_EINVAL, "sg_block_importance: need M >= 1 and T >= 0");
    SG_REQUIRE((int64_t)B * L <= 0x7fffffff, SG_EINVAL, "sg_block_importance: too many rows");
    SG_REQUIRE(cu_seqlens && scores && imp, SG_EINVAL, "sg_block_importance: null pointer");
    const int64_t nchunk = ceil_div(M, BI_BLOCKS);
    SG_REQUIRE((int64_t)B * L * nchunk <= 0x7fffffff, SG_EINVAL, "sg_block_importance: too many blocks");
    block_importance_kernel<<<(unsigned)(B * L * nchunk), BLK_THREADS, 0, as_stream(stream)>>>(
        B, L, Hkv, cu_seqlens, T, M, (int)nchunk, scores, imp);
    return launch_status("sg_block_importance");
}

extern "C" int64_t sg_block_budget(int M, int L, double Tp, double Tt) {
    if (M < 1 || L < 1 || !(Tp >= 0.0) || !(Tt >= 0.0)) return -1;
    const int64_t lm = (int64_t)L * M;
    int64_t k = lm;
    if (Tt > 0.0) {
        const double x = floor((double)M * (double)(L - 1) * (Tp / Tt));
        k = x >= (double)lm ? lm : (int64_t)x;
    }
    return std::min<int64_t>(lm, std::max<int64_t>(2 * (int64_t)M, k));
}

extern "C" size_t sg_pack_blocks_bytes(sg_dtype dt, int Hkv, int d, int64_t N, int M, int nblk) {
    if (Hkv <= 0 || d <= 0 || N < 0 || M <= 0 || nblk < 0) return 0;
    const size_t Nb = (size_t)((N + M - 1) / M);
    const size_t S = (size_t)nblk * Hkv * Nb;
    return 2 * S * (size_t)d * esize_of(dt) + 4 * (size_t)nblk;
}

extern "C" int sg_pack_blocks(void *stream, sg_dtype dt, int L, int Hkv, int d, int64_t T, int64_t s0, int64_t N,
                              int M, const void *k, const void *v, int64_t kv_layer_rows, int nblk,
                              const int32_t *ids, void *dst, size_t dst_bytes) {
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "sg_pack_blocks: unknown dtype %d", (int)dt);
    SG_REQUIRE(L >= 1 && Hkv >= 1 && M >= 1, SG_EINVAL, "sg_pack_blocks: L, Hkv, M must be >= 1");
    SG_REQUIRE(d == 64 || d == 128, SG_EUNSUPPORTED, "sg_pack_blocks: head dimension %d not supported", d);
    SG_REQUIRE(T >= 0 && s0 >= 0 && N >= 0 && s0 + N <= T && kv_layer_rows >= 0 && nblk >= 0, SG_EINVAL,
               "sg_pack_blocks: the request's tokens [s0, s0 + N) must lie in [0, T)");
    const size_t need = sg_pack_blocks_bytes(dt, Hkv, d, N, M, nblk);
    SG_REQUIRE(dst_bytes >= need, SG_EWORKSPACE, "sg_pack_blocks: destination holds %zu bytes, needs %zu",
               dst_bytes, need);
    if (nblk == 0) return SG_OK;
    SG_REQUIRE(k && v && ids && dst, SG_EINVAL, "sg_pack_blocks: null pointer");
    SG_REQUIRE(aligned16(k) && aligned16(v) && aligned16(dst), SG_EINVAL,
               "sg_pack_blocks: k, v and dst must be 16-byte aligned");
    SG_REQUIRE(N > 0, SG_EINVAL, "sg_pack_blocks: blocks of an empty request");
    const int cpr = d * esize_of(dt) / 16;
    const int64_t Nb = (N + M - 1) / M;
    const int64_t S = (int64_t)nblk * Hkv * Nb;
    v4u *dk = reinterpret_cast<v4u *>(dst);
    v4u *dv = dk + S * cpr;
    int32_t *di = reinterpret_cast<int32_t *>(dv + S * cpr);
    const int64_t total = S * cpr;
    const int64_t grid = std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, BLK_THREADS * PB_UNROLL), 65536));
    hipStream_t s = as_stream(stream);
    const v4u *kk = reinterpret_cast<const v4u *>(k);
    const v4u *vv = reinterpret_cast<const v4u *>(v);
    switch (cpr) {
        case 8: pack_blocks_kernel<8><<<(unsigned)grid, BLK_THREADS, 0, s>>>(L, Hkv, T, s0, N, M, Nb, kk, vv, kv_layer_rows, nblk, ids, dk, dv, di); break;
        case 16: pack_blocks_kernel<16><<<(unsigned)grid, BLK_THREADS, 0, s>>>(L, Hkv, T, s0, N, M, Nb, kk, vv, kv_layer_rows, nblk, ids, dk, dv, di); break;
        case 32: pack_blocks_kernel<32><<<(unsigned)grid, BLK_THREADS, 0, s>>>(L, Hkv, T, s0, N, M, Nb, kk, vv, kv_layer_rows, nblk, ids, dk, dv, di); break;
        default: set_error("sg_pack_blocks: internal row size"); return SG_EINTERNAL;
    }
    return launch_status("sg_pack_blocks");
}

extern "C" int64_t sg_spec_quota(int64_t blocks, int ratio_bp) {
    if (blocks < 0 || ratio_bp < 1) return -1;
    if (blocks == 0) return 0;
    if (blocks > (INT64_MAX - 9999) / ratio_bp) return -1;
    return std::min<int64_t>(blocks, std::max<int64_t>(1, (blocks * ratio_bp + 9999) / 10000));
}

extern "C" int sg_spec_push(void *stream, sg_dtype dt, int L, int Hkv, int d, int64_t T, int64_t s0, int64_t N,
                            int M, const void *k_src, const void *v_src, int64_t src_layer_rows, void *k_dst,
                            void *v_dst, int64_t dst_layer_rows, int nblk, const int32_t *ids, int8_t *mask,
                            float *rem) {
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "sg_spec_push: unknown dtype %d", (int)dt);
    SG_REQUIRE(L >= 1 && Hkv >= 1 && M >= 1, SG_EINVAL, "sg_spec_push: L, Hkv, M must be >= 1");
    SG_REQUIRE(d == 64 || d == 128, SG_EUNSUPPORTED, "sg_spec_push: head dimension %d not supported", d);
    SG_REQUIRE(T >= 0 && s0 >= 0 && N >= 0 && s0 + N <= T && nblk >= 0, SG_EINVAL,
               "sg_spec_push: the request's tokens [s0, s0 + N) must lie in [0, T)");
    SG_REQUIRE(src_layer_rows >= 0 && dst_layer_rows >= 0, SG_EINVAL, "sg_spec_push: negative layer stride");
    if (nblk == 0) return SG_OK;
    SG_REQUIRE(k_src && v_src && k_dst && v_dst && ids, SG_EINVAL, "sg_spec_push: null pointer");
    SG_REQUIRE(aligned16(k_src) && aligned16(v_src) && aligned16(k_dst) && aligned16(v_dst), SG_EINVAL,
               "sg_spec_push: row arrays must be 16-byte aligned");
    SG_REQUIRE(N > 0, SG_EINVAL, "sg_spec_push: blocks of an empty request");
    const int cpr = d * esize_of(dt) / 16;
    const int64_t Nb = (N + M - 1) / M;
    const int64_t total = (int64_t)nblk * Hkv * Nb * cpr;
    const int64_t cap = host_memory(k_src) || host_memory(v_src) ? HOST_LINK_WORKGROUPS : 65536;
    const int64_t grid = std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, BLK_THREADS * PB_UNROLL), cap));
    hipStream_t s = as_stream(stream);
    auto ks = reinterpret_cast<const v4u *>(k_src);
    auto vs = reinterpret_cast<const v4u *>(v_src);
    auto kd = reinterpret_cast<v4u *>(k_dst);
    auto vd = reinterpret_cast<v4u *>(v_dst);
    switch (cpr) {
        case 8:
            if (mask) spec_push_kernel<8, true><<<(unsigned)grid, BLK_THREADS, 0, s>>>(L, Hkv, T, s0, N, M, Nb, ks, vs, src_layer_rows, kd, vd, dst_layer_rows, nblk, ids, mask, rem);
            else spec_push_kernel<8, false><<<(unsigned)grid, BLK_THREADS, 0, s>>>(L, Hkv, T, s0, N, M, Nb, ks, vs, src_layer_rows, kd, vd, dst_layer_rows, nblk, ids, nullptr, nullptr);
            break;
        case 16:
            if (mask) spec_push_kernel<16, true><<<(unsigned)grid, BLK_THREADS, 0, s>>>(L, Hkv, T, s0, N, M, Nb, ks, vs, src_layer_rows, kd, vd, dst_layer_rows, nblk, ids, mask, rem);
            else spec_push_kernel<16, false><<<(unsigned)grid, BLK_THREADS, 0, s>>>(L, Hkv, T, s0, N, M, Nb, ks, vs, src_layer_rows, kd, vd, dst_layer_rows, nblk, ids, nullptr, nullptr);
            break;
        case 32:
            if (mask) spec_push_kernel<32, true><<<(unsigned)grid, BLK_THREADS, 0, s>>>(L, Hkv, T, s0, N, M, Nb, ks, vs, src_layer_rows, kd, vd, dst_layer_rows, nblk, ids, mask, rem);
            else spec_push_kernel<32, false><<<(unsigned)grid, BLK_THREADS, 0, s>>>(L, Hkv, T, s0, N, M, Nb, ks, vs, src_layer_rows, kd, vd, dst_layer_rows, nblk, ids, nullptr, nullptr);
            break;
        default: set_error("sg_spec_push: internal row size"); return SG_EINTERNAL;
    }
    return launch_status("sg_spec_push");
}

extern "C" int sg_spec_commit(void *stream, int L, int Hkv, int64_t T, int64_t s0, int64_t N, int M, int nblk,
                              const int32_t *ids, int8_t *mask, float *rem) {
    SG_REQUIRE(L >= 1 && Hkv >= 1 && M >= 1, SG_EINVAL, "sg_spec_commit: L, Hkv, M must be >= 1");
    SG_REQUIRE(T >= 0 && s0 >= 0 && N >= 0 && s0 + N <= T && nblk >= 0, SG_EINVAL,
               "sg_spec_commit: the request's tokens [s0, s0 + N) must lie in [0, T)");
    if (nblk == 0) return SG_OK;
    SG_REQUIRE(ids && mask, SG_EINVAL, "sg_spec_commit: null pointer");
    SG_REQUIRE(N > 0, SG_EINVAL, "sg_spec_commit: blocks of an empty request");
    const int64_t Nb = (N + M - 1) / M;
    const int64_t total = (int64_t)nblk * Hkv * Nb;
    const int64_t grid = std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, BLK_THREADS), 65536));
    spec_commit_kernel<<<(unsigned)grid, BLK_THREADS, 0, as_stream(stream)>>>(L, Hkv, T, s0, N, M, Nb, nblk, ids, mask,
                                                                               rem);
    return launch_status("sg_spec_commit");
}
