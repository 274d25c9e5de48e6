// sg_decode_attn: GQA decode attention over a partial, page-addressed KV set.
//
// Grid: x = (sequence, KV head) unit, y = split of the unit's rows (one split
// whenever the units fill the chip), z = group of up to 8 q heads of the KV
// head.  Between one and four units per CU the grid is instead one-dimensional
// over (shader engine, slot): every unit is cut into two equal parts for the
// two engines of one engine pair of its XCD, the units are dealt to the pairs
// in snake order of length, and each engine takes its units longest first
// (the equal-parts mode in the kernel).  A workgroup serves all the q heads of its
// group, so each K/V row is read from HBM once per step (twice for 16-head
// groups).
//
// Memory side.  The split's page entries are staged in LDS once (one round
// trip, overlapped with the query loads); every wavefront owns one contiguous
// range of rows and streams it through a private LDS ring with direct
// global->LDS loads (non-temporal), NS - 1 steps ahead of its arithmetic,
// without holding registers for the data in flight and without workgroup
// barriers.
//
// Arithmetic side.  LPR lanes cover one row, each with E = d / LPR elements
// (LPR = 4 for up to 2 heads at d = 128, 8 for 4 heads, 16 for 8 heads, so
// the output accumulators fit in registers); a wavefront step covers 64 / LPR
// rows.
//   logits : each lane dots its slices of q (held in registers) with its K
//            slices (v_dot2_f32_bf16 for bf16, fp32 accumulation); DPP adds
//            sum the partials over the row's LPR lanes.  With 8 heads over
//            16-lane rows the sums are transposed instead (each level of
//            lane pairs halves the values a lane holds), so a lane ends with
//            one head's logit and takes one exponential, and row broadcasts
//            hand the probabilities to the row;
//   softmax: online, against a wavefront-uniform reference max per head that
//            is raised only when a logit passes it by more than 2^16 (exp2,
//            log2(e) folded into the scale), so the outputs are rescaled
//            only on those rare steps;
//   values : each lane accumulates its V slices weighted by the row's
//            probability for every head in fp32.
// At the end each wavefront sums its row groups with DPP adds and its four
// DPP rows with lane swaps (permlane32 / permlane16, in transposed form, so
// every swap and add halves the registers to reduce), then as soon as its own
// rows are done stores its state in LDS; the wavefronts' states are merged
// with (max, sum, output) rescaling.  With one split the normalised output is written
// directly; otherwise the split's state goes to the workspace and a merge
// kernel combines the splits in a fixed order.  All reductions have a fixed
// order, so results are deterministic.
#include <mutex>

#include "sg_internal.h"

namespace sg {

template <typename T>
struct Elem;
template <>
struct Elem<float> {
    static constexpr int PER16 = 4;
    __device__ static void unpack(const v4u &w, float *x) {
        x[0] = __uint_as_float(w.x); x[1] = __uint_as_float(w.y);
        x[2] = __uint_as_float(w.z); x[3] = __uint_as_float(w.w);
    }
};
template <>
struct Elem<uint16_t> {  // bfloat16 bits
    static constexpr int PER16 = 8;
    __device__ static void unpack(const v4u &w, float *x) {
        x[0] = bf16_lo(w.x); x[1] = bf16_hi(w.x); x[2] = bf16_lo(w.y); x[3] = bf16_hi(w.y);
        x[4] = bf16_lo(w.z); x[5] = bf16_hi(w.z); x[6] = bf16_lo(w.w); x[7] = bf16_hi(w.w);
    }
};

// Work shape for HG heads per workgroup.
//   LPR  lanes per row: at least 4, and enough that the HG * E output
//        accumulators stay within 64 registers and the query slices within
//        32;
//   VPL  16-byte vectors per lane per row; a step moves VPL KB of K and of V;
//   ring four wavefronts (one per SIMD), each with NS slots, so that about
//        12 KB per wavefront (48 KB per workgroup) are in flight.  Measured on
//        MI355X: deeper rings or more wavefronts per CU lower the bandwidth
//        these gathers reach (more outstanding requests per CU than the
//        memory system serves well), shallower ones leave it idle.
template <typename T, int D, int HG>
struct DecodeShape {
    static constexpr int ESZ = (int)sizeof(T);
    static constexpr int LPR_A = HG * D / 64, LPR_B = HG * D * ESZ / 128;
    static constexpr int LPR_C = LPR_A > LPR_B ? LPR_A : LPR_B;
    static constexpr int LPR = LPR_C < 4 ? 4 : (LPR_C > 16 ? 16 : LPR_C);
    static constexpr int E = D / LPR;
    static constexpr int VPL = D * ESZ / 16 / LPR;
    static constexpr int RPS = 64 / LPR;
    static constexpr int STEPB = VPL * 1024;
    static constexpr int SLOTB = 2 * STEPB;
    static constexpr int WAVES = 4;
    static constexpr int NS_A = 1 + (12 * 1024 + SLOTB - 1) / SLOTB;
    static constexpr int NS = NS_A < 2 ? 2 : (NS_A > 8 ? 8 : NS_A);
    static_assert(LPR <= 16 && VPL >= 1, "decode work shape");
};
constexpr int DEC_MAX_HG = 8;       // heads served by one workgroup; larger groups use several
constexpr int DEC_PT_CAP = 2048;    // page entries of one split staged in LDS
constexpr int DEC_MIN_SPLIT_ROWS = 128;
constexpr int64_t DEC_CAP_ROWS = 1024;    // split length when units number one to four per CU
// The workgroup dispatcher of MI355X sends consecutive workgroup ids round
// robin over its 8 XCDs, and the ids an XCD receives round robin over its 4
// shader engines (measured: workgroup L runs on XCD L mod 8 and on engine
// (L / 8) mod 4 of that XCD's rotation), each engine then filling its own
// CUs.  Work handed to one engine never moves to another.
constexpr int DEC_XCDS = 8;
constexpr int DEC_ENGINES = 4;
constexpr int DEC_BIN_MAX = 128;          // units of one XCD in the equal-parts mode
constexpr int DEC_PARTS = 2;              // parts per unit; units go to DEC_ENGINES / DEC_PARTS engine groups
constexpr float DEC_LAZY = 16.f;    // log2 headroom before the reference max is raised

// partial state of one split: per head (m, l) then o[d]
__device__ __forceinline__ float *part_ptr(float *ws, int64_t unit, int nsplit, int split, int G, int d) {
    return ws + ((unit * nsplit + split) * G) * (int64_t)(d + 2);
}

// DPP lane moves (gfx9 encodings): quad_perm, row rotate, row half-mirror
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int DPP_XOR1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int DPP_XOR2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141;
constexpr int DPP_ROR4 = 0x124;
constexpr int DPP_ROR8 = 0x128;
constexpr int DPP_MIRROR = 0x140;     // row_mirror: lane i <-> 15 - i within each 16-lane row
constexpr int DPP_NEWBCAST = 0x150;   // row_newbcast:n = DPP_NEWBCAST + n: lane n of each row to the row

// sum over each group of N consecutive lanes (N = 4, 8 or 16); every lane of
// the group receives the group's sum
template <int N>
__device__ __forceinline__ float group_sum(float x) {
    x += dpp<DPP_XOR1>(x);
    x += dpp<DPP_XOR2>(x);
    if constexpr (N == 8) {
        x += dpp<DPP_HALF_MIRROR>(x);
    } else if constexpr (N == 16) {
        x += dpp<DPP_ROR4>(x);
        x += dpp<DPP_ROR8>(x);
    }
    return x;
}

// sum over the 16 / N lanes of a 16-lane DPP row that sit N apart (lanes
// holding the same slice of different rows); every such lane receives it
template <int N>
__device__ __forceinline__ float row_groups_sum(float x) {
    if constexpr (N <= 4) x += dpp<DPP_ROR4>(x);
    if constexpr (N <= 8) x += dpp<DPP_ROR8>(x);
    return x;
}

// Grid: x = (sequence, KV head) unit, y = split of the unit's rows, z = group
// of HG q heads within the KV head's G.  See the top of the file.
template <typename T, int D, int HG>
__global__ __launch_bounds__((64 * DecodeShape<T, D, HG>::WAVES)) void decode_kernel(
    int Hq, int Hkv, float scale_log2, const T *__restrict__ q, const v4u *__restrict__ k_pool,
    const v4u *__restrict__ v_pool, int64_t pool_rows, const int32_t *__restrict__ page_table,
    const int32_t *__restrict__ n_rows, int page_size, uint32_t page_mul, int page_shift, int max_pages,
    int64_t split_rows, float *__restrict__ out, float *__restrict__ ws, int nunits, int parts) {
    using S = DecodeShape<T, D, HG>;
    constexpr int PER16 = Elem<T>::PER16;  // elements per 16-byte vector
    constexpr int LPR = S::LPR, VPL = S::VPL, RPS = S::RPS, WAVES = S::WAVES, NS = S::NS;
    constexpr int STEPB = S::STEPB, SLOTB = S::SLOTB;
    constexpr int CPR = D / PER16;         // 16-byte vectors per row
    constexpr int NPART = WAVES * 4;       // partial states: the 4 DPP rows of every wavefront
    constexpr int RINGB = WAVES * NS * SLOTB;
    static_assert((NS - 1) * 2 * VPL <= 63, "loads in flight per wavefront");
    __shared__ __attribute__((aligned(16))) char ring[RINGB];
    // a wavefront's partial outputs [HG][D] go to its own ring once its loads have drained
    static_assert(NS * SLOTB >= HG * D * 4, "partial state fits a wavefront's ring");
    __shared__ int32_t pte[DEC_PT_CAP];
    __shared__ float m_s[WAVES][HG], l_s[NPART][HG];

    const int tid = threadIdx.x, lane = tid % 64;
    const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
    const int64_t max_rows = (int64_t)max_pages * page_size;

    // Which rows this workgroup reads: [r0, rend) of unit `unit`.
    //   split mode: unit blockIdx.x, fixed split blockIdx.y of split_rows rows;
    //   equal-parts mode (parts > 0, a one-dimensional grid): workgroup L
    //     belongs to engine k = (L / 8) mod 4 of XCD x = L mod 8, whose units
    //     are x, x + 8, ...  Those units, ranked by length, are dealt to the
    //     XCD's engine groups (4 / parts engines each) in snake order (ranks
    //     0, 3, 4, 7, ... to the first of two groups, 1, 2, 5, 6, ... to the
    //     second), so the groups carry nearly equal rows; each unit is cut
    //     into `parts` equal parts, one per engine of its group, and slot
    //     L / 32 of an engine takes its group's units longest first.
    int64_t unit, n, r0, rend;
    int split, nsplit;
    if (parts > 0) {
        static_assert(DEC_BIN_MAX == 128 && WAVES == 4, "the rank below splits 128 members over 4 quarters");
        __shared__ __attribute__((aligned(16))) int32_t bin_n[DEC_BIN_MAX];
        __shared__ int32_t chosen;
        const int L = (int)blockIdx.x;
        const int bx = L % DEC_XCDS, bk = (L / DEC_XCDS) % DEC_ENGINES, bj = L / (DEC_XCDS * DEC_ENGINES);
        const int members = (nunits - bx + DEC_XCDS - 1) / DEC_XCDS;
        // engine group of bk and the rank (by length) of the unit its bj-th
        // workgroup takes: ranks are dealt to the groups in snake order
        constexpr int NGRP = DEC_ENGINES / DEC_PARTS;
        const int grp = bk / parts, part = bk % parts;
        const int target = 2 * NGRP * (bj / 2) + ((bj & 1) ? 2 * NGRP - 1 - grp : grp);
        if (target >= members) return;      // uniform: the bins' last slots past the units
        if (tid < DEC_BIN_MAX)
            bin_n[tid] = tid < members
                             ? (int32_t)max<int64_t>(0, min<int64_t>(n_rows[bx + (int64_t)DEC_XCDS * tid], max_rows))
                             : -1;
        __syncthreads();
        // rank of member m = the members longer than it, or as long and listed
        // earlier.  Four adjacent threads count for one member, each over a
        // quarter of the list (32 entries, eight 16-byte LDS reads), and quad
        // DPP adds join the counts; 64 members per pass.
        for (int mbase = 0; mbase < members; mbase += 64) {
            const int m = mbase + tid / 4, qtr = tid % 4;
            const int32_t v = m < members ? bin_n[m] : -1;
            const int4 *row = reinterpret_cast<const int4 *>(bin_n + qtr * 32);
            int cnt = 0;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int4 w = row[i];
                const int t = qtr * 32 + 4 * i;
                cnt += (w.x > v) || (w.x == v && t < m);
                cnt += (w.y > v) || (w.y == v && t + 1 < m);
                cnt += (w.z > v) || (w.z == v && t + 2 < m);
                cnt += (w.w > v) || (w.w == v && t + 3 < m);
            }
            cnt += __builtin_amdgcn_update_dpp(0, cnt, DPP_XOR1, 0xf, 0xf, false);
            cnt += __builtin_amdgcn_update_dpp(0, cnt, DPP_XOR2, 0xf, 0xf, false);
            if (qtr == 0 && m < members && cnt == target) chosen = m;
        }
        __syncthreads();
        const int sel = min(max((int)chosen, 0), members - 1);   // the ranks are a permutation: one match
        unit = bx + (int64_t)DEC_XCDS * sel;
        n = bin_n[sel];
        split = part;
        nsplit = parts;
        r0 = n * part / parts;
        rend = n * (part + 1) / parts;
    } else {
        unit = blockIdx.x;
        split = blockIdx.y;
        nsplit = gridDim.y;
        r0 = (int64_t)split * split_rows;
        rend = r0 + split_rows;
        n = -1;                           // loaded below, beside the query and the page entries
    }
    const int b = (int)(unit / Hkv), h = (int)(unit % Hkv);
    const int G = Hq / Hkv;
    const int gq0 = h * G + (int)blockIdx.z * HG;      // first q head served
    const int c = lane % LPR, r = lane / LPR;       // slice within the row, row within the step

    // this lane's slices of the HG query vectors: vectors j * LPR + c, j < VPL
    v4u qs[HG][VPL];
    {
        const v4u *qv = reinterpret_cast<const v4u *>(q + ((int64_t)b * Hq + gq0) * D);
#pragma unroll
        for (int g = 0; g < HG; ++g)
#pragma unroll
            for (int j = 0; j < VPL; ++j) qs[g][j] = qv[g * CPR + j * LPR + c];
    }
    // page entries covering the rows [r0, rend)
    const int64_t pg0 = r0 / page_size;
    const int64_t pg1 = min<int64_t>(max_pages, ceil_div(min<int64_t>(max_rows, rend), page_size));
    const int npg = (int)min<int64_t>(DEC_PT_CAP, max<int64_t>(0, pg1 - pg0));   // the host keeps it within the cap
    const int32_t *pt = page_table + unit * max_pages + pg0;
    for (int i = tid; i < npg; i += 64 * WAVES) pte[i] = pt[i];

    if (parts == 0) n = max<int64_t>(0, min<int64_t>((int64_t)n_rows[unit], max_rows));
    // rows whose pages lie past the staged entries are not reached (the host
    // sizes splits so that this never cuts anything)
    const int64_t r1 = min<int64_t>(min<int64_t>(n, rend), (pg0 + npg) * (int64_t)page_size);
    const int64_t len = pool_rows > 0 ? max<int64_t>(0, r1 - r0) : 0;     // an empty pool: every row is skipped
    const int64_t per = ceil_div(ceil_div(len, WAVES), RPS) * RPS;
    const int64_t w0 = r0 + (int64_t)wave * per;
    const int64_t w1 = min<int64_t>(r0 + len, w0 + per);
    // the query slices are used first inside the loop; waiting for them here
    // keeps the compiler from placing that wait inside the loop, where it
    // would also drain the ring's loads (it does not see them)
#pragma unroll
    for (int g = 0; g < HG; ++g)
#pragma unroll
        for (int j = 0; j < VPL; ++j) asm volatile("" ::"v"(qs[g][j]));
    // a split that starts past the unit's rows writes no state (the merge
    // reads the row count and skips it): it ends after one round trip instead
    // of holding a workgroup slot through the barriers and the state stores.
    // Every part of a unit with rows starts below its row count.
    if (nsplit > 1 && r0 >= n) return;
    __syncthreads();    // page entries staged

    // m: reference max per head, wavefront-uniform; l and o: this lane's
    // partials over the rows of its row group
    float m[HG], l[HG], o[HG][VPL][PER16];
    // Transposed logits (8 heads over 16-lane rows): after the reduction lane
    // i of a row holds the logit of head hd = (i >> 3 & 1) + 2 (i >> 2 & 1) +
    // 4 (i >> 1 & 1) (lanes i and i ^ 1 alike), so each lane takes one
    // exponential instead of eight; the probabilities then go to the whole
    // row by row broadcasts.  m_lane and l_lane are the reference and sum of
    // the lane's head.
    constexpr bool TRANS = HG == 8 && LPR == 16;
    const int hd = ((lane >> 3) & 1) | (((lane >> 2) & 1) << 1) | (((lane >> 1) & 1) << 2);
    float m_lane = -INFINITY, l_lane = 0.f, z_lane = -INFINITY;
#pragma unroll
    for (int g = 0; g < HG; ++g) {
        m[g] = -INFINITY;
        l[g] = 0.f;
#pragma unroll
        for (int j = 0; j < VPL; ++j)
#pragma unroll
            for (int e = 0; e < PER16; ++e) o[g][j][e] = 0.f;
    }

    // pool row of logical row lr, or -1 (past the range or outside the pool).
    // rel < npg * page_size <= max_rows <= 2^30, and rel / page_size is the
    // exact multiply-shift (rel * page_mul) >> page_shift set up by the host
    auto pool_row = [&](int64_t lr) -> int {
        const uint32_t rel = (uint32_t)(min<int64_t>(lr, w1 - 1) - pg0 * page_size);
        const uint32_t pi = (uint32_t)(((uint64_t)rel * page_mul) >> page_shift);
        const int64_t x = (int64_t)pte[pi] + (int)(rel - pi * (uint32_t)page_size);
        return (lr < w1 && x >= 0 && x < pool_rows) ? (int)x : -1;
    };
    char *myring = ring + wave * (NS * SLOTB);
    // the loads of the step at row t into ring slot `slot`: vector j * LPR + c
    // of the lane's row lands at slot + j KB + 16 lane.  A row left out reads
    // pool row 0 (in bounds: the pool is not empty when a wavefront has rows;
    // the repeated address stays in L2) and its bit in `valid` clears.
    auto issue = [&](int64_t t, int slot, unsigned &valid) {
        char *sb = myring + slot * SLOTB;
        const int pr = pool_row(t + r);
        const int64_t off = (int64_t)max(pr, 0) * CPR + c;
#pragma unroll
        for (int j = 0; j < VPL; ++j) {
            dma16_nt(k_pool + off + j * LPR, lds_addr(sb + j * 1024));
            dma16_nt(v_pool + off + j * LPR, lds_addr(sb + STEPB + j * 1024));
        }
        valid = (valid & ~(1u << slot)) | ((pr >= 0 ? 1u : 0u) << slot);
    };
    // logits of the lane's row for every head (log2 units; -inf for a row
    // left out), and whether any passes its reference max by more than
    // DEC_LAZY anywhere in the wavefront
    auto logits = [&](const char *sb, bool ok, float (&z)[HG]) -> bool {
        v4u kv[VPL];
#pragma unroll
        for (int j = 0; j < VPL; ++j) kv[j] = *reinterpret_cast<const v4u *>(sb + j * 1024 + lane * 16);
        bool grow = false;
        if constexpr (TRANS) {
            float a[HG];
#pragma unroll
            for (int g = 0; g < HG; ++g) {
                a[g] = 0.f;
#pragma unroll
                for (int j = 0; j < VPL; ++j) a[g] = SliceDot<T>::run(qs[g][j], kv[j], a[g]);
            }
            // each level pairs lanes that differ in one more lane bit (3, 2, 1);
            // a lane keeps the member of each value pair its bit selects and
            // adds the partner's copy of it
            const bool b3 = (lane >> 3) & 1, b2 = (lane >> 2) & 1, b1 = (lane >> 1) & 1;
            float w[4], x[2];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                w[i] = (b3 ? a[2 * i + 1] : a[2 * i]) + dpp<DPP_MIRROR>(b3 ? a[2 * i] : a[2 * i + 1]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
                x[i] = (b2 ? w[2 * i + 1] : w[2 * i]) + dpp<DPP_HALF_MIRROR>(b2 ? w[2 * i] : w[2 * i + 1]);
            float y = (b1 ? x[1] : x[0]) + dpp<DPP_XOR2>(b1 ? x[0] : x[1]);
            y += dpp<DPP_XOR1>(y);
            z_lane = ok ? y * scale_log2 : -INFINITY;
            grow = z_lane > m_lane + DEC_LAZY;
            return __any(grow);
        }
#pragma unroll
        for (int g = 0; g < HG; ++g) {
            float a = 0.f;
#pragma unroll
            for (int j = 0; j < VPL; ++j) a = SliceDot<T>::run(qs[g][j], kv[j], a);
            a = group_sum<LPR>(a);
            z[g] = ok ? a * scale_log2 : -INFINITY;
            grow |= z[g] > m[g] + DEC_LAZY;
        }
        return __any(grow);
    };
    // p = 2^(z - m) into l and, weighted over the lane's V slices, into o
    auto accumulate = [&](const char *sb, const float (&z)[HG]) {
        v4u vv[VPL];
#pragma unroll
        for (int j = 0; j < VPL; ++j) vv[j] = *reinterpret_cast<const v4u *>(sb + STEPB + j * 1024 + lane * 16);
        float p[HG];
        if constexpr (TRANS) {
            const float ref = m_lane == -INFINITY ? 0.f : m_lane;
            const float pl = __builtin_amdgcn_exp2f(z_lane - ref);
            l_lane += pl;
            p[0] = dpp<DPP_NEWBCAST + 0>(pl);
            p[1] = dpp<DPP_NEWBCAST + 8>(pl);
            p[2] = dpp<DPP_NEWBCAST + 4>(pl);
            p[3] = dpp<DPP_NEWBCAST + 12>(pl);
            p[4] = dpp<DPP_NEWBCAST + 2>(pl);
            p[5] = dpp<DPP_NEWBCAST + 10>(pl);
            p[6] = dpp<DPP_NEWBCAST + 6>(pl);
            p[7] = dpp<DPP_NEWBCAST + 14>(pl);
        } else {
#pragma unroll
            for (int g = 0; g < HG; ++g) {
                const float ref = m[g] == -INFINITY ? 0.f : m[g];     // nothing seen yet: z is -inf too
                p[g] = __builtin_amdgcn_exp2f(z[g] - ref);
                l[g] += p[g];
            }
        }
#pragma unroll
        for (int j = 0; j < VPL; ++j) {
            float x[PER16];
            Elem<T>::unpack(vv[j], x);
#pragma unroll
            for (int g = 0; g < HG; ++g)
#pragma unroll
                for (int e = 0; e < PER16; ++e) o[g][j][e] = fmaf(p[g], x[e], o[g][j][e]);
        }
    };
    // raise every head's reference max to cover z (rare)
    auto rescale = [&](float (&z)[HG]) {
        if constexpr (TRANS) {
            // every head's logit of the row, for the wavefront maxima below
            z[0] = dpp<DPP_NEWBCAST + 0>(z_lane);
            z[1] = dpp<DPP_NEWBCAST + 8>(z_lane);
            z[2] = dpp<DPP_NEWBCAST + 4>(z_lane);
            z[3] = dpp<DPP_NEWBCAST + 12>(z_lane);
            z[4] = dpp<DPP_NEWBCAST + 2>(z_lane);
            z[5] = dpp<DPP_NEWBCAST + 10>(z_lane);
            z[6] = dpp<DPP_NEWBCAST + 6>(z_lane);
            z[7] = dpp<DPP_NEWBCAST + 14>(z_lane);
            float al = 1.f, ml = m_lane;
#pragma unroll
            for (int g = 0; g < HG; ++g) {
                const float mn = fmaxf(m[g], wave_max(z[g]));
                const float alpha = mn == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m[g] - mn);
#pragma unroll
                for (int j = 0; j < VPL; ++j)
#pragma unroll
                    for (int e = 0; e < PER16; ++e) o[g][j][e] *= alpha;
                m[g] = mn;
                al = hd == g ? alpha : al;
                ml = hd == g ? mn : ml;
            }
            l_lane *= al;
            m_lane = ml;
            return;
        }
#pragma unroll
        for (int g = 0; g < HG; ++g) {
            const float mn = fmaxf(m[g], wave_max(z[g]));
            const float alpha = mn == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m[g] - mn);   // 0 while nothing was seen
            l[g] *= alpha;
#pragma unroll
            for (int j = 0; j < VPL; ++j)
#pragma unroll
                for (int e = 0; e < PER16; ++e) o[g][j][e] *= alpha;
            m[g] = mn;
        }
    };

    if (w0 < w1) {      // wavefront-uniform
        const int nst = (int)ceil_div(w1 - w0, RPS);
        unsigned valid = 0u;
#pragma unroll
        for (int s = 0; s < NS - 1; ++s) issue(w0 + (int64_t)s * RPS, s, valid);
        // The hot loop has no rescale in it (a rescale inside makes the
        // compiler copy every accumulator each step): a step whose logits
        // would pass the reference leaves the loop, is rescaled and
        // accumulated outside, and the loop resumes at the next step.
        int i = 0;
        float z[HG];
        for (;;) {
            bool grew = false;
            for (; i < nst; ++i) {
                // past the range these loads read pool row 0 (kept uniform so
                // the wait below is a constant)
                issue(w0 + (int64_t)(i + NS - 1) * RPS, (i + NS - 1) % NS, valid);
                wait_vmem<(NS - 1) * 2 * VPL>();          // step i has landed
                const char *sb = myring + (i % NS) * SLOTB;
                if (logits(sb, (valid >> (i % NS)) & 1u, z)) {
                    grew = true;
                    break;
                }
                accumulate(sb, z);
            }
            if (!grew) break;
            rescale(z);
            accumulate(myring + (i % NS) * SLOTB, z);
            ++i;
        }
        wait_vmem<0>();     // the ring is reused below
    }

    if constexpr (TRANS) {
        // each head's sum from the first lane holding it, for the whole row
        l[0] = dpp<DPP_NEWBCAST + 0>(l_lane);
        l[1] = dpp<DPP_NEWBCAST + 8>(l_lane);
        l[2] = dpp<DPP_NEWBCAST + 4>(l_lane);
        l[3] = dpp<DPP_NEWBCAST + 12>(l_lane);
        l[4] = dpp<DPP_NEWBCAST + 2>(l_lane);
        l[5] = dpp<DPP_NEWBCAST + 10>(l_lane);
        l[6] = dpp<DPP_NEWBCAST + 6>(l_lane);
        l[7] = dpp<DPP_NEWBCAST + 14>(l_lane);
    }
    // The wavefront's partial state.  First the row groups within each 16-lane
    // DPP row are summed (m is wavefront-uniform) ...
#pragma unroll
    for (int g = 0; g < HG; ++g) {
        l[g] = row_groups_sum<LPR>(l[g]);
#pragma unroll
        for (int j = 0; j < VPL; ++j)
#pragma unroll
            for (int e = 0; e < PER16; ++e) o[g][j][e] = row_groups_sum<LPR>(o[g][j][e]);
    }
    // ... then the four DPP rows, in transposed form: a swap of the wave halves
    // (permlane32) and an add turn two values into one register holding one
    // value's half-sums in lanes 0-31 and the other's in lanes 32-63; a swap of
    // neighbouring rows (permlane16) and an add do the same again.  Afterwards
    // register k of DPP row rho holds the wavefront's total of value
    // 4 k + {0, 2, 1, 3}[rho] (value n = (g * VPL + j) * PER16 + e) for the
    // row's slices.
    constexpr int NV = HG * VPL * PER16, COP = 16 / LPR;
    static_assert(NV % (4 * COP) == 0, "transposed reduction shape");
    float s2[NV / 4];
    {
        float s1[NV / 2];
#pragma unroll
        for (int i = 0; i < NV / 2; ++i) {
            const int n0 = 2 * i, n1 = 2 * i + 1;
            const float a0 = o[n0 / (VPL * PER16)][(n0 / PER16) % VPL][n0 % PER16];
            const float a1 = o[n1 / (VPL * PER16)][(n1 / PER16) % VPL][n1 % PER16];
            const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a0), __float_as_uint(a1), false, false);
            s1[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
        }
#pragma unroll
        for (int k = 0; k < NV / 4; ++k) {
            const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(s1[2 * k]), __float_as_uint(s1[2 * k + 1]),
                                                            false, false);
            s2[k] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
        }
    }
    // The COP lanes of a row holding the same slice split the registers; each
    // store instruction then covers 64 consecutive floats of one head.  The
    // state goes to the wavefront's own ring, whose loads have all landed.
    {
        const int rho = lane / 16, cp = (lane % 16) / LPR;
        const int pr = rho == 1 ? 2 : (rho == 2 ? 1 : rho);
#pragma unroll
        for (int i = 0; i < NV / (4 * COP); ++i) {
            float x = s2[i * COP];
#pragma unroll
            for (int q = 1; q < COP; ++q) x = cp == q ? s2[i * COP + q] : x;
            const int n = 4 * (i * COP + cp) + pr;
            const int g = n / (VPL * PER16), j = (n / PER16) % VPL, e = n % PER16;
            reinterpret_cast<float *>(ring + wave * (NS * SLOTB))[g * D + (j * LPR + c) * PER16 + e] = x;
        }
    }
    const int part = wave * 4 + lane / 16;
    if (lane % 16 == 0) {
#pragma unroll
        for (int g = 0; g < HG; ++g) l_s[part][g] = l[g];
    }
    if (lane == 0) {
#pragma unroll
        for (int g = 0; g < HG; ++g) m_s[wave][g] = m[g];
    }
    __syncthreads();    // partial states written

    // Combine.  An item is 4 consecutive output columns of one head; SUB
    // adjacent threads share an item, each rescaling and adding WAVES / SUB of
    // the wavefronts' states, and DPP adds combine them.
    constexpr int ITEMS = HG * D / 4, THREADS = 64 * WAVES;
    constexpr int SUB_T = THREADS / ITEMS >= 4 ? 4 : (THREADS / ITEMS >= 2 ? 2 : 1);
    constexpr int SUB = SUB_T < WAVES ? SUB_T : WAVES;
    constexpr int PW = WAVES / SUB;
    static_assert(WAVES % SUB == 0, "combine split");
    const int sub = tid % SUB;
    for (int it = tid / SUB; it < ITEMS; it += THREADS / SUB) {     // uniform within a SUB group
        const int g = it * 4 / D, cc = it * 4 % D;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) M = fmaxf(M, m_s[w][g]);
        float Lsum = 0.f;
        float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
        if (M > -INFINITY) {
#pragma unroll
            for (int wp = 0; wp < PW; ++wp) {
                const int w = sub * PW + wp;
                const float a = m_s[w][g] > -INFINITY ? __builtin_amdgcn_exp2f(m_s[w][g] - M) : 0.f;
                const float lw = (l_s[4 * w][g] + l_s[4 * w + 1][g]) + (l_s[4 * w + 2][g] + l_s[4 * w + 3][g]);
                const float4 x = *reinterpret_cast<const float4 *>(ring + w * (NS * SLOTB) + (g * D + cc) * 4);
                Lsum = fmaf(a, lw, Lsum);
                O.x = fmaf(a, x.x, O.x);
                O.y = fmaf(a, x.y, O.y);
                O.z = fmaf(a, x.z, O.z);
                O.w = fmaf(a, x.w, O.w);
            }
        }
        if constexpr (SUB >= 2) {
            Lsum += dpp<DPP_XOR1>(Lsum);
            O.x += dpp<DPP_XOR1>(O.x);
            O.y += dpp<DPP_XOR1>(O.y);
            O.z += dpp<DPP_XOR1>(O.z);
            O.w += dpp<DPP_XOR1>(O.w);
        }
        if constexpr (SUB == 4) {
            Lsum += dpp<DPP_XOR2>(Lsum);
            O.x += dpp<DPP_XOR2>(O.x);
            O.y += dpp<DPP_XOR2>(O.y);
            O.z += dpp<DPP_XOR2>(O.z);
            O.w += dpp<DPP_XOR2>(O.w);
        }
        const int gl = (int)blockIdx.z * HG + g;       // head within the KV group
        if (sub == 0) {
            if (nsplit == 1) {
                float *po = out + ((int64_t)b * Hq + gq0 + g) * D + cc;
                const float inv = Lsum > 0.f ? 1.f / Lsum : 0.f;
                if ((reinterpret_cast<uintptr_t>(po) & 15u) == 0) {
                    *reinterpret_cast<float4 *>(po) = make_float4(O.x * inv, O.y * inv, O.z * inv, O.w * inv);
                } else {
                    po[0] = O.x * inv;
                    po[1] = O.y * inv;
                    po[2] = O.z * inv;
                    po[3] = O.w * inv;
                }
            } else {
                float *pp = part_ptr(ws, unit, nsplit, split, G, D) + (int64_t)gl * (D + 2);
                if (cc == 0) { pp[0] = M; pp[1] = Lsum; }
                pp[2 + cc] = O.x;
                pp[3 + cc] = O.y;
                pp[4 + cc] = O.z;
                pp[5 + cc] = O.w;
            }
        }
    }
}

// Combines the states of a unit's splits; splits that start at or past the
// unit's (clamped) row count wrote none and are skipped.  split_rows == 0:
// equal parts, all of which a unit with rows wrote.
template <int D, int G>
__global__ __launch_bounds__(256) void decode_merge_kernel(int Hq, int Hkv, int nsplit, const int32_t *__restrict__ n_rows,
                                                          int64_t max_rows, int64_t split_rows,
                                                          const float *__restrict__ ws, float *__restrict__ out) {
    const int64_t unit = blockIdx.x;
    const int b = (int)(unit / Hkv), h = (int)(unit % Hkv);
    const int64_t n = max<int64_t>(0, min<int64_t>(n_rows[unit], max_rows));
    const int used = split_rows > 0 ? (int)min<int64_t>(nsplit, ceil_div(n, split_rows)) : (n > 0 ? nsplit : 0);
    float *w = const_cast<float *>(ws);
    for (int i = threadIdx.x; i < G * D; i += 256) {
        const int g = i / D, c = i % D;
        float M = -INFINITY;
        for (int s = 0; s < used; ++s) M = fmaxf(M, part_ptr(w, unit, nsplit, s, G, D)[g * (D + 2)]);
        float Lsum = 0.f, O = 0.f;
        if (M > -INFINITY) {
            for (int s = 0; s < used; ++s) {
                const float *pp = part_ptr(w, unit, nsplit, s, G, D) + (int64_t)g * (D + 2);
                if (pp[0] > -INFINITY) {
                    const float a = __builtin_amdgcn_exp2f(pp[0] - M);
                    Lsum += a * pp[1];
                    O += a * pp[2 + c];
                }
            }
        }
        out[((int64_t)b * Hq + (int64_t)h * G + g) * D + c] = Lsum > 0.f ? O / Lsum : 0.f;
    }
}

// Most splits a call can use (the workspace is sized for it): splits are at
// least DEC_MIN_SPLIT_ROWS rows long.
static int64_t max_splits(int64_t max_rows) { return std::max<int64_t>(1, ceil_div(max_rows, DEC_MIN_SPLIT_ROWS)); }

// Rows per split, where the equal-parts mode does not apply:
//   - fewer units than CUs: enough splits to give every CU a workgroup;
//   - between one and four units per CU: splits of at most DEC_CAP_ROWS, so
//     that long units (a batch of prompts of different lengths) do not leave
//     the chip idle behind them once the short ones are done (measured on
//     the 64-request workload, one launch per layer: 0.67 of HBM peak against
//     0.61 with one split per unit).  The equal-parts mode, which also
//     balances the shader engines and orders each engine's work longest
//     first, reached 0.68-0.70 there (and 0.45 against 0.39 for the 80-layer
//     8-head launch);
//   - more units: one split per unit (the workgroups balance by themselves,
//     and extra splits only add merge work).
// A split never spans more page entries than the LDS stage holds and starts
// on a page boundary.
static int64_t plan_split_rows(int64_t wgs_per_split, int64_t max_rows, int page_size) {
    int64_t want = 1;
    if (wgs_per_split < device_cus()) want = ceil_div(device_cus(), wgs_per_split);
    int64_t rows = std::max<int64_t>(ceil_div(max_rows, want), DEC_MIN_SPLIT_ROWS);
    if (wgs_per_split > device_cus() && wgs_per_split < 4 * (int64_t)device_cus())
        rows = std::min<int64_t>(rows, DEC_CAP_ROWS);
    rows = std::min<int64_t>(rows, (int64_t)DEC_PT_CAP * page_size);
    return ceil_div(rows, page_size) * page_size;
}

template <typename T, int D, int G>
static int launch_decode(const char *fn, hipStream_t s, int B, int Hq, int Hkv, float scale_log2, const void *q,
                         const void *k_pool, const void *v_pool, int64_t pool_rows, const int32_t *page_table,
                         const int32_t *n_rows, int page_size, int max_pages, float *out, float *ws, size_t ws_bytes) {
    constexpr int HG = G < DEC_MAX_HG ? G : DEC_MAX_HG;
    constexpr int NHG = G / HG;
    constexpr int WAVES = DecodeShape<T, D, HG>::WAVES;
    const int64_t units = (int64_t)B * Hkv;
    const int64_t max_rows = (int64_t)max_pages * page_size;
    // between one and four units per CU: equal parts spread over the shader
    // engines (see the kernel), where the unit counts and sizes allow it
    const int64_t wgs = units * NHG;
    const bool parts = NHG == 1 && wgs > device_cus() && wgs < 4 * (int64_t)device_cus() &&
                       ceil_div(units, DEC_XCDS) <= DEC_BIN_MAX && max_rows >= DEC_PARTS * DEC_MIN_SPLIT_ROWS &&
                       ceil_div(ceil_div(max_rows, DEC_PARTS), page_size) + 1 <= DEC_PT_CAP;
    const int64_t split_rows = parts ? 0 : plan_split_rows(wgs, max_rows, page_size);
    const int64_t nsplit = parts ? DEC_PARTS : ceil_div(max_rows, split_rows);
    if (nsplit > 65535 || nsplit > max_splits(max_rows)) {
        set_error("%s: %lld splits of %lld rows are not supported", fn, (long long)nsplit, (long long)split_rows);
        return SG_EUNSUPPORTED;
    }
    const size_t need = nsplit > 1 ? (size_t)units * nsplit * G * (D + 2) * sizeof(float) : 0;
    if (need > ws_bytes || (need && !ws)) {
        set_error("%s: the split states need %zu bytes of workspace, %zu given", fn, need, ws_bytes);
        return SG_EWORKSPACE;
    }
    // division by the page size as a multiply-shift, exact for dividends below
    // 2^30 (Granlund and Montgomery, 1994): with l = ceil(log2 P) and
    // k = 30 + l, floor(n / P) = (n * ceil(2^k / P)) >> k, and the multiplier
    // is at most 2^31
    int lg = 0;
    while ((1ll << lg) < page_size) ++lg;
    const int page_shift = 30 + lg;
    const uint32_t page_mul = (uint32_t)(((1ull << page_shift) + (uint64_t)page_size - 1) / (uint64_t)page_size);
    dim3 grid((unsigned)units, (unsigned)nsplit, (unsigned)NHG);
    if (parts)
        grid = dim3((unsigned)(DEC_XCDS * DEC_ENGINES *
                               ceil_div(ceil_div(units, DEC_XCDS), DEC_ENGINES / DEC_PARTS)), 1, 1);
    decode_kernel<T, D, HG><<<grid, 64 * WAVES, 0, s>>>(
        Hq, Hkv, scale_log2, reinterpret_cast<const T *>(q), reinterpret_cast<const v4u *>(k_pool),
        reinterpret_cast<const v4u *>(v_pool), pool_rows, page_table, n_rows, page_size, page_mul, page_shift,
        max_pages, split_rows, out, ws, (int)units, parts ? DEC_PARTS : 0);
    if (nsplit > 1)
        decode_merge_kernel<D, G><<<(unsigned)units, 256, 0, s>>>(Hq, Hkv, (int)nsplit, n_rows, max_rows, split_rows, ws,
                                                                  out);
    return launch_status(fn);
}

template <typename T, int D>
static int dispatch_g(const char *fn, int G, hipStream_t s, int B, int Hq, int Hkv, float sl2, const void *q, const void *kp,
                      const void *vp, int64_t pr, const int32_t *pt, const int32_t *nr, int ps, int mp, float *out,
                      float *ws, size_t wsb) {
    switch (G) {
        case 1: return launch_decode<T, D, 1>(fn, s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, wsb);
        case 2: return launch_decode<T, D, 2>(fn, s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, wsb);
        case 4: return launch_decode<T, D, 4>(fn, s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, wsb);
        case 8: return launch_decode<T, D, 8>(fn, s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, wsb);
        case 16: return launch_decode<T, D, 16>(fn, s, B, Hq, Hkv, sl2, q, kp, vp, pr, pt, nr, ps, mp, out, ws, wsb);
        default: set_error("%s: group size %d not supported (1, 2, 4, 8, 16)", fn, G); return SG_EUNSUPPORTED;
    }
}

// The checks and the dispatch shared by sg_decode_attn and
// sg_decode_attn_noalloc (which differ only in where the split states live).
static int decode_attn_call(const char *fn, void *stream, sg_dtype dt, int B, int Hq, int Hkv, int d, float scale,
                            const void *q, const void *k_pool, const void *v_pool, int64_t pool_rows,
                            const int32_t *page_table, const int32_t *n_rows, int page_size, int max_pages,
                            float *out, void *ws, size_t ws_bytes) {
    SG_REQUIRE(dt == SG_F32 || dt == SG_BF16, SG_EINVAL, "%s: unknown dtype %d", fn, (int)dt);
    SG_REQUIRE(B >= 0 && Hq >= 1 && Hkv >= 1 && Hq % Hkv == 0, SG_EINVAL,
               "%s: need Hq %% Hkv == 0 (Hq=%d, Hkv=%d)", fn, Hq, Hkv);
    SG_REQUIRE(d == 64 || d == 128, SG_EUNSUPPORTED, "%s: head dimension %d not supported", fn, d);
    SG_REQUIRE(page_size >= 1 && max_pages >= 1 && pool_rows >= 0, SG_EINVAL, "%s: bad page geometry", fn);
    SG_REQUIRE((int64_t)max_pages * page_size <= (1ll << 30), SG_EINVAL, "%s: page table too large", fn);
    SG_REQUIRE(pool_rows <= 0x7fffffffll, SG_EUNSUPPORTED, "%s: pool above 2^31 rows", fn);
    SG_REQUIRE(scale == scale && scale > 0.f, SG_EINVAL, "%s: scale must be positive", fn);
    if (B == 0) return SG_OK;
    SG_REQUIRE(q && k_pool && v_pool && page_table && n_rows && out, SG_EINVAL, "%s: null pointer", fn);
    SG_REQUIRE(aligned16(k_pool) && aligned16(v_pool) && aligned16(q), SG_EINVAL,
               "%s: q and pools must be 16-byte aligned", fn);
    SG_REQUIRE((int64_t)B * Hkv <= 0x7fffffffll, SG_EINVAL, "%s: too many units", fn);
    const float sl2 = scale * 1.4426950408889634f;  // log2(e)
    const int G = Hq / Hkv;
    hipStream_t s = as_stream(stream);
    float *w = reinterpret_cast<float *>(ws);
    if (dt == SG_F32) {
        if (d == 64) return dispatch_g<float, 64>(fn, G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, ws_bytes);
        return dispatch_g<float, 128>(fn, G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, ws_bytes);
    }
    if (d == 64) return dispatch_g<uint16_t, 64>(fn, G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, ws_bytes);
    return dispatch_g<uint16_t, 128>(fn, G, s, B, Hq, Hkv, sl2, q, k_pool, v_pool, pool_rows, page_table, n_rows, page_size, max_pages, out, w, ws_bytes);
}

// Split states of sg_decode_attn_noalloc: a file-scope device array, one copy
// per GPU, held until the process ends.  Host code never passes the array's
// name to a kernel (on the host it only stands for the symbol); it uses the
// device address resolved once per device below.
constexpr size_t DEC_SCRATCH_BYTES = (size_t)16 << 20;
static __device__ __align__(256) char scratch[DEC_SCRATCH_BYTES];
constexpr int DEC_SCRATCH_DEVICES = 64;

// Device address of `scratch` on the current device, resolved with
// hipGetSymbolAddress on the first call per device; nullptr (with the error
// set) when that fails.
static void *scratch_address(const char *fn) {
    static std::mutex mu;
    static void *addr[DEC_SCRATCH_DEVICES] = {};
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= DEC_SCRATCH_DEVICES) {
        (void)hipGetLastError();
        set_error("%s: no usable current device (%d)", fn, dev);
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            set_error("%s: hipGetSymbolAddress of the scratch array failed on device %d: %s", fn, dev,
                      hipGetErrorString(e));
            return nullptr;
        }
        addr[dev] = p;
    }
    return addr[dev];
}

}  // namespace sg

using namespace sg;

extern "C" size_t sg_decode_attn_workspace_size(int B, int Hq, int Hkv, int d, int max_pages, int page_size) {
    if (B <= 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv != 0 || d <= 0 || max_pages <= 0 || page_size <= 0) return 0;
    const int G = Hq / Hkv;
    const int64_t cap = max_splits((int64_t)max_pages * page_size);
    if (cap <= 1) return 0;
    return (size_t)B * Hkv * cap * G * (size_t)(d + 2) * sizeof(float);
}

extern "C" int sg_decode_attn(void *stream, sg_dtype dt, int B, int Hq, int Hkv, int d, float scale, const void *q,
                              const void *k_pool, const void *v_pool, int64_t pool_rows, const int32_t *page_table,
                              const int32_t *n_rows, int page_size, int max_pages, float *out, void *ws,
                              size_t ws_bytes) {
    return decode_attn_call("sg_decode_attn", stream, dt, B, Hq, Hkv, d, scale, q, k_pool, v_pool, pool_rows,
                            page_table, n_rows, page_size, max_pages, out, ws, ws_bytes);
}

extern "C" size_t sg_decode_attn_noalloc_scratch_bytes(void) { return DEC_SCRATCH_BYTES; }

extern "C" int sg_decode_attn_noalloc(void *stream, sg_dtype dt, int B, int Hq, int Hkv, int d, float scale,
                                      const void *q, const void *k_pool, const void *v_pool, int64_t pool_rows,
                                      const int32_t *page_table, const int32_t *n_rows, int page_size, int max_pages,
                                      float *out) {
    void *ws = scratch_address("sg_decode_attn_noalloc");
    if (!ws) return SG_EHIP;
    return decode_attn_call("sg_decode_attn_noalloc", stream, dt, B, Hq, Hkv, d, scale, q, k_pool, v_pool, pool_rows,
                            page_table, n_rows, page_size, max_pages, out, ws, DEC_SCRATCH_BYTES);
}
