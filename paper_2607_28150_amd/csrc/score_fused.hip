// sg_score, single pass: every logit is computed once.
//
// A job is one 128-key chunk of one unit.  The job's workgroup (ceil(R/64)
// wavefronts, 64 query rows each) multiplies its rows against the chunk with
// MFMA and keeps the resulting 64 x 128 block per wavefront in registers.  It
// turns the block into p~ = exp2(z - m_c) with the chunk's own row maxima
// m_c, and publishes (m_c, sum p~) per row.  The unit's jobs then meet twice:
//
//   barrier A: all chunks published -> each job merges the partials of its
//              own share of the rows into the row's log-sum-exp (log2 units);
//   barrier B: all row LSEs written -> each job scales its rows by
//              alpha = exp2(m_c - lse) and sums its registers over the rows,
//              which gives the normalised column sums of its 128 keys.
//
// The launch is cooperative and persistent (every workgroup resident), jobs
// are assigned round by round, and the chunks of one unit always share a
// round, so a job only ever waits for jobs that are running: no deadlock is
// possible.  Where a round holds whole units per XCD (chunks <= slots per XCD)
// the chunks of a unit are placed on one XCD, keeping the exchange inside one
// L2.  Waits are bounded; a timed-out wait sets the workspace status word.
// Counters start at zero: a small kernel clears them before every launch.
#include "score_common.h"

namespace sg {

constexpr int SF_NT = 128;                  // keys per job
constexpr int SF_KB = SF_NT / 16;           // 16-key blocks per job
constexpr uint32_t SF_SPIN_LIMIT = 1u << 26;  // bounded waits (seconds of polling)

struct FusedArgs {
    int B, L, Hq, Hkv, W, G, R;
    const int32_t *cu_seqlens;
    int64_t T;
    const void *q_win;
    const void *k;
    int64_t k_layer_rows;
    float c2;            // log2(e) / sqrt(d)
    int C;               // chunk slots per unit (ceil(max_seqlen / 128))
    int units;
    int rounds;
    int units_per_round;
    int xcd_local;       // 1: a unit's chunks sit on one XCD
    float2 *part;        // [units][C][R] (m, s), log2 units
    float *lse2;         // [units][R]
    int *cnt;            // [units][2][C] arrival flags
    int *status;         // [1]
    float *scores;
};

__device__ __forceinline__ float ld_agent(const float *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(float *p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// All data a unit's jobs exchange (row partials, row LSEs, arrival flags) is
// written and read with device-scope (sc1) accesses, which are coherent across
// CUs and XCDs without whole-cache write-back or invalidation.  Arrival: every
// wavefront waits for its own device-scope stores to complete, the workgroup
// meets, and one thread raises this job's flag (no shared counter, so nothing
// serialises on one address).  Waiting: wavefront 0 reads all Cu flags of the
// phase at once (one lane per flag) until every one is raised; then the
// workgroup meets again before reading the partners' data.
__device__ __forceinline__ void unit_barrier(int *flags, int c, int Cu, int *status) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) __hip_atomic_store(flags + c, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        uint32_t spins = 0;
        while (true) {
            bool up = true;
            for (int j = lane; j < Cu; j += 64)
                up = up && __hip_atomic_load(flags + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
            if (__ballot(!up) == 0) break;
            __builtin_amdgcn_s_sleep(1);
            // after any timed-out wait every later wait gives up at once
            if (++spins > SF_SPIN_LIMIT || __hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                if (lane == 0) __hip_atomic_store(status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
        }
    }
    __syncthreads();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// max / sum over the 16 lanes of a row of 16 (DPP within a row of the wave)
template <int CTRL>
__device__ __forceinline__ float dppf(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float row16_max(float x) {
    x = fmaxf(x, dppf<0xB1>(x));   // quad_perm [1,0,3,2]
    x = fmaxf(x, dppf<0x4E>(x));   // quad_perm [2,3,0,1]
    x = fmaxf(x, dppf<0x124>(x));  // row_ror:4
    x = fmaxf(x, dppf<0x128>(x));  // row_ror:8
    return x;
}
__device__ __forceinline__ float row16_sum(float x) {
    x += dppf<0xB1>(x);
    x += dppf<0x4E>(x);
    x += dppf<0x124>(x);
    x += dppf<0x128>(x);
    return x;
}

template <typename T, int D>
__global__ __launch_bounds__(512) void score_fused_kernel(FusedArgs a) {
    __shared__ __attribute__((aligned(16))) char tile[2 * SC_TK * Frag<T, D>::ROWB];
    __shared__ float csum[SC_MAXR / 64][SF_NT];
    __shared__ float lse_s[SC_MAXR];
    using F = Frag<T, D>;
    const int lane = threadIdx.x % 64;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const int nwave = blockDim.x / 64;
    const int R = a.R, W = a.W, C = a.C;
    const int slots = gridDim.x;

    for (int round = 0; round < a.rounds; ++round) {
        // ---- job of this workgroup in this round
        const int s = blockIdx.x;
        int ui, c;
        if (a.xcd_local) {
            const int per = slots / 8;                       // slots per XCD
            ui = (s % 8) + 8 * ((s / 8) / C);
            c = (s / 8) % C;
            if ((s / 8) / C >= per / C) ui = a.units_per_round;   // slot beyond the last whole unit
        } else {
            ui = s / C;
            c = s % C;
        }
        if (ui >= a.units_per_round) continue;
        const int64_t u = (int64_t)round * a.units_per_round + ui;
        if (u >= a.units) continue;
        const UnitGeom g = unit_geom(u, a.B, a.Hkv, a.cu_seqlens, a.T);
        const int N = (int)g.N;
        if (N < W) continue;                                  // such units get zero scores elsewhere
        const int Cu = min(C, (N + SF_NT - 1) / SF_NT);       // real chunks of this unit
        if (c >= Cu) continue;
        const int key0 = c * SF_NT;

        const T *qunit = reinterpret_cast<const T *>(a.q_win) +
                         (((int64_t)g.b * a.L + g.l) * a.Hq + (int64_t)g.h * a.G) * W * D;
        const T *kunit = reinterpret_cast<const T *>(a.k) + ((int64_t)g.l * a.k_layer_rows + (int64_t)g.h * a.T + g.s0) * D;

        // ---- logits of the chunk: acc[rb][kb] = Q(rows rb) . K(keys kb), kept in registers
        typename F::A qa[4][F::KSTEPS];
        load_q<T, D>(qunit, R, wave, lane, qa);
        __syncthreads();                                      // previous job done with the tile
        stage_tile<T, D>(tile, kunit, key0, N);
        stage_tile<T, D>(tile + SC_TK * F::ROWB, kunit, key0 + SC_TK, N);
        __syncthreads();
        f32x4 acc[4][SF_KB];
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int kb = 0; kb < SF_KB; ++kb) acc[rb][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < F::KSTEPS; ++ks) {
#pragma unroll
            for (int kb = 0; kb < SF_KB; ++kb) {
                const auto bf = F::load_lds(tile, kb * 16 + lane % 16, ks, lane);
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) acc[rb][kb] = F::mma(qa[rb][ks], bf, acc[rb][kb]);
            }
        }

        // ---- chunk row statistics; acc becomes p~ = exp2(z - m_c)
        // this lane's rows: r = wave*64 + rb*16 + 4*(lane/16) + i; its keys: kb*16 + lane%16
        const bool full = key0 + SF_NT - 1 <= N - W;          // every row sees every key
        float mrow[4][4];
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = wave * 64 + rb * 16 + 4 * (lane / 16) + i;
                const int pos = r < R ? N - W + (r % W) : -1;   // causal limit of the row
                float mx = -INFINITY;
                if (full) {
#pragma unroll
                    for (int kb = 0; kb < SF_KB; ++kb) mx = fmaxf(mx, acc[rb][kb][i]);
                } else {
#pragma unroll
                    for (int kb = 0; kb < SF_KB; ++kb) {
                        const int key = key0 + kb * 16 + lane % 16;
                        if (key > pos) acc[rb][kb][i] = -INFINITY;
                        mx = fmaxf(mx, acc[rb][kb][i]);
                    }
                }
                mx = row16_max(mx) * a.c2;                       // log2 units (scale > 0)
                float sum = 0.f;
                if (mx > -INFINITY) {
#pragma unroll
                    for (int kb = 0; kb < SF_KB; ++kb) {
                        const float p = __builtin_amdgcn_exp2f(fmaf(acc[rb][kb][i], a.c2, -mx));
                        acc[rb][kb][i] = p;
                        sum += p;
                    }
                } else {
#pragma unroll
                    for (int kb = 0; kb < SF_KB; ++kb) acc[rb][kb][i] = 0.f;
                }
                sum = row16_sum(sum);
                mrow[rb][i] = mx;
                if (lane % 16 == 0 && r < R) {
                    float *pp = reinterpret_cast<float *>(a.part + ((int64_t)u * C + c) * R + r);
                    st_agent(pp, mx);
                    st_agent(pp + 1, sum);
                }
            }

        // ---- barrier A, then merge this job's share of the rows into the LSE
        int *flags = a.cnt + (int64_t)u * 2 * C;              // [phase][chunk]
        unit_barrier(flags, c, Cu, a.status);
        // merge: rows [c*rpj, (c+1)*rpj) of the unit; one wavefront per row, one
        // lane per chunk partial (Cu <= 64 here, else lanes loop), all loads in flight at once
        const int rpj = (R + Cu - 1) / Cu;                    // rows merged per job
        for (int rr = wave; rr < rpj; rr += nwave) {
            const int r = c * rpj + rr;
            if (r >= R) break;                                 // uniform per wavefront
            const float *pp = reinterpret_cast<const float *>(a.part + (int64_t)u * C * R + r);
            float mj[4], sj[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int j = lane + 64 * t;
                mj[t] = -INFINITY;
                sj[t] = 0.f;
                if (j < Cu) {
                    mj[t] = ld_agent(pp + 2 * (int64_t)j * R);
                    sj[t] = ld_agent(pp + 2 * (int64_t)j * R + 1);
                }
            }
            float M = fmaxf(fmaxf(mj[0], mj[1]), fmaxf(mj[2], mj[3]));
            M = wave_max(M);
            float S = 0.f;
#pragma unroll
            for (int t = 0; t < 4; ++t)
                if (mj[t] > -INFINITY) S += sj[t] * __builtin_amdgcn_exp2f(mj[t] - M);
            S = wave_sum(S);
            if (lane == 0) st_agent(a.lse2 + (int64_t)u * R + r, M + __log2f(S));
        }
        unit_barrier(flags + C, c, Cu, a.status);
        // the unit's row LSEs, once per workgroup, into LDS
        for (int r = threadIdx.x; r < R; r += blockDim.x) lse_s[r] = ld_agent(a.lse2 + (int64_t)u * R + r);
        __syncthreads();

        // ---- normalised column sums of this chunk's keys
        float cs[SF_KB];
#pragma unroll
        for (int kb = 0; kb < SF_KB; ++kb) cs[kb] = 0.f;
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = wave * 64 + rb * 16 + 4 * (lane / 16) + i;
                float alpha = 0.f;
                if (r < R && mrow[rb][i] > -INFINITY) alpha = __builtin_amdgcn_exp2f(mrow[rb][i] - lse_s[r]);
#pragma unroll
                for (int kb = 0; kb < SF_KB; ++kb) cs[kb] = fmaf(alpha, acc[rb][kb][i], cs[kb]);
            }
#pragma unroll
        for (int kb = 0; kb < SF_KB; ++kb) {
            cs[kb] += __shfl_xor(cs[kb], 16, 64);
            cs[kb] += __shfl_xor(cs[kb], 32, 64);
        }
        if (lane < 16) {
#pragma unroll
            for (int kb = 0; kb < SF_KB; ++kb) csum[wave][kb * 16 + lane] = cs[kb];
        }
        __syncthreads();
        for (int j = threadIdx.x; j < SF_NT; j += blockDim.x) {
            float t = 0.f;
            for (int w = 0; w < nwave; ++w) t += csum[w][j];
            const int key = key0 + j;
            if (key < N) a.scores[((int64_t)g.l * a.Hkv + g.h) * a.T + g.s0 + key] = t;
        }
    }
}

__global__ void score_fused_clear(int *cnt, int n, int *status) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) cnt[i] = 0;
    if (i == 0) *status = 0;
}

// zero scores for units whose prompt is shorter than the window (documented fallback)
__global__ void score_short_units(int B, int L, int Hkv, int W, const int32_t *cu_seqlens, int64_t T,
                                  float *scores) {
    const int64_t u = blockIdx.x;
    const UnitGeom g = unit_geom(u, B, Hkv, cu_seqlens, T);
    if (g.N >= W) return;
    for (int64_t j = threadIdx.x; j < g.N; j += blockDim.x) scores[((int64_t)g.l * Hkv + g.h) * T + g.s0 + j] = 0.f;
}

static int fused_slots(const void *kernel, int threads) {
    int dev = 0, cus = 0, coop = 0, per = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess || !coop) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, threads, 0) != hipSuccess) return 0;
    return per * cus;
}

size_t score_fused_workspace(int B, int L, int Hq, int Hkv, int W, int max_seqlen) {
    const int64_t R = (int64_t)(Hq / Hkv) * W;
    const int64_t units = (int64_t)L * Hkv * B;
    const int64_t C = ceil_div(max_seqlen, SF_NT);
    size_t bytes = (size_t)(units * C * R) * sizeof(float2);       // partials
    bytes += (size_t)(units * R) * sizeof(float);                   // row LSEs
    bytes = (bytes + 255) / 256 * 256;
    bytes += (size_t)units * 2 * C * sizeof(int) + 256;             // arrival flags + status
    return bytes;
}

template <typename T, int D>
static int launch_fused_t(hipStream_t s, int B, int L, int Hq, int Hkv, int W, const int32_t *cu_seqlens,
                          int64_t T_, int max_seqlen, const void *q_win, const void *k, int64_t k_layer_rows,
                          float *scores, void *ws, size_t ws_bytes) {
    const int R = (Hq / Hkv) * W;
    const int threads = (int)ceil_div(R, 64) * 64;
    const int slots = fused_slots(reinterpret_cast<const void *>(&score_fused_kernel<T, D>), threads);
    const int C = (int)ceil_div(max_seqlen, SF_NT);
    if (slots <= 0 || C > slots || C > 256) return SG_EUNSUPPORTED;
    const int64_t units = (int64_t)L * Hkv * B;
    if (units > 0x7fffffff) return SG_EUNSUPPORTED;
    const size_t need = score_fused_workspace(B, L, Hq, Hkv, W, max_seqlen);
    if (ws_bytes < need) {
        set_error("sg_score: workspace %zu < %zu", ws_bytes, need);
        return SG_EWORKSPACE;
    }
    FusedArgs a;
    a.B = B; a.L = L; a.Hq = Hq; a.Hkv = Hkv; a.W = W; a.G = Hq / Hkv; a.R = R;
    a.cu_seqlens = cu_seqlens; a.T = T_; a.q_win = q_win; a.k = k; a.k_layer_rows = k_layer_rows;
    a.c2 = 1.4426950408889634f / sqrtf((float)D);
    a.C = C;
    a.units = (int)units;
    const int per_xcd = slots / 8;
    a.xcd_local = (slots % 8 == 0 && C <= per_xcd) ? 1 : 0;
    a.units_per_round = a.xcd_local ? 8 * (per_xcd / C) : slots / C;
    a.rounds = (int)ceil_div(units, a.units_per_round);
    char *w = reinterpret_cast<char *>(ws);
    a.part = reinterpret_cast<float2 *>(w);
    a.lse2 = reinterpret_cast<float *>(w + units * C * R * sizeof(float2));
    size_t off = ((size_t)(units * C * R) * sizeof(float2) + (size_t)(units * R) * sizeof(float) + 255) / 256 * 256;
    a.cnt = reinterpret_cast<int *>(w + off);
    a.status = a.cnt + 2 * units * C;
    a.scores = scores;
    const int ncnt = (int)(2 * units * C);
    score_fused_clear<<<(unsigned)ceil_div(ncnt, 256), 256, 0, s>>>(a.cnt, ncnt, a.status);
    score_short_units<<<(unsigned)units, 256, 0, s>>>(B, L, Hkv, W, cu_seqlens, T_, scores);
    void *args[] = {&a};
    hipError_t e = hipLaunchCooperativeKernel(reinterpret_cast<const void *>(&score_fused_kernel<T, D>),
                                              dim3((unsigned)slots), dim3((unsigned)threads), args, 0, s);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        set_error("sg_score: cooperative launch failed: %s", hipGetErrorString(e));
        return SG_EHIP;
    }
    return launch_status("sg_score");
}

int launch_score_fused(hipStream_t s, sg_dtype dt, int d, int B, int L, int Hq, int Hkv, int W,
                       const int32_t *cu_seqlens, int64_t T_, int max_seqlen, const void *q_win, const void *k,
                       int64_t k_layer_rows, float *scores, void *ws, size_t ws_bytes) {
    if (dt == SG_BF16) {
        if (d == 128) return launch_fused_t<uint16_t, 128>(s, B, L, Hq, Hkv, W, cu_seqlens, T_, max_seqlen, q_win, k, k_layer_rows, scores, ws, ws_bytes);
        return launch_fused_t<uint16_t, 64>(s, B, L, Hq, Hkv, W, cu_seqlens, T_, max_seqlen, q_win, k, k_layer_rows, scores, ws, ws_bytes);
    }
    if (d == 64) return launch_fused_t<float, 64>(s, B, L, Hq, Hkv, W, cu_seqlens, T_, max_seqlen, q_win, k, k_layer_rows, scores, ws, ws_bytes);
    return SG_EUNSUPPORTED;   // fp32 with d = 128 would not fit the register budget
}

}  // namespace sg
