// Internal helpers shared by the HIP sources of libsmartgen (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>

#include "smartgen.h"

namespace sg {

// native 16-byte vector (usable with the non-temporal load/store builtins)
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// thread-local error detail, read through sg_last_error()
void set_error(const char *fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

#define SG_REQUIRE(cond, code, ...)            \
    do {                                       \
        if (!(cond)) {                         \
            ::sg::set_error(__VA_ARGS__);      \
            return (code);                     \
        }                                      \
    } while (0)

// map the state after a launch to a status
int launch_status(const char *what);
// True for pinned host memory (reached over the host link).  Copies from it
// run on HOST_LINK_WORKGROUPS workgroups, two per XCD (host reads are served
// per XCD: 8 workgroups reached 33 GB/s, 12 reached 48): measured on MI355X,
// that keeps the link near its full rate (57 GB/s), while every further
// outstanding host read also delays the HBM reads of kernels on other streams
// (decode attention beside a host-source copy ran 1.5x slower with 16
// workgroups, 2.7x with 32 and 7x with 64 or more).
bool host_memory(const void *p);
constexpr int HOST_LINK_WORKGROUPS = 16;

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline int esize_of(sg_dtype dt) { return dt == SG_F32 ? 4 : 2; }

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------- device helpers

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// reinterpret a 32-bit word as two bf16 lanes (element 0 = low half); a copy
// through a local word, not a bit_cast of a vector element
__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t w) {
    bf16x2 r;
    __builtin_memcpy(&r, &w, sizeof(r));
    return r;
}

// acc + the dot product of one 16-byte slice of q with the same slice of a K
// row (fp32 accumulation)
template <typename T>
struct SliceDot;
template <>
struct SliceDot<uint16_t> {   // bf16: four chained v_dot2_f32_bf16
    __device__ static float run(const v4u &q, const v4u &k, float acc) {
        acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.x), as_bf16x2(k.x), acc, false);
        acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.y), as_bf16x2(k.y), acc, false);
        acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.z), as_bf16x2(k.z), acc, false);
        return __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.w), as_bf16x2(k.w), acc, false);
    }
};
template <>
struct SliceDot<float> {
    __device__ static float run(const v4u &q, const v4u &k, float acc) {
        acc = fmaf(__uint_as_float(q.x), __uint_as_float(k.x), acc);
        acc = fmaf(__uint_as_float(q.y), __uint_as_float(k.y), acc);
        acc = fmaf(__uint_as_float(q.z), __uint_as_float(k.z), acc);
        return fmaf(__uint_as_float(q.w), __uint_as_float(k.w), acc);
    }
};

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
    return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

__device__ __forceinline__ int wave_sum_int(int x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
    const unsigned lane = __lane_id();
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// LDS offset of a workgroup-shared address.
__device__ __forceinline__ unsigned lds_addr(const void *p) {
    return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) char *)p;
}

// Direct global->LDS load: lane i's 16 bytes land at LDS offset lds + 16 i;
// lds is wavefront-uniform and travels in M0.  Issued from inline assembly:
// the compiler then neither reorders LDS accesses across them (memory
// clobber) nor inserts conservative waits for them before unrelated LDS
// reads; callers wait for completion themselves (vector memory counter)
// before reading the destination.  The s_nop is the wait state a direct LDS
// load needs after M0 is written.  The _nt form marks the read non-temporal
// (streamed data that is not read again soon).
__device__ __forceinline__ void dma16(const void *src, unsigned lds) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(lds) : "memory");
}
__device__ __forceinline__ void dma16_nt(const void *src, unsigned lds) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(src), "{m0}"(lds) : "memory");
}

// Wait until at most N vector memory operations of this wavefront are in
// flight (direct LDS loads included); a compiler barrier for memory.
template <int N>
__device__ __forceinline__ void wait_vmem() {
    static_assert(N >= 0 && N <= 63, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Compute units of the current device (read once; 256 when the query fails).
inline int device_cus() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0, v = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
            cus = v;
        else
            cus = 256;
    }
    return cus;
}

}  // namespace sg
