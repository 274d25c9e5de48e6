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

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline int esize_of(sg_dtype dt) { return dt == SG_F32 ? 4 : 2; }

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------- device helpers

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

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

}  // namespace sg
