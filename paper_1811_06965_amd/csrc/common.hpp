// common.hpp -- device helpers shared by the partition's HIP kernels (gfx950,
// wave64).  Element types: `float` (fp32 partitions) and `bf16` (__bf16
// storage; arithmetic is always fp32).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace gp {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int WAVE = 64;

// fp32 -> storage type, round to nearest even (the gfx950 conversion
// instruction rounds RNE and keeps NaN quiet).
template <typename T> __device__ __forceinline__ T to_elt(float v);
template <> __device__ __forceinline__ float to_elt<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 to_elt<bf16>(float v) { return (bf16)v; }

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, WAVE));
    return v;
}

// ---- OCP e2m1 (fp4) with one E8M0 scale per row: the low-precision operand
// of a GEMM correction term (see GemmArgs::a4).  The scale of a row is
// 2^(e - 2), e = floor(log2 max|v|), so every |v| / scale < 8; values round to
// the nearest of 0, 0.5, 1, 1.5, 2, 3, 4, 6 (ties to the even code) and
// saturate at 6.
__device__ __forceinline__ unsigned e8m0_for_amax(float amax) {
    const int eb = (int)((__float_as_uint(amax) >> 23) & 255u);  // biased exponent of max|v|
    return eb >= 2 ? (unsigned)(eb - 2) : 0u;                    // 0: the row is (nearly) zero
}
// 1 / scale for an E8M0 code (0 when the code is 0, which zeroes the row)
__device__ __forceinline__ float e8m0_inv(unsigned code) {
    return code ? __uint_as_float((254u - code) << 23) : 0.f;
}
__device__ __forceinline__ unsigned e2m1_code(float q) {
    const float a = fabsf(q);
    unsigned c = a > 0.25f ? 1u : 0u;
    c = a >= 0.75f ? 2u : c;
    c = a > 1.25f ? 3u : c;
    c = a >= 1.75f ? 4u : c;
    c = a > 2.5f ? 5u : c;
    c = a >= 3.5f ? 6u : c;
    c = a > 5.f ? 7u : c;
    return c | ((q < 0.f && c) ? 8u : 0u);
}
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}

// 16-byte vector of storage elements (8 bf16 or 4 float).
template <typename T> struct Vec16;
template <> struct Vec16<bf16> {
    static constexpr int N = 8;
    typedef bf16x8 type;
};
template <> struct Vec16<float> {
    static constexpr int N = 4;
    typedef f32x4 type;
};

} // namespace gp

// Host-side launch checking (used inside functions returning gp_status):
// reports the first failed launch (klaunch) of the calling thread since the
// last check.
#define GP_LAUNCH_CHECK()                                                   \
    do {                                                                    \
        hipError_t e_ = ::gp::take_launch_status();                          \
        if (e_ != hipSuccess) return ::gp::hip_fail(e_, __FILE__, __LINE__); \
    } while (0)

#define GP_HIP(call)                                                        \
    do {                                                                    \
        hipError_t e_ = (call);                                             \
        if (e_ != hipSuccess) return ::gp::hip_fail(e_, __FILE__, __LINE__); \
    } while (0)

#include <hip/hip_ext.h>
#include <tuple>
#include "../../include/gp.h"
namespace gp {
gp_status hip_fail(hipError_t e, const char* file, int line);
gp_status set_error(gp_status s, const char* msg);

// Launch timing: while a launch role is timed, the first kernel launched
// takes `start` (its dispatch start timestamp) and every kernel takes `stop`
// (so the last one's completion ends the interval).  Thread-local, set by the
// partition around one role's launches.
struct LaunchEvents {
    hipEvent_t start = nullptr, stop = nullptr;
    bool started = false;
};
LaunchEvents& launch_events();
hipError_t& launch_status();  // first failed launch of the calling thread, or hipSuccess
inline hipError_t take_launch_status() {
    hipError_t& e = launch_status();
    const hipError_t r = e;
    e = hipSuccess;
    return r;
}

// Kernel launch.  While a role is timed, through hipExtLaunchKernelGGL with
// the timing events attached to the dispatch (no extra stream packets);
// otherwise a plain hipLaunchKernel (which stream capture records as an
// ordinary kernel node).
template <typename... Args, typename... P>
inline void klaunch(void (*k)(Args...), dim3 grid, dim3 block, uint32_t shmem, hipStream_t st, P... p) {
    LaunchEvents& ev = launch_events();
    auto args = std::make_tuple(static_cast<Args>(p)...);
    void* ptrs[sizeof...(Args) > 0 ? sizeof...(Args) : 1];
    std::apply([&](auto&... a) {
        int i = 0;
        ((ptrs[i++] = static_cast<void*>(&a)), ...);
    }, args);
    hipError_t e;
    if (ev.stop) {
        hipEvent_t e0 = nullptr;
        if (!ev.started) {
            e0 = ev.start;
            ev.started = true;
        }
        e = hipExtLaunchKernel(reinterpret_cast<const void*>(k), grid, block, ptrs, shmem, st, e0, ev.stop, 0);
    } else {
        e = hipLaunchKernel(reinterpret_cast<const void*>(k), grid, block, ptrs, shmem, st);
    }
    if (e != hipSuccess && launch_status() == hipSuccess) launch_status() = e;
}
}
