// Internal helpers shared by the library's translation units: error
// reporting across the C ABI and the bf16 vector types of the gfx950 MFMA
// builtins.  Not part of the public interface.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <functional>

#include "../../include/sparseserve.h"

namespace ss {

// Records `fmt` as this thread's last error and returns `code`.
ss_status fail(ss_status code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// Checks the last launch on this thread; maps a failure to SS_ERR_HIP.
ss_status check_launch(const char *what);

inline bool supported_blk(int blk) { return blk == 8 || blk == 16 || blk == 32; }
constexpr int kHeadDim = 128;
constexpr int kMaxGroup = 16;
constexpr int kMaxBlocks = 65536;

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// block scoring (score.hip): argument checks and the launch
ss_status check_score_args(const void *q, const void *meta, const int32_t *nblk, int B, int Hq, int Hkv,
                           int nblk_max, int d, const void *scores, const char *who, int meta_kind, int agg);
ss_status launch_score(const void *q, const void *meta, int meta_kind, int agg, const int32_t *nblk, int B, int Hq,
                       int Hkv, int nblk_max, float *scores, hipStream_t s);

// f(begin, end) over [0, n) on the library's host worker threads
void parallel_for(int64_t n, int max_threads, const std::function<void(int64_t, int64_t)> &f);

// Start/stop events that a measurement attaches to the next kernel the
// calling thread launches (ss_time_next_kernel); the launch takes and
// clears them.
struct kernel_timing {
    hipEvent_t start = nullptr, stop = nullptr;
};
kernel_timing take_kernel_timing();
void set_kernel_timing(hipEvent_t start, hipEvent_t stop);

// Launches `k`, attaching this thread's pending timing events, if any, to
// the dispatch itself, so they bracket the kernel's execution and not the
// queue's dispatch latency.
// `lds` bytes of dynamic LDS are allocated per workgroup on top of the
// kernel's static LDS.
template <typename... P, typename... A>
inline void launch_lds(void (*k)(P...), dim3 grid, dim3 block, size_t lds, hipStream_t s, A... args)
{
    const kernel_timing t = take_kernel_timing();
    if (t.start || t.stop)
        hipExtLaunchKernelGGL(k, grid, block, lds, s, t.start, t.stop, 0, static_cast<P>(args)...);
    else
        k<<<grid, block, lds, s>>>(static_cast<P>(args)...);
}

template <typename... P, typename... A>
inline void launch(void (*k)(P...), dim3 grid, dim3 block, hipStream_t s, A... args)
{
    launch_lds(k, grid, block, 0, s, args...);
}

}  // namespace ss

namespace ss {
// two fp32 values rounded to bf16 (nearest, ties to even; inputs finite),
// packed low then high
__device__ __forceinline__ uint32_t pack_bf16_rne(float a, float b)
{
    uint32_t x = __float_as_uint(a), y = __float_as_uint(b);
    x += 0x7FFFu + ((x >> 16) & 1u);
    y += 0x7FFFu + ((y >> 16) & 1u);
    return (x >> 16) | (y & 0xFFFF0000u);
}

// fp64 -> fp32 rounded to odd: truncated toward zero, with the lowest
// significand bit set if anything was cut off.  fp32 keeps 16 more
// significand bits than bf16 (at every exponent, subnormals included), so
// rounding this value to bf16, nearest-even, gives the bf16 nearest to the
// fp64 value: one rounding, no double-rounding error.
__device__ __forceinline__ float f64_to_f32_odd(double x)
{
    const float f = __double2float_rz(x);
    uint32_t u = __float_as_uint(f);
    if ((double)f != x) u |= 1u;
    return __uint_as_float(u);
}

// two finite fp64 values rounded once to bf16 (nearest, ties to even),
// packed low then high
__device__ __forceinline__ uint32_t pack_bf16_rne_f64(double a, double b)
{
    return pack_bf16_rne(f64_to_f32_odd(a), f64_to_f32_odd(b));
}
}  // namespace ss

// 8 x bf16 operand fragment of v_mfma_f32_16x16x32_bf16 and its fp32 accumulator.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

#define SS_CHECK_ARG(cond, ...)                                   \
    do {                                                          \
        if (!(cond)) return ss::fail(SS_ERR_INVALID_ARG, __VA_ARGS__); \
    } while (0)
#define SS_CHECK_SUPPORTED(cond, ...)                             \
    do {                                                          \
        if (!(cond)) return ss::fail(SS_ERR_UNSUPPORTED, __VA_ARGS__); \
    } while (0)
