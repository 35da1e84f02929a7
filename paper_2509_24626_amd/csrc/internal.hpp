// Internal helpers shared by the library's translation units: error
// reporting across the C ABI and the bf16 vector types of the gfx950 MFMA
// builtins.  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>

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
