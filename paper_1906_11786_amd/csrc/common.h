// Internal helpers shared by the host and device translation units of the
// library: thread-local error text and argument checks.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/ggnn.h"

namespace ggnn {

// Records a formatted message for ggnn_last_error() and returns `st`.
ggnn_status fail(ggnn_status st, const char* fmt, ...);
void clear_error();

inline bool supported_B(int32_t B) { return B == 32 || B == 64 || B == 128 || B == 256 || B == 512; }
inline bool supported_H(int32_t H) { return H == 32 || H == 64 || H == 128 || H == 256; }
inline bool supported_dtype(int32_t dt) { return dt == GGNN_F32 || dt == GGNN_BF16; }
inline size_t dtype_bytes(int32_t dt) { return dt == GGNN_BF16 ? 2 : 4; }

}  // namespace ggnn

#define GGNN_CHECK_ARG(cond, ...)                                   \
  do {                                                              \
    if (!(cond)) return ::ggnn::fail(GGNN_ERR_INVALID_ARG, __VA_ARGS__); \
  } while (0)
