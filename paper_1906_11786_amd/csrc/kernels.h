// Launchers of the gfx950 kernels, one per device operation.  Arguments are
// validated by the C-ABI layer before these are called; each returns the
// hipGetLastError() of its launches.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

#include "../../include/ggnn.h"

namespace ggnn {

hipError_t launch_banded_fwd(int dt, int n_pad, int B, int H, int E, const void* band, const float* M, float* a,
                             hipStream_t st);
hipError_t launch_banded_bwd(int dt, int n_pad, int B, int H, int E, const void* band, const void* da, void* dM,
                             hipStream_t st);

// out[i] += sum_s part[s * stride + i], i < count, fixed summation order.
hipError_t launch_reduce_partials(const float* part, float* out, int nsplit, int count, long stride,
                                  hipStream_t st);

// 1-bit band: fused aggregate-first forward and transposed-band reverse.
hipError_t launch_step_fwd_bits(int dt, int n_pad, int B, int H, int E, const void* bits, const void* X,
                                const void* W, const float* bias, float* a, hipStream_t st);
hipError_t launch_banded_bwd_bits(int dt, int n_pad, int B, int H, int E, const void* bits_t, const void* da,
                                  void* dM, hipStream_t st);

hipError_t launch_transform_fwd(int dt, int n_pad, int H, int E, const void* X, const void* W, const float* bias,
                                float* M, hipStream_t st);
// Workspace layout of the transform backward (floats): partial dW then
// partial dbias, one slice per node split.
size_t transform_bwd_workspace(int dt, int n_pad, int H, int E);
// partial_mode 0: dW, dbias += this call's gradient (partials written, then
// reduced); 1: the call only adds its gradient into the partials of `ws`
// (cleared and reduced by the two functions below), for multi-step loops.
hipError_t launch_transform_bwd(int dt, int n_pad, int H, int E, const void* X, const void* W, const void* dM,
                                const float* dX_in, float* dX_out, float* dW, float* dbias, void* ws,
                                hipStream_t st, int partial_mode = 0);
hipError_t launch_transform_bwd_partials_clear(int dt, int n_pad, int H, int E, void* ws, hipStream_t st);
hipError_t launch_transform_bwd_partials_reduce(int dt, int n_pad, int H, int E, float* dW, float* dbias, void* ws,
                                                hipStream_t st);
hipError_t launch_fill_zero(float* p, size_t count, hipStream_t st);

hipError_t launch_gru_fwd(int dt, int n_pad, int H, const float* a, const void* h, const void* Wi, const void* U,
                          const float* b, void* h_out, void* saved, hipStream_t st);
size_t gru_bwd_workspace(int dt, int n_pad, int H);
hipError_t launch_gru_bwd(int dt, int n_pad, int H, const float* dh_out, const float* a, const void* h,
                          const void* saved, const void* Wi, const void* U, void* da, float* dh, float* dWi,
                          float* dU, float* db, void* ws, hipStream_t st, int partial_mode = 0);
hipError_t launch_gru_bwd_partials_clear(int dt, int n_pad, int H, void* ws, hipStream_t st);
hipError_t launch_gru_bwd_partials_reduce(int dt, int n_pad, int H, float* dWi, float* dU, float* db, void* ws,
                                          hipStream_t st);

}  // namespace ggnn
