// Readout, loss and parameter update: the steps that close one training
// iteration after T steps of propagation.
//
//  * readout (Background, "Variable misuse"): a learned linear map R^H -> R on
//    the final embeddings of each graph's candidate nodes gives one logit per
//    candidate;
//  * loss: softmax over each graph's candidates, cross-entropy of the correct
//    one, mean over the graphs of the supergraph;
//  * update (Appendix, "Optimization"): the Momentum optimizer, optionally
//    Nesterov, with L2 weight decay, on float32 master parameters; the
//    compute-dtype copy the propagation reads is rewritten in the same pass.
//
// Candidate lists are CSR-like: graph g owns candidates cand_ptr[g] ..
// cand_ptr[g+1]-1, candidate c is node cand_node[c], target[g] the index of
// the correct candidate within the graph's list.
#include <math.h>

#include "device_common.h"
#include "kernels.h"

namespace ggnn {
namespace dev {

constexpr int kReadoutWaves = 4;   // graphs (forward) or candidates (reverse) per workgroup

// logit of candidate node `node`, identical on every lane: the lanes split
// the features, partial products are summed with an xor butterfly (each
// stage adds the same two values on both partner lanes, so all lanes end
// with the same bits).
template <typename S, int H>
__device__ __forceinline__ float cand_logit(const S* __restrict__ X, const float (&w)[(H + 63) / 64], int node,
                                            int lane, float b_out) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < (H + 63) / 64; ++i) {
    const int h = lane + 64 * i;
    if (h < H) s += to_f<S>(X[(size_t)node * H + h]) * w[i];
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
  return s + b_out;
}

// One wave per graph: logits, the graph's loss and d(mean loss)/d(logits).
// Two passes over the candidates (the second recomputes each logit with the
// same arithmetic): an online maximum and normaliser, then the gradients.
template <typename S, int H>
__global__ __launch_bounds__(kReadoutWaves * kWave) void readout_loss_kernel(
    const S* __restrict__ X, const float* __restrict__ w_out, const float* __restrict__ b_out,
    const int32_t* __restrict__ cand_node, const int32_t* __restrict__ cand_ptr, const int32_t* __restrict__ target,
    int n_graphs, float* __restrict__ logits, float* __restrict__ loss, float* __restrict__ dlogit) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int gi = blockIdx.x * kReadoutWaves + wave;
  if (gi >= n_graphs) return;   // no barriers in this kernel
  const int lo = cand_ptr[gi], hi = cand_ptr[gi + 1];
  const int t = target[gi];
  const float bo = *b_out;
  float w[(H + 63) / 64];
#pragma unroll
  for (int i = 0; i < (H + 63) / 64; ++i) w[i] = (lane + 64 * i < H) ? w_out[lane + 64 * i] : 0.f;
  if (hi <= lo) {
    if (lane == 0) loss[gi] = 0.f;
    return;
  }
  const float inv_g = 1.0f / static_cast<float>(n_graphs);
  float m = -INFINITY, s = 0.f, zt = NAN;
  for (int c = lo; c < hi; ++c) {
    const float z = cand_logit<S, H>(X, w, cand_node[c], lane, bo);
    if (lane == 0) logits[c] = z;
    if (c - lo == t) zt = z;
    const float mn = fmaxf(m, z);
    s = s * expf(m - mn) + expf(z - mn);
    m = mn;
  }
  if (lane == 0) loss[gi] = logf(s) + m - zt;   // NaN when target is outside [0, hi - lo)
  const float inv_s = 1.0f / s;
  for (int c = lo; c < hi; ++c) {
    const float z = cand_logit<S, H>(X, w, cand_node[c], lane, bo);
    const float p = expf(z - m) * inv_s;
    if (lane == 0) dlogit[c] = (p - (c - lo == t ? 1.f : 0.f)) * inv_g;
  }
}

// One wave per candidate: dX[cand_node[c]] = dlogit[c] * w_out (the rows of
// other nodes are cleared by a fill launched before this kernel).
template <int H>
__global__ __launch_bounds__(kReadoutWaves * kWave) void readout_dx_kernel(const float* __restrict__ w_out,
                                                                           const int32_t* __restrict__ cand_node,
                                                                           const float* __restrict__ dlogit,
                                                                           int n_cand, float* __restrict__ dX) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int c = blockIdx.x * kReadoutWaves + wave;
  if (c >= n_cand) return;
  const float d = dlogit[c];
  float* row = dX + (size_t)cand_node[c] * H;
#pragma unroll
  for (int i = 0; i < (H + 63) / 64; ++i) {
    const int h = lane + 64 * i;
    if (h < H) row[h] = d * w_out[h];
  }
}

// Per block of kReadoutCands candidates (in order): partial dw_out[h] =
// sum_c dlogit[c] X[cand_node[c]][h] and partial db_out = sum_c dlogit[c],
// written to part[blockIdx.x * (H + 1) + .] and summed by the fixed-order
// partial reduction.
constexpr int kReadoutCands = 64;
template <typename S, int H>
__global__ __launch_bounds__(256) void readout_wgrad_kernel(const S* __restrict__ X,
                                                            const int32_t* __restrict__ cand_node,
                                                            const float* __restrict__ dlogit, int n_cand,
                                                            float* __restrict__ part) {
  const int h = threadIdx.x;
  const int c0 = blockIdx.x * kReadoutCands;
  const int c1 = min(n_cand, c0 + kReadoutCands);
  float acc = 0.f, bacc = 0.f;
#pragma unroll 8
  for (int c = c0; c < c1; ++c) {
    const float d = dlogit[c];
    if (h < H) acc += d * to_f<S>(X[(size_t)cand_node[c] * H + h]);
    bacc += d;
  }
  if (h < H) part[(size_t)blockIdx.x * (H + 1) + h] = acc;
  if (h == 0) part[(size_t)blockIdx.x * (H + 1) + H] = bacc;
}

}  // namespace dev

namespace {
template <typename S, int H>
hipError_t readout_loss_h(int n_graphs, const void* X, const float* w_out, const float* b_out,
                          const int32_t* cand_node, const int32_t* cand_ptr, const int32_t* target, float* logits,
                          float* loss, float* dlogit, hipStream_t st) {
  const int blocks = (n_graphs + dev::kReadoutWaves - 1) / dev::kReadoutWaves;
  hipLaunchKernelGGL((dev::readout_loss_kernel<S, H>), dim3(blocks), dim3(dev::kReadoutWaves * 64), 0, st,
                     static_cast<const S*>(X), w_out, b_out, cand_node, cand_ptr, target, n_graphs, logits, loss,
                     dlogit);
  return hipGetLastError();
}

template <typename S, int H>
hipError_t readout_bwd_h(int n_pad, int n_cand, const void* X, const float* w_out, const int32_t* cand_node,
                         const float* dlogit, float* dX, float* dw_out, float* db_out, float* part, hipStream_t st) {
  hipError_t err = launch_fill_zero(dX, (size_t)n_pad * H, st);
  if (err != hipSuccess || n_cand == 0) return err;
  const int blocks = (n_cand + dev::kReadoutWaves - 1) / dev::kReadoutWaves;
  hipLaunchKernelGGL((dev::readout_dx_kernel<H>), dim3(blocks), dim3(dev::kReadoutWaves * 64), 0, st, w_out,
                     cand_node, dlogit, n_cand, dX);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int ns = (n_cand + dev::kReadoutCands - 1) / dev::kReadoutCands;
  hipLaunchKernelGGL((dev::readout_wgrad_kernel<S, H>), dim3(ns), dim3(256), 0, st, static_cast<const S*>(X),
                     cand_node, dlogit, n_cand, part);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  err = launch_reduce_partials(part, dw_out, ns, H, H + 1, st);
  if (err != hipSuccess) return err;
  return launch_reduce_partials(part + H, db_out, ns, 1, H + 1, st);
}
}  // namespace

namespace GGNN_IMPL_NS {
hipError_t launch_readout_loss(int H, int n_graphs, const void* X, const float* w_out, const float* b_out,
                               const int32_t* cand_node, const int32_t* cand_ptr, const int32_t* target,
                               float* logits, float* loss, float* dlogit, hipStream_t st) {
  using S = dev::dt_t;
  switch (H) {
    case 32: return readout_loss_h<S, 32>(n_graphs, X, w_out, b_out, cand_node, cand_ptr, target, logits, loss, dlogit, st);
    case 64: return readout_loss_h<S, 64>(n_graphs, X, w_out, b_out, cand_node, cand_ptr, target, logits, loss, dlogit, st);
    case 128: return readout_loss_h<S, 128>(n_graphs, X, w_out, b_out, cand_node, cand_ptr, target, logits, loss, dlogit, st);
    case 256: return readout_loss_h<S, 256>(n_graphs, X, w_out, b_out, cand_node, cand_ptr, target, logits, loss, dlogit, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_readout_bwd(int n_pad, int H, int n_cand, const void* X, const float* w_out,
                              const int32_t* cand_node, const float* dlogit, float* dX, float* dw_out, float* db_out,
                              void* ws, hipStream_t st) {
  using S = dev::dt_t;
  float* part = static_cast<float*>(ws);
  switch (H) {
    case 32: return readout_bwd_h<S, 32>(n_pad, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out, part, st);
    case 64: return readout_bwd_h<S, 64>(n_pad, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out, part, st);
    case 128: return readout_bwd_h<S, 128>(n_pad, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out, part, st);
    case 256: return readout_bwd_h<S, 256>(n_pad, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out, part, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace GGNN_IMPL_NS

#if GGNN_DT_BF16   // dtype-independent: built once
namespace dev {
// Momentum update of float32 master parameters, element-wise:
//   g = grad + wd * theta;  v = mu * v + g;  theta -= lr * (nesterov ? g + mu * v : v)
// and the compute copy (COPY: 0 none, 1 bf16, 2 float32) rewritten from theta.
template <int COPY>
__global__ __launch_bounds__(256) void sgd_momentum_kernel(long count, float* __restrict__ theta,
                                                           float* __restrict__ vel, const float* __restrict__ grad,
                                                           float lr, float mu, float wd, int nesterov,
                                                           void* __restrict__ copy) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (long)gridDim.x * blockDim.x) {
    const float th = theta[i];
    const float g = grad[i] + wd * th;
    const float v = mu * vel[i] + g;
    const float nt = th - lr * (nesterov ? g + mu * v : v);
    vel[i] = v;
    theta[i] = nt;
    if constexpr (COPY == 1) static_cast<bf16s*>(copy)[i] = f2bf(nt);
    if constexpr (COPY == 2) static_cast<float*>(copy)[i] = nt;
  }
}
}  // namespace dev

size_t readout_bwd_workspace(int H, int n_cand) {
  const size_t ns = (size_t)(n_cand + dev::kReadoutCands - 1) / dev::kReadoutCands;
  return (ns > 0 ? ns : 1) * (size_t)(H + 1) * sizeof(float);
}

hipError_t launch_sgd_momentum(long count, float* theta, float* vel, const float* grad, float lr, float mu, float wd,
                               int nesterov, int copy_dt, void* copy, hipStream_t st) {
  if (count == 0) return hipSuccess;
  long blocks = (count + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (copy == nullptr) {
    hipLaunchKernelGGL((dev::sgd_momentum_kernel<0>), dim3((unsigned)blocks), dim3(256), 0, st, count, theta, vel,
                       grad, lr, mu, wd, nesterov, copy);
  } else if (copy_dt == GGNN_BF16) {
    hipLaunchKernelGGL((dev::sgd_momentum_kernel<1>), dim3((unsigned)blocks), dim3(256), 0, st, count, theta, vel,
                       grad, lr, mu, wd, nesterov, copy);
  } else {
    hipLaunchKernelGGL((dev::sgd_momentum_kernel<2>), dim3((unsigned)blocks), dim3(256), 0, st, count, theta, vel,
                       grad, lr, mu, wd, nesterov, copy);
  }
  return hipGetLastError();
}
#endif

}  // namespace ggnn
