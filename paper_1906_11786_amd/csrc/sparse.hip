// Sparse propagation over an explicit edge list, for evaluation on every edge
// of graphs whose bandwidth exceeds the block size a model was trained with:
// the weights learned on the block band are the same parameters the sparse
// model uses, so they can be evaluated with messages passed along all edges
// (Experiments, "Training time to validation accuracy").
//
//   a[i] = sum_e ( sum_{j -> i of type e} X[j] ) W_e  (+ deg_e(i) b_e)
//
// in the operand order of Algorithm 1 (aggregate per type, then transform),
// the aggregate gathered exactly from the receiver-major lists of
// ggnn_sparse_csr.  One wave per 16 receivers: lane (q, g) gathers, for
// receiver q, features 32kk + 8g .. + 7 of every sender row (the four lanes of
// a receiver read whole rows together), sums them in float32, and the
// per-type transform runs on the matrix cores with the aggregate as the B
// operand (bf16 hi + lo in bf16 mode) and rows of W_e^T as the A operand.
#include "device_common.h"
#include "kernels.h"

namespace ggnn {
namespace dev {

constexpr int kSparseWaves = 4;

template <typename S, int H>
__global__ __launch_bounds__(kSparseWaves * kWave) void sparse_step_kernel(
    const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col, const S* __restrict__ X,
    const S* __restrict__ Wt, const float* __restrict__ bias, float* __restrict__ out, int n_pad, int E) {
  constexpr int HK = H / 32, MT = H / 16;
  constexpr int NP = sizeof(S) == 2 ? 2 : 1;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int q = lane % 16, g = lane / 16;
  const int n0 = (blockIdx.x * kSparseWaves + wave) * 16;
  if (n0 >= n_pad) return;   // no barriers in this kernel
  const int node = n0 + q;

  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int e = 0; e < E; ++e) {
    const int lo = row_ptr[(size_t)node * E + e], hi = row_ptr[(size_t)node * E + e + 1];
    float p[HK][8];
#pragma unroll
    for (int kk = 0; kk < HK; ++kk)
#pragma unroll
      for (int x = 0; x < 8; ++x) p[kk][x] = 0.f;
    for (int k = lo; k < hi; ++k) {
      const S* row = X + (size_t)col[k] * H + 8 * g;
#pragma unroll
      for (int kk = 0; kk < HK; ++kk) {
        const frag_t<S> v = load8(row + 32 * kk);
#pragma unroll
        for (int x = 0; x < 8; ++x) p[kk][x] += static_cast<float>(v[x]);
      }
    }
    frag_t<S> pf[NP][HK];
#pragma unroll
    for (int kk = 0; kk < HK; ++kk) {
      if constexpr (NP == 2) {
        split8(p[kk], pf[0][kk], pf[NP - 1][kk]);
      } else {
        pf[0][kk] = pack8<S>(p[kk]);
      }
    }
    const S* we = Wt + (size_t)e * H * H;
#pragma unroll
    for (int mo = 0; mo < MT; ++mo) {
#pragma unroll
      for (int kk = 0; kk < HK; ++kk) {
        const frag_t<S> wf = load8(we + (size_t)(16 * mo + q) * H + 32 * kk + 8 * g);
#pragma unroll
        for (int part = 0; part < NP; ++part) mma(acc[mo], wf, pf[part][kk]);
      }
    }
    if (bias != nullptr) {
      const float d = static_cast<float>(hi - lo);
#pragma unroll
      for (int mo = 0; mo < MT; ++mo) {
        const f32x4 b4 = *reinterpret_cast<const f32x4*>(bias + (size_t)e * H + 16 * mo + 4 * g);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[mo][j] += d * b4[j];
      }
    }
  }
  // acc[mo] = D[feature 16mo + 4g + j][receiver q]
#pragma unroll
  for (int mo = 0; mo < MT; ++mo)
    *reinterpret_cast<f32x4*>(out + (size_t)node * H + 16 * mo + 4 * g) = acc[mo];
}

}  // namespace dev

namespace GGNN_IMPL_NS {
hipError_t launch_sparse_step(int n_pad, int H, int E, const int32_t* row_ptr, const int32_t* col, const void* X,
                              const void* Wt, const float* bias, float* a, hipStream_t st) {
  using S = dev::dt_t;
  const int blocks = (n_pad / 16 + dev::kSparseWaves - 1) / dev::kSparseWaves;
#define GGNN_SPARSE(HH)                                                                                        \
  hipLaunchKernelGGL((dev::sparse_step_kernel<S, HH>), dim3(blocks), dim3(dev::kSparseWaves * 64), 0, st, row_ptr, \
                     col, static_cast<const S*>(X), static_cast<const S*>(Wt), bias, a, n_pad, E)
  switch (H) {
    case 32: GGNN_SPARSE(32); break;
    case 64: GGNN_SPARSE(64); break;
    case 128: GGNN_SPARSE(128); break;
    case 256: GGNN_SPARSE(256); break;
    default: return hipErrorInvalidValue;
  }
#undef GGNN_SPARSE
  return hipGetLastError();
}
}  // namespace GGNN_IMPL_NS

}  // namespace ggnn
