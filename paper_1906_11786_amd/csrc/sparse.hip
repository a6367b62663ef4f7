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
// ggnn_sparse_csr.  One workgroup per 16 receivers, its waves taking turns
// over the edge types: lane (q, g) gathers, for receiver q, features
// 32kk + 8g .. + 7 of every sender row (the four lanes of
// a receiver read whole rows together), sums them in float32, and the
// per-type transform runs on the matrix cores with the aggregate as the B
// operand (bf16 hi + lo in bf16 mode) and rows of W_e^T as the A operand.
#include "device_common.h"
#include "kernels.h"

namespace ggnn {
namespace dev {

// On small graphs (few groups of 16 receivers) the waves of a workgroup share
// 16 receivers and split the edge types among them (wave w takes types w,
// w + NW, ...), which multiplies the waves in flight by NW and shortens each
// wave's chain of dependent loads (list bounds, column index, sender row) by
// the same factor. Their partial results are added through LDS in wave
// order, so the output does not depend on timing. NW = 8 up to H = 64, 4
// above (the partials take NW * H * 64 bytes of LDS). Larger graphs give
// every SIMD several waves already: there NW = 1 (one wave walks all types).
template <int H>
constexpr int sparse_waves() { return H <= 64 ? 8 : 4; }
#ifndef GGNN_SPARSE_SPLIT_MAX_GROUPS
#define GGNN_SPARSE_SPLIT_MAX_GROUPS 2048
#endif

template <typename S, int H, int NW>
__global__ __launch_bounds__(NW * kWave) void sparse_step_kernel(
    const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col, const S* __restrict__ X,
    const S* __restrict__ Wt, const float* __restrict__ bias, float* __restrict__ out, int n_pad, int E) {
  constexpr int HK = H / 32, MT = H / 16;
  constexpr int NP = sizeof(S) == 2 ? 2 : 1;
  // partial results: red[wave][mo][lane], one f32x4 per lane and output tile
  __shared__ f32x4 red[NW > 1 ? NW : 1][NW > 1 ? MT : 1][kWave];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int q = lane % 16, g = lane / 16;
  const int n0 = blockIdx.x * 16;
  if (n0 >= n_pad) return;   // uniform over the workgroup, before its one barrier
  const int node = n0 + q;

  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Up to two of the wave's edge types per pass: their gathers are
  // independent, so both lists' loads are in flight together. Each list is
  // still walked in order, so every type's sum is formed as with one type at
  // a time. Above H = 64 a second set of partial sums costs occupancy.
  constexpr int NE = H <= 64 ? 2 : 1;
  for (int k0 = 0; wave + NW * k0 < E; k0 += NE) {
    // List bounds of the pass's types; a type index past E is clamped to the
    // node's last bound and so gets an empty list.
    int lo[NE], len[NE];
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      const int e = wave + NW * (k0 + i);
      const int a0 = e < E ? e : E, a1 = e + 1 < E ? e + 1 : E;
      lo[i] = row_ptr[(size_t)node * E + a0];
      len[i] = row_ptr[(size_t)node * E + a1] - lo[i];
    }
    float p[NE][HK][8];
#pragma unroll
    for (int i = 0; i < NE; ++i)
#pragma unroll
      for (int kk = 0; kk < HK; ++kk)
#pragma unroll
        for (int x = 0; x < 8; ++x) p[i][kk][x] = 0.f;
    int steps = len[0];
#pragma unroll
    for (int i = 1; i < NE; ++i) steps = len[i] > steps ? len[i] : steps;
    // Every list's loads are issued before any sum is formed, so the chains
    // of the types overlap, and nothing branches on which lists are
    // exhausted. A lane inside the loop has a non-empty list, so col[0]
    // exists; it stands in for an exhausted list (it names a valid sender)
    // and the values it brings are dropped.
    for (int j = 0; j < steps; ++j) {
      int c[NE];
#pragma unroll
      for (int i = 0; i < NE; ++i) c[i] = col[j < len[i] ? lo[i] + j : 0];
      frag_t<S> v[NE][HK];
#pragma unroll
      for (int i = 0; i < NE; ++i) {
        const S* row = X + (size_t)c[i] * H + 8 * g;
#pragma unroll
        for (int kk = 0; kk < HK; ++kk) v[i][kk] = load8(row + 32 * kk);
      }
#pragma unroll
      for (int i = 0; i < NE; ++i) {
        const bool live = j < len[i];
#pragma unroll
        for (int kk = 0; kk < HK; ++kk)
#pragma unroll
          for (int x = 0; x < 8; ++x) p[i][kk][x] += live ? static_cast<float>(v[i][kk][x]) : 0.f;
      }
    }
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      const int e = wave + NW * (k0 + i);
      if (e >= E) break;
      frag_t<S> pf[NP][HK];
#pragma unroll
      for (int kk = 0; kk < HK; ++kk) {
        if constexpr (NP == 2) {
          split8(p[i][kk], pf[0][kk], pf[NP - 1][kk]);
        } else {
          pf[0][kk] = pack8<S>(p[i][kk]);
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
        const float d = static_cast<float>(len[i]);
#pragma unroll
        for (int mo = 0; mo < MT; ++mo) {
          const f32x4 b4 = *reinterpret_cast<const f32x4*>(bias + (size_t)e * H + 16 * mo + 4 * g);
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[mo][j] += d * b4[j];
        }
      }
    }
  }
  if constexpr (NW == 1) {
    // acc[mo] = D[feature 16mo + 4g + j][receiver q]
#pragma unroll
    for (int mo = 0; mo < MT; ++mo)
      *reinterpret_cast<f32x4*>(out + (size_t)node * H + 16 * mo + 4 * g) = acc[mo];
    return;
  }
#pragma unroll
  for (int mo = 0; mo < MT; ++mo) red[wave][mo][lane] = acc[mo];
  __syncthreads();
  // acc[mo] = D[feature 16mo + 4g + j][receiver q]; wave w writes the tiles
  // mo = w, w + NW, ..., each the sum of the waves' parts in order.
  for (int mo = wave; mo < MT; mo += NW) {
    f32x4 sum = red[0][mo][lane];
#pragma unroll
    for (int w = 1; w < NW; ++w) {
      const f32x4 t = red[w][mo][lane];
#pragma unroll
      for (int j = 0; j < 4; ++j) sum[j] += t[j];
    }
    *reinterpret_cast<f32x4*>(out + (size_t)node * H + 16 * mo + 4 * g) = sum;
  }
}

}  // namespace dev

namespace GGNN_IMPL_NS {
hipError_t launch_sparse_step(int n_pad, int H, int E, const int32_t* row_ptr, const int32_t* col, const void* X,
                              const void* Wt, const float* bias, float* a, hipStream_t st) {
  using S = dev::dt_t;
  const int blocks = n_pad / 16;   // n_pad is a multiple of 32 (checked by the caller)
  const bool split = blocks <= GGNN_SPARSE_SPLIT_MAX_GROUPS;
#define GGNN_SPARSE_NW(HH, NWV)                                                                               \
  hipLaunchKernelGGL((dev::sparse_step_kernel<S, HH, NWV>), dim3(blocks), dim3((NWV) * 64), 0, st, row_ptr, col, \
                     static_cast<const S*>(X), static_cast<const S*>(Wt), bias, a, n_pad, E)
#define GGNN_SPARSE(HH)                                  \
  if (split) {                                           \
    GGNN_SPARSE_NW(HH, dev::sparse_waves<HH>());         \
  } else {                                               \
    GGNN_SPARSE_NW(HH, 1);                               \
  }
  switch (H) {
    case 32: GGNN_SPARSE(32); break;
    case 64: GGNN_SPARSE(64); break;
    case 128: GGNN_SPARSE(128); break;
    case 256: GGNN_SPARSE(256); break;
    default: return hipErrorInvalidValue;
  }
#undef GGNN_SPARSE
#undef GGNN_SPARSE_NW
  return hipGetLastError();
}
}  // namespace GGNN_IMPL_NS

}  // namespace ggnn
