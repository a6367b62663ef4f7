// GRU node update (Eq. 1's GRU, Cho et al. 2014 form) and its reverse on
// gfx950 matrix cores, with the gate nonlinearities fused into the GEMM
// epilogues.
//
// Layouts: a [n_pad][H] float, h / h_out [n_pad][H] dt, Wi and U [H][3H] dt
// (columns r | z | n), b [3H] float, saved [n_pad][3H] dt (r | z | n),
// da [H][n_pad] dt feature-major, dh [n_pad][H] float.
//
// k order ("accumulator-compatible"): inside a 32-wide feature step kk, lane
// group g holds features 32kk + 4g + {0,1,2,3} and 32kk + 16 + 4g + {0,1,2,3}.
// These are exactly the features a lane holds in the accumulator of the two
// 16-feature output tiles 2kk and 2kk+1 (rows 4g + j), for the same node
// (lane % 16).  So a gate computed in registers is already an operand
// fragment of the next product: (r*h) U_n in the forward and every product of
// the backward chain without any cross-lane exchange.
#include "device_common.h"
#include "gru_wave.h"
#include "kernels.h"

namespace ggnn {
namespace dev {

// Stage the transpose of a 32-column slice of a [H][3H] weight into LDS:
// dst[f * PW + i] = src[i * 3H + col0 + f], f < 32, i < H.
template <typename S, int H, int PW, int NT>
__device__ __forceinline__ void stage_wT(S* dst, const S* src, int col0, int tid) {
  constexpr int V = 16 / sizeof(S);
  constexpr int UPR = 32 / V;  // 16-byte units per row slice
  for (int lin = tid; lin < H * UPR; lin += NT) {
    int i = lin / UPR, f0 = (lin % UPR) * V;
    u32x4 v = *reinterpret_cast<const u32x4*>(src + (size_t)i * 3 * H + col0 + f0);
    const S* pv = reinterpret_cast<const S*>(&v);
#pragma unroll
    for (int x = 0; x < V; ++x) dst[(f0 + x) * PW + i] = pv[x];
  }
}

// ---------------------------------------------------------------------------
// Forward.  Workgroup: 16*WAVES nodes, wave w: 16 nodes (lane % 16), all
// features.  D[feature][node]: A operand = weight^T rows from LDS, B operand
// = a / h / r*h fragments held in registers.  Phase A computes the reset
// gate for all features (needed in full by (r*h) U_n), phase B the update
// gate, the candidate and the new state, 32 features at a time.
// ---------------------------------------------------------------------------
template <typename S, int H, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void gru_fwd_kernel(const float* __restrict__ a, const S* __restrict__ h,
                                                                 const S* __restrict__ Wi, const S* __restrict__ U,
                                                                 const float* __restrict__ b, S* __restrict__ h_out,
                                                                 S* __restrict__ saved, int n_pad) {
  constexpr int NT = WAVES * kWave;
  constexpr int V = 16 / sizeof(S);
  constexpr int PW = H + V;
  constexpr int KS = H / 32;
  __shared__ __attribute__((aligned(16))) S wt[4][32 * PW];

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int n0 = xcd_swizzle(blockIdx.x, gridDim.x) * (16 * WAVES) + 16 * wave;
  const bool valid = n0 < n_pad;
  const int node = n0 + q;

  // a is fp32; in bf16 mode it enters the matrix cores as hi + lo parts
  // (al holds the lo part), so a Wi keeps fp32-level accuracy.
  constexpr int NP = sizeof(S) == 2 ? 2 : 1;
  frag_t<S> af[NP][KS], hf[KS], rh[KS];
  if (valid) {
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const float* row = a + (size_t)node * H;
      f32x4 x = *reinterpret_cast<const f32x4*>(row + 32 * kk + 4 * g);
      f32x4 y = *reinterpret_cast<const f32x4*>(row + 32 * kk + 16 + 4 * g);
      float v[8] = {x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
      if constexpr (NP == 2) {
        split8(v, af[0][kk], af[NP - 1][kk]);
      } else {
        af[0][kk] = pack8<S>(v);
      }
      hf[kk] = rowfrag<S>(h + (size_t)node * H, kk, g);
    }
  }
  auto afrag = [&](const S* t, int p, int kk) __attribute__((always_inline)) {
    return load4x2(t + (16 * p + q) * PW + 32 * kk + 4 * g, t + (16 * p + q) * PW + 32 * kk + 16 + 4 * g);
  };

  // Phase A: r = sigmoid(a Wi_r + h U_r + b_r); keep r*h as operand fragments.
  for (int c = 0; c < KS; ++c) {
    __syncthreads();
    stage_wT<S, H, PW, NT>(wt[0], Wi, 32 * c, tid);
    stage_wT<S, H, PW, NT>(wt[1], U, 32 * c, tid);
    __syncthreads();
    if (!valid) continue;
    f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const frag_t<S> w0 = afrag(wt[0], p, kk);
#pragma unroll
        for (int part = 0; part < NP; ++part) mma(acc[p], w0, af[part][kk]);
        mma(acc[p], afrag(wt[1], p, kk), hf[kk]);
      }
    float rhv[8];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int f = 32 * c + 16 * p + 4 * g;
      float r[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        r[j] = sigmoidf_(acc[p][j] + b[f + j]);
        rhv[4 * p + j] = r[j] * static_cast<float>(hf[c][4 * p + j]);
      }
      if (saved) store4(saved + (size_t)node * 3 * H + f, r[0], r[1], r[2], r[3]);
    }
    rh[c] = pack8<S>(rhv);
  }
  // Phase B: z, n and the new state, 32 features at a time.
  for (int c = 0; c < KS; ++c) {
    __syncthreads();
    stage_wT<S, H, PW, NT>(wt[0], Wi, H + 32 * c, tid);
    stage_wT<S, H, PW, NT>(wt[1], U, H + 32 * c, tid);
    stage_wT<S, H, PW, NT>(wt[2], Wi, 2 * H + 32 * c, tid);
    stage_wT<S, H, PW, NT>(wt[3], U, 2 * H + 32 * c, tid);
    __syncthreads();
    if (!valid) continue;
    f32x4 az[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
    f32x4 an[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const frag_t<S> w0 = afrag(wt[0], p, kk), w2 = afrag(wt[2], p, kk);
#pragma unroll
        for (int part = 0; part < NP; ++part) {
          mma(az[p], w0, af[part][kk]);
          mma(an[p], w2, af[part][kk]);
        }
        mma(az[p], afrag(wt[1], p, kk), hf[kk]);
        mma(an[p], afrag(wt[3], p, kk), rh[kk]);
      }
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int f = 32 * c + 16 * p + 4 * g;
      float z[4], n[4], o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        z[j] = sigmoidf_(az[p][j] + b[H + f + j]);
        n[j] = tanhf_(an[p][j] + b[2 * H + f + j]);
        const float hv = static_cast<float>(hf[c][4 * p + j]);
        o[j] = z[j] * hv + (1.f - z[j]) * n[j];
      }
      store4(h_out + (size_t)node * H + f, o[0], o[1], o[2], o[3]);
      if (saved) {
        store4(saved + (size_t)node * 3 * H + H + f, z[0], z[1], z[2], z[3]);
        store4(saved + (size_t)node * 3 * H + 2 * H + f, n[0], n[1], n[2], n[3]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Backward, per node (wave w: 16 nodes, lane % 16 = node): gru_bwd_wave.
// For H <= 64 the weights are staged once per workgroup in LDS (plain
// copies: the reverse products read rows of Wi and U, contiguous in the gate
// dimension); larger H reads their fragments from global memory (cached).
// ---------------------------------------------------------------------------
template <typename S, int H, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void gru_bwd_kernel(const float* __restrict__ gin, const S* __restrict__ h,
                                                                 const S* __restrict__ saved, const S* __restrict__ Wi,
                                                                 const S* __restrict__ U, S* __restrict__ daT,
                                                                 float* __restrict__ dh, S* __restrict__ ghat,
                                                                 int n_pad) {
  constexpr int MTL = H / 16;
  constexpr int NT = WAVES * kWave;
  constexpr int V = 16 / sizeof(S);
  constexpr bool LDSW = H <= 64;                       // weights fit in LDS
  constexpr int WROW = 3 * H + V;                       // LDS row pitch of a staged weight
  __shared__ __attribute__((aligned(16))) S wl[LDSW ? 2 : 1][LDSW ? H * WROW : 1];

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int n0 = xcd_swizzle(blockIdx.x, gridDim.x) * (16 * WAVES) + 16 * wave;
  const bool valid = n0 < n_pad;
  const int node = n0 + q;

  if constexpr (LDSW) {
    for (int lin = tid; lin < H * (3 * H / V); lin += NT) {
      const int r = lin / (3 * H / V), c = (lin % (3 * H / V)) * V;
      *reinterpret_cast<u32x4*>(&wl[0][r * WROW + c]) = *reinterpret_cast<const u32x4*>(Wi + (size_t)r * 3 * H + c);
      *reinterpret_cast<u32x4*>(&wl[1][r * WROW + c]) = *reinterpret_cast<const u32x4*>(U + (size_t)r * 3 * H + c);
    }
    __syncthreads();
  }
  if (!valid) return;   // no barrier follows
  f32x4 gg[MTL];
#pragma unroll
  for (int m = 0; m < MTL; ++m) gg[m] = *reinterpret_cast<const f32x4*>(gin + (size_t)node * H + 16 * m + 4 * g);
  if constexpr (LDSW) {
    gru_bwd_wave<S, H, WROW>(gg, n0, q, g, h, saved, &wl[0][0], &wl[1][0], daT, n_pad, dh, ghat);
  } else {
    gru_bwd_wave<S, H, 3 * H>(gg, n0, q, g, h, saved, Wi, U, daT, n_pad, dh, ghat);
  }
}

// ---------------------------------------------------------------------------
// Weight gradients of the GRU over one split of the rows k:
//   P[split][0][i][c] = sum_k a[k][i] G^[k][c]          (dWi)
//   P[split][1][i][c] = sum_k x_c[k][i] G^[k][c]        (dU)
// with x_c = h for the r and z columns and r*h for the n columns, and
//   Pb[split][c] = sum_k G^[k][c]                       (db).
// The rows are the nodes of one step (K = n_pad) or of all T steps at once
// (K = T * n_pad: a, h, saved and G^ stacked over t).  Tile TI x TI
// (TI = min(H, 64)); both operands are node-major, staged in LDS and read
// with a stride along k.  The tile index runs fastest over the logical
// workgroup index, so the tiles of one split share their rows in one L2.
// ---------------------------------------------------------------------------
template <typename S, int H>
__global__ __launch_bounds__((H < 64 ? H : 64) / 16 * kWave) void gru_wgrad_kernel(
    const float* __restrict__ a, const S* __restrict__ h, const S* __restrict__ saved, const S* __restrict__ ghat,
    float* __restrict__ P, float* __restrict__ Pb, long K, int rows_per_split) {
  constexpr int TI = H < 64 ? H : 64;
  constexpr int WAVES = TI / 16;
  constexpr int NT = WAVES * kWave;
  constexpr int KN = 64;
  constexpr int PX = TI + 4 / sizeof(S);
  constexpr int NTL = TI / 16;
  constexpr int TIN = H / TI, TOUT = 3 * H / TI;
  __shared__ __attribute__((aligned(16))) S ta[KN * PX];
  __shared__ __attribute__((aligned(16))) S tb[KN * PX];

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  int bid = xcd_swizzle(blockIdx.x, gridDim.x);
  const int to = bid % TOUT; bid /= TOUT;
  const int ti = bid % TIN; bid /= TIN;
  const int which = bid % 2;
  const int split = bid / 2;
  const long nlo = (long)split * rows_per_split;
  const long nhi = min(K, nlo + rows_per_split);
  const int col0 = to * TI;                      // gate column of this tile
  const bool rh_src = (which == 1 && col0 >= 2 * H);
  const bool do_bias = (which == 0 && ti == 0 && wave == 0);

  f32x4 acc[NTL];
  float bsum[NTL];
#pragma unroll
  for (int n = 0; n < NTL; ++n) {
    acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    bsum[n] = 0.f;
  }
  // Software pipeline: the next chunk's operands are loaded into registers
  // (a, h, r*h and G^ as four-element groups) while the current chunk is
  // multiplied.
  constexpr int TU = KN * TI / 4;
  constexpr int UN = (TU + NT - 1) / NT;
  f32x4 ar[UN];
  u32x2 gr[UN];     // four G^ elements (8 bytes for bf16; fp32 uses two of these per group below)
  f32x4 gf32[sizeof(S) == 4 ? UN : 1];
  auto load_chunk = [&](long c0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      const int lin = u * NT + tid;
      const int r = lin / (TI / 4), c = (lin % (TI / 4)) * 4;
      const long node = c0 + r;
      if ((TU % NT == 0 || lin < TU) && node < nhi) {
        const int fi = ti * TI + c;
        if (which == 0) {
          ar[u] = *reinterpret_cast<const f32x4*>(a + (size_t)node * H + fi);
        } else {
          f32x4 x = load4f(h + (size_t)node * H + fi);
          if (rh_src) {
            const f32x4 r4 = load4f(saved + (size_t)node * 3 * H + fi);
            x = f32x4{x.x * r4.x, x.y * r4.y, x.z * r4.z, x.w * r4.w};
          }
          ar[u] = x;
        }
        const S* gsrc = ghat + (size_t)node * 3 * H + col0 + c;
        if constexpr (sizeof(S) == 2) {
          gr[u] = *reinterpret_cast<const u32x2*>(gsrc);
        } else {
          gf32[u] = *reinterpret_cast<const f32x4*>(gsrc);
        }
      }
    }
  };
  if (nlo < nhi) load_chunk(nlo);
  for (long c0 = nlo; c0 < nhi; c0 += KN) {
    __syncthreads();
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      const int lin = u * NT + tid;
      const int r = lin / (TI / 4), c = (lin % (TI / 4)) * 4;
      if ((TU % NT == 0 || lin < TU) && c0 + r < nhi) {
        S* pa = &ta[r * PX + c];
        S* pb = &tb[r * PX + c];
        if constexpr (sizeof(S) == 2) {
          // rows are 4-byte aligned: write as two 32-bit words
          const uint32_t lo = pk2(ar[u].x, ar[u].y);
          const uint32_t hi = pk2(ar[u].z, ar[u].w);
          reinterpret_cast<uint32_t*>(pa)[0] = lo;
          reinterpret_cast<uint32_t*>(pa)[1] = hi;
          reinterpret_cast<uint32_t*>(pb)[0] = gr[u].x;
          reinterpret_cast<uint32_t*>(pb)[1] = gr[u].y;
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            pa[j] = from_f<S>(ar[u][j]);
            pb[j] = from_f<S>(gf32[sizeof(S) == 4 ? u : 0][j]);
          }
        }
      }
    }
    __syncthreads();
    if (c0 + KN < nhi) load_chunk(c0 + KN);
#pragma unroll
    for (int kk = 0; kk < KN / 32; ++kk) {
      if (c0 + 32 * kk >= nhi) break;
      frag_t<S> afr = load8_strided(&ta[(32 * kk + 8 * g) * PX + 16 * wave + q], PX);
#pragma unroll
      for (int n = 0; n < NTL; ++n) {
        frag_t<S> bf = load8_strided(&tb[(32 * kk + 8 * g) * PX + 16 * n + q], PX);
        mma(acc[n], afr, bf);
        if (do_bias) {
#pragma unroll
          for (int x = 0; x < 8; ++x) bsum[n] += static_cast<float>(bf[x]);
        }
      }
    }
  }
  float* out = P + ((size_t)split * 2 + which) * H * 3 * H;
#pragma unroll
  for (int n = 0; n < NTL; ++n) {
    const int c = col0 + 16 * n + q;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      out[(size_t)(ti * TI + 16 * wave + 4 * g + j) * 3 * H + c] = acc[n][j];
    }
  }
  if (do_bias) {
#pragma unroll
    for (int n = 0; n < NTL; ++n) {
      float v = bsum[n];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g == 0) Pb[(size_t)split * 3 * H + col0 + 16 * n + q] = v;
    }
  }
}

}  // namespace dev

namespace {
// Row split of the weight-gradient contraction (same policy as the message
// transform's): about 2048 workgroups, splits of at least GGNN_WGRAD_MIN_ROWS
// rows, a multiple of 64.
#ifndef GGNN_WGRAD_MIN_ROWS
#define GGNN_WGRAD_MIN_ROWS 1024
#endif
struct Split {
  int nsplit, per;
};
Split gru_split(long K, int H) {
  const long TI = H < 64 ? H : 64;
  const long tiles = 2 * (H / TI) * (3 * H / TI);
  const long want = (2048 + tiles - 1) / tiles;
  long per = ((K + want - 1) / want + 63) / 64 * 64;
  if (per < GGNN_WGRAD_MIN_ROWS) per = GGNN_WGRAD_MIN_ROWS;
  return {(int)((K + per - 1) / per), (int)per};
}

template <typename S, int H>
hipError_t gru_fwd_h(int n_pad, const float* a, const void* h, const void* Wi, const void* U, const float* b,
                     void* h_out, void* saved, hipStream_t st) {
  constexpr int WAVES = 4;
  hipLaunchKernelGGL((dev::gru_fwd_kernel<S, H, WAVES>), dim3((n_pad + 16 * WAVES - 1) / (16 * WAVES)),
                     dim3(WAVES * 64), 0, st, a, static_cast<const S*>(h), static_cast<const S*>(Wi),
                     static_cast<const S*>(U), b, static_cast<S*>(h_out), static_cast<S*>(saved), n_pad);
  return hipGetLastError();
}

template <typename S, int H>
hipError_t gru_bwd_nodes_h(int n_pad, const float* dh_out, const void* h, const void* saved, const void* Wi,
                           const void* U, void* da, float* dh, void* ghat, hipStream_t st) {
  constexpr int WAVES = 4;
  hipLaunchKernelGGL((dev::gru_bwd_kernel<S, H, WAVES>), dim3((n_pad + 16 * WAVES - 1) / (16 * WAVES)),
                     dim3(WAVES * 64), 0, st, dh_out, static_cast<const S*>(h), static_cast<const S*>(saved),
                     static_cast<const S*>(Wi), static_cast<const S*>(U), static_cast<S*>(da), dh,
                     static_cast<S*>(ghat), n_pad);
  return hipGetLastError();
}

template <typename S, int H>
hipError_t gru_wgrad_h(long K, const float* a, const void* h, const void* saved, const void* ghat, float* dWi,
                       float* dU, float* db, void* ws, hipStream_t st) {
  constexpr int TI = H < 64 ? H : 64;
  Split sp = gru_split(K, H);
  float* P = static_cast<float*>(ws);
  float* Pb = P + (size_t)sp.nsplit * 2 * H * 3 * H;
  const int blocks = sp.nsplit * 2 * (H / TI) * (3 * H / TI);
  hipLaunchKernelGGL((dev::gru_wgrad_kernel<S, H>), dim3(blocks), dim3(TI / 16 * 64), 0, st, a,
                     static_cast<const S*>(h), static_cast<const S*>(saved), static_cast<const S*>(ghat), P, Pb, K,
                     sp.per);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const long slice = 2L * H * 3 * H;  // partials are [split][which][H][3H]
  err = launch_reduce_partials(P, dWi, sp.nsplit, H * 3 * H, slice, st);
  if (err != hipSuccess) return err;
  err = launch_reduce_partials(P + (size_t)H * 3 * H, dU, sp.nsplit, H * 3 * H, slice, st);
  if (err != hipSuccess) return err;
  return launch_reduce_partials(Pb, db, sp.nsplit, 3 * H, 3L * H, st);
}

#define GGNN_GRU_SWITCH(CALL)                  \
  switch (H) {                                 \
    case 32: { constexpr int HH = 32; CALL; }  \
    case 64: { constexpr int HH = 64; CALL; }  \
    case 128: { constexpr int HH = 128; CALL; } \
    case 256: { constexpr int HH = 256; CALL; } \
  }                                            \
  return hipErrorInvalidValue;

template <typename S>
hipError_t gru_fwd_t(int n_pad, int H, const float* a, const void* h, const void* Wi, const void* U, const float* b,
                     void* h_out, void* saved, hipStream_t st) {
  GGNN_GRU_SWITCH(return (gru_fwd_h<S, HH>(n_pad, a, h, Wi, U, b, h_out, saved, st)))
}
template <typename S>
hipError_t gru_bwd_nodes_t(int n_pad, int H, const float* dh_out, const void* h, const void* saved, const void* Wi,
                           const void* U, void* da, float* dh, void* ghat, hipStream_t st) {
  GGNN_GRU_SWITCH(return (gru_bwd_nodes_h<S, HH>(n_pad, dh_out, h, saved, Wi, U, da, dh, ghat, st)))
}
template <typename S>
hipError_t gru_wgrad_t(long K, int H, const float* a, const void* h, const void* saved, const void* ghat, float* dWi,
                       float* dU, float* db, void* ws, hipStream_t st) {
  GGNN_GRU_SWITCH(return (gru_wgrad_h<S, HH>(K, a, h, saved, ghat, dWi, dU, db, ws, st)))
}
#undef GGNN_GRU_SWITCH
}  // namespace

#if GGNN_DT_BF16   // dtype-independent helpers: built once
size_t ghat_bytes(int dt, long rows, int H) {
  size_t b = (size_t)rows * 3 * H * (dt == GGNN_BF16 ? 2 : 4);
  return (b + 255) / 256 * 256;
}

size_t gru_wgrad_workspace(long K, int H) {
  Split sp = gru_split(K, H);
  return ((size_t)sp.nsplit * 2 * H * 3 * H + (size_t)sp.nsplit * 3 * H) * sizeof(float);
}

size_t gru_bwd_workspace(int dt, int n_pad, int H) {
  return ghat_bytes(dt, n_pad, H) + gru_wgrad_workspace(n_pad, H);
}

hipError_t launch_gru_bwd(int dt, int n_pad, int H, const float* dh_out, const float* a, const void* h,
                          const void* saved, const void* Wi, const void* U, void* da, float* dh, float* dWi,
                          float* dU, float* db, void* ws, hipStream_t st) {
  void* ghat = ws;
  void* part = static_cast<char*>(ws) + ghat_bytes(dt, n_pad, H);
  hipError_t err = launch_gru_bwd_nodes(dt, n_pad, H, dh_out, h, saved, Wi, U, da, dh, ghat, st);
  if (err != hipSuccess) return err;
  return launch_gru_wgrad(dt, n_pad, H, a, h, saved, ghat, dWi, dU, db, part, st);
}
#endif

namespace GGNN_IMPL_NS {
hipError_t launch_gru_fwd(int n_pad, int H, const float* a, const void* h, const void* Wi, const void* U,
                          const float* b, void* h_out, void* saved, hipStream_t st) {
  return gru_fwd_t<dev::dt_t>(n_pad, H, a, h, Wi, U, b, h_out, saved, st);
}

hipError_t launch_gru_bwd_nodes(int n_pad, int H, const float* dh_out, const void* h, const void* saved,
                                const void* Wi, const void* U, void* da, float* dh, void* ghat, hipStream_t st) {
  return gru_bwd_nodes_t<dev::dt_t>(n_pad, H, dh_out, h, saved, Wi, U, da, dh, ghat, st);
}

hipError_t launch_gru_wgrad(long K, int H, const float* a, const void* h, const void* saved, const void* ghat,
                            float* dWi, float* dU, float* db, void* ws, hipStream_t st) {
  return gru_wgrad_t<dev::dt_t>(K, H, a, h, saved, ghat, dWi, dU, db, ws, st);
}
}  // namespace GGNN_IMPL_NS

}  // namespace ggnn
