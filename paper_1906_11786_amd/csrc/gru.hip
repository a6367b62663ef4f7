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
  __shared__ __attribute__((aligned(16))) S wl[LDSW ? 2 * 3 * H * H : 1];   // Wi, U in fragment order

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int n0 = xcd_swizzle(blockIdx.x, gridDim.x) * (16 * WAVES) + 16 * wave;
  const bool valid = n0 < n_pad;
  const int node = n0 + q;

  // The node's inputs are loaded first, so that they are in flight while the
  // weights are staged (all of a thread's weight loads issued before its
  // LDS writes).
  f32x4 gg[MTL];
  GruBwdIn<S, H> in;
  if (valid) {
#pragma unroll
    for (int m = 0; m < MTL; ++m) gg[m] = *reinterpret_cast<const f32x4*>(gin + (size_t)node * H + 16 * m + 4 * g);
    in.load(saved, h, node, g);
  }
  if constexpr (LDSW) {
    constexpr int UNITS = 2 * H * (3 * H / V), ITS = (UNITS + NT - 1) / NT;
    u32x4 w[ITS];
#pragma unroll
    for (int it = 0; it < ITS; ++it) {
      const int lin = it * NT + tid;
      if (lin < UNITS) {
        const int mat = lin / (H * (3 * H / V)), rem = lin % (H * (3 * H / V));
        const int r = rem / (3 * H / V), c = (rem % (3 * H / V)) * V;
        w[it] = *reinterpret_cast<const u32x4*>((mat ? U : Wi) + (size_t)r * 3 * H + c);
      }
    }
#pragma unroll
    for (int it = 0; it < ITS; ++it) {
      const int lin = it * NT + tid;
      if (lin < UNITS) {
        const int mat = lin / (H * (3 * H / V)), rem = lin % (H * (3 * H / V));
        const int r = rem / (3 * H / V), c = (rem % (3 * H / V)) * V;
        const S* pw = reinterpret_cast<const S*>(&w[it]);
#pragma unroll
        for (int i = 0; i < V; i += 4)
          put4<S>(wl, gru_rev_idx<S, H>(mat, r / 16, (c + i) / H, ((c + i) % H) / 32), r % 16, (c + i) % H, pw + i);
      }
    }
    __syncthreads();
  }
  if (!valid) return;   // no barrier follows
  if constexpr (LDSW) {
    auto wf = [&](int which, int row, int gate, int kk) __attribute__((always_inline)) {
      return load_fragi<S>(wl, gru_rev_idx<S, H>(which, row / 16, gate, kk), lane);
    };
    gru_bwd_wave<S, H>(gg, n0, q, g, in, wf, daT, n_pad, dh, ghat);
  } else {
    auto wf = [&](int which, int row, int gate, int kk) __attribute__((always_inline)) {
      return rowfrag<S>((which ? U : Wi) + (size_t)row * 3 * H + gate * H, kk, g);
    };
    gru_bwd_wave<S, H>(gg, n0, q, g, in, wf, daT, n_pad, dh, ghat);
  }
}

// ---------------------------------------------------------------------------
// Weight staging of the large-H kernels.  Both stream Wi and U through LDS in
// stages kept in fragment order; a staging unit is one lane vector (eight
// elements, 16 bytes) of one fragment, and unit `lin` of a stage lands at
// element 8 lin of the stage buffer.  The units are gathered from the
// row-major weights, or copied from a packed array that holds every stage's
// units back to back (GruPack), which turns staging into contiguous 16-byte
// loads.
//   forward stage s < NC:  16 columns 16s.. of gate r, blocks {Wi, U};
//   forward stage s >= NC: 16 columns of gates z and n, {Wi_z, U_z, Wi_n, U_n};
//     block unit (kk, lane (qq, gg)): column qq of the tile at input rows
//     32kk + 4gg + {0..3}, 32kk + 16 + 4gg + {0..3};
//   reverse pass 1, block m: U rows 16m.., gate n, fragments kk;
//   reverse pass 2, block m: Wi rows 16m.., gates r, z, n, then U gates r, z;
//     unit (gate, kk, lane (qq, gg)): row 16m + qq at gate columns
//     32kk + 4gg + {0..3}, 32kk + 16 + 4gg + {0..3}.
// ---------------------------------------------------------------------------
template <int H>
struct GruPack {
  static constexpr int KS = H / 32, NC = H / 16, FRU = KS * 64;   // units per 16-wide block
  static constexpr int UNITS = 6 * NC * FRU;                      // units per region (6 H^2 / 8)
  // first unit of forward stage s / reverse block m of pass p
  __host__ __device__ static constexpr int fwd_stage(int s) {
    return s < NC ? 2 * s * FRU : 2 * NC * FRU + 4 * (s - NC) * FRU;
  }
  __host__ __device__ static constexpr int rev_stage(int p, int m) {
    return p == 1 ? m * FRU : NC * FRU + 5 * m * FRU;
  }
};

template <typename S, int H>
__device__ __forceinline__ u32x4 gru_fwd_unit(const S* __restrict__ Wi, const S* __restrict__ U, int s, int lin) {
  constexpr int NC = H / 16, UPB = GruPack<H>::FRU;
  const int blk = lin / UPB, rem = lin % UPB;
  const int kk = rem / 64, l = rem % 64, qq = l % 16, gg = l / 16;
  const int t16 = s < NC ? s : s - NC;
  const int gate = s < NC ? 0 : 1 + blk / 2;
  const S* src = ((blk % 2) ? U : Wi) + gate * H + 16 * t16 + qq;
  const int r0 = 32 * kk + 4 * gg;
  uint32_t w[4];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    w[j] = static_cast<uint32_t>(src[(size_t)(r0 + 2 * j) * 3 * H]) |
           (static_cast<uint32_t>(src[(size_t)(r0 + 2 * j + 1) * 3 * H]) << 16);
    w[2 + j] = static_cast<uint32_t>(src[(size_t)(r0 + 16 + 2 * j) * 3 * H]) |
               (static_cast<uint32_t>(src[(size_t)(r0 + 16 + 2 * j + 1) * 3 * H]) << 16);
  }
  return u32x4{w[0], w[1], w[2], w[3]};
}

template <typename S, int H>
__device__ __forceinline__ u32x4 gru_rev_unit(const S* __restrict__ Wi, const S* __restrict__ U, int pass, int m,
                                              int lin) {
  constexpr int KS = H / 32;
  const int frag = lin / 64, l = lin % 64, qq = l % 16, gg = l / 16;
  const S* mat;
  int gate, kk;
  if (pass == 1) {
    mat = U;
    gate = 2;
    kk = frag;
  } else if (frag < 3 * KS) {
    mat = Wi;
    gate = frag / KS;
    kk = frag % KS;
  } else {
    mat = U;
    gate = (frag - 3 * KS) / KS;
    kk = (frag - 3 * KS) % KS;
  }
  const S* p = mat + (size_t)(16 * m + qq) * 3 * H + gate * H + 32 * kk + 4 * gg;
  const u32x2 a = *reinterpret_cast<const u32x2*>(p);
  const u32x2 b = *reinterpret_cast<const u32x2*>(p + 16);
  return u32x4{a[0], a[1], b[0], b[1]};
}

// One thread per unit: forward region, then reverse region.
template <typename S, int H>
__global__ __launch_bounds__(256) void gru_pack_kernel(const S* __restrict__ Wi, const S* __restrict__ U,
                                                       S* __restrict__ out) {
  using P = GruPack<H>;
  const int u = blockIdx.x * 256 + threadIdx.x;
  if (u >= 2 * P::UNITS) return;
  u32x4 v;
  if (u < P::UNITS) {
    int s, lin;
    if (u < 2 * P::NC * P::FRU) {
      s = u / (2 * P::FRU);
      lin = u % (2 * P::FRU);
    } else {
      const int x = u - 2 * P::NC * P::FRU;
      s = P::NC + x / (4 * P::FRU);
      lin = x % (4 * P::FRU);
    }
    v = gru_fwd_unit<S, H>(Wi, U, s, lin);
  } else {
    const int x = u - P::UNITS;
    int pass, m, lin;
    if (x < P::NC * P::FRU) {
      pass = 1;
      m = x / P::FRU;
      lin = x % P::FRU;
    } else {
      const int y = x - P::NC * P::FRU;
      pass = 2;
      m = y / (5 * P::FRU);
      lin = y % (5 * P::FRU);
    }
    v = gru_rev_unit<S, H>(Wi, U, pass, m, lin);
  }
  *reinterpret_cast<u32x4*>(out + (size_t)u * 8) = v;
}


// ---------------------------------------------------------------------------
// Forward for large H (bf16, H >= 128), the arithmetic of gru_fwd_kernel
// with the weights shared through LDS: a workgroup of 8 waves (16 nodes
// each) streams Wi and U once per 128 nodes in stages of one 16-column gate
// tile, kept in fragment order, two stages per barrier and double buffered.
// Pass 1 (tiles of the r gate) forms r and keeps r*h as operand fragments;
// pass 2 (tiles of z and n) finishes the state.
// ---------------------------------------------------------------------------
template <typename S, int H, bool PK>
__global__ __launch_bounds__(512) void gru_fwd_big_kernel(const float* __restrict__ a, const S* __restrict__ h,
                                                          const S* __restrict__ Wi, const S* __restrict__ U,
                                                          const S* __restrict__ pk, const float* __restrict__ b,
                                                          S* __restrict__ h_out, S* __restrict__ saved, int n_pad) {
  static_assert(sizeof(S) == 2, "bf16 only");
  constexpr int NT = 512;
  constexpr int KS = H / 32, NC = H / 16;
  constexpr int FR = KS * 64 * 8;                  // elements of one (matrix, 16-column tile) block
  // Stages are staged in pairs (one barrier per two stages; NC is even, so a
  // pair never spans the two passes), double buffered: four stage buffers.
  constexpr int SS = 2;
  __shared__ __attribute__((aligned(16))) S lw[2 * SS][4 * FR];   // up to four blocks per stage

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int n0 = xcd_swizzle(blockIdx.x, gridDim.x) * 128 + 16 * wave;
  const bool valid = n0 < n_pad;
  const int node = n0 + q;

  // Stage s of 2 NC: s < NC is pass 1, tile s (Wi, U columns of gate r);
  // s >= NC is pass 2, tile s - NC (Wi, U columns of gates z and n); units
  // as gru_fwd_unit, from the packed forward region when PK.
  constexpr int UPB = KS * 64;                     // units per block
  constexpr int RMAX = (4 * UPB + NT - 1) / NT;
  u32x4 rr[SS][RMAX];
  auto load_stage = [&](int s, int j) __attribute__((always_inline)) {
    const int nblk = s < NC ? 2 : 4;
#pragma unroll
    for (int u = 0; u < RMAX; ++u) {
      const int lin = u * NT + tid;
      if (lin < nblk * UPB) {
        if constexpr (PK)
          rr[j][u] = *reinterpret_cast<const u32x4*>(pk + ((size_t)GruPack<H>::fwd_stage(s) + lin) * 8);
        else
          rr[j][u] = gru_fwd_unit<S, H>(Wi, U, s, lin);
      }
    }
  };
  auto store_stage = [&](int s, int j, int bf) __attribute__((always_inline)) {
    const int nblk = s < NC ? 2 : 4;
#pragma unroll
    for (int u = 0; u < RMAX; ++u) {
      const int lin = u * NT + tid;
      if (lin < nblk * UPB) *reinterpret_cast<u32x4*>(&lw[bf][lin * 8]) = rr[j][u];
    }
  };

  // Operand fragments of the 16 nodes (accumulator-compatible k order):
  // a as hi + lo, h, and later r*h.
  frag_t<S> af[2][KS], hf[KS], rh[KS];
  if (valid) {
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const float* row = a + (size_t)node * H;
      const f32x4 x = *reinterpret_cast<const f32x4*>(row + 32 * kk + 4 * g);
      const f32x4 y = *reinterpret_cast<const f32x4*>(row + 32 * kk + 16 + 4 * g);
      const float v[8] = {x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
      split8(v, af[0][kk], af[1][kk]);
      hf[kk] = rowfrag<S>(h + (size_t)node * H, kk, g);
    }
  }
  float rhv[8];
  static_assert(NC % SS == 0, "stage pairs must not span the two passes");
#pragma unroll
  for (int j = 0; j < SS; ++j) load_stage(j, j);
  auto compute = [&](int s, const S* L) __attribute__((always_inline)) {
    if (s < NC) {
      f32x4 ar = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const frag_t<S> w0 = load_fragi<S>(L, kk, lane);
        mma(ar, w0, af[0][kk]);
        mma(ar, w0, af[1][kk]);
        mma(ar, load_fragi<S>(L + FR, kk, lane), hf[kk]);
      }
      const int f = 16 * s + 4 * g;
      float r[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        r[j] = sigmoidf_(ar[j] + b[f + j]);
        rhv[4 * (s % 2) + j] = r[j] * static_cast<float>(hf[s / 2][4 * (s % 2) + j]);
      }
      if (saved) store4(saved + (size_t)node * 3 * H + f, r[0], r[1], r[2], r[3]);
      if (s % 2 == 1) rh[s / 2] = pack8<S>(rhv);
    } else {
      const int t16 = s - NC;
      f32x4 az = {0.f, 0.f, 0.f, 0.f}, an = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const frag_t<S> wz = load_fragi<S>(L, kk, lane), wn = load_fragi<S>(L + 2 * FR, kk, lane);
        mma(az, wz, af[0][kk]);
        mma(az, wz, af[1][kk]);
        mma(an, wn, af[0][kk]);
        mma(an, wn, af[1][kk]);
        mma(az, load_fragi<S>(L + FR, kk, lane), hf[kk]);
        mma(an, load_fragi<S>(L + 3 * FR, kk, lane), rh[kk]);
      }
      const int f = 16 * t16 + 4 * g;
      float z[4], nn[4], o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        z[j] = sigmoidf_(az[j] + b[H + f + j]);
        nn[j] = tanhf_(an[j] + b[2 * H + f + j]);
        const float hv = static_cast<float>(hf[t16 / 2][4 * (t16 % 2) + j]);
        o[j] = z[j] * hv + (1.f - z[j]) * nn[j];
      }
      store4(h_out + (size_t)node * H + f, o[0], o[1], o[2], o[3]);
      if (saved) {
        store4(saved + (size_t)node * 3 * H + H + f, z[0], z[1], z[2], z[3]);
        store4(saved + (size_t)node * 3 * H + 2 * H + f, nn[0], nn[1], nn[2], nn[3]);
      }
    }
  };
#pragma unroll
  for (int s0 = 0; s0 < 2 * NC; s0 += SS) {
    const int bf = ((s0 / SS) & 1) * SS;
#pragma unroll
    for (int j = 0; j < SS; ++j) store_stage(s0 + j, j, bf + j);
    __syncthreads();
    if (s0 + SS < 2 * NC) {
#pragma unroll
      for (int j = 0; j < SS; ++j) load_stage(s0 + SS + j, j);
    }
    if (!valid) continue;
#pragma unroll
    for (int j = 0; j < SS; ++j) compute(s0 + j, lw[bf + j]);
  }
}

// ---------------------------------------------------------------------------
// Backward for large H (bf16, H >= 128), the same arithmetic as
// gru_bwd_wave, with the weights shared through LDS: a workgroup of 8 waves
// (16 nodes each) streams the weights once per 128 nodes, in blocks of 16
// input features (rows of Wi and U) kept in fragment order and double
// buffered (the next block's loads are in flight during the current one).
//   pass 1: q' = n^ U_n^T, block m gives q' for input features 16m..16m+15,
//           hence r^ and the q' r term of dh for them;
//   pass 2: block n gives da for input features 16n..16n+15 (G^ Wi^T, all
//           three gates) and finishes dh for them (r^ U_r^T + z^ U_z^T).
// ---------------------------------------------------------------------------
template <typename S, int H, bool PK>
__global__ __launch_bounds__(512) void gru_bwd_big_kernel(const float* __restrict__ gin, const S* __restrict__ h,
                                                          const S* __restrict__ saved, const S* __restrict__ Wi,
                                                          const S* __restrict__ U, const S* __restrict__ pk,
                                                          S* __restrict__ daT,
                                                          float* __restrict__ dh, S* __restrict__ ghat, int n_pad) {
  static_assert(sizeof(S) == 2, "bf16 only");
  constexpr int NT = 512, V = 8;
  constexpr int KS = H / 32, MTL = H / 16;
  // LDS per buffer: pass 1 the n-gate part of a U block; pass 2 a Wi block
  // (three gates) and the r, z part of a U block, both in fragment order
  // (index gate * KS + kk within the block).
  constexpr int BLK_W = 3 * KS * 64 * 8, BLK_U = 2 * KS * 64 * 8;   // elements
  // Pass 1 reads all of U_n (MTL blocks) from one staging, without barriers
  // between blocks; pass 2's two block buffers then reuse the same LDS.
  constexpr int P1E = MTL * KS * 64 * 8;                               // elements of U_n's blocks
  constexpr int LDSE = P1E > 2 * (BLK_W + BLK_U) ? P1E : 2 * (BLK_W + BLK_U);
  __shared__ __attribute__((aligned(16))) S lds_all[LDSE];
  S (*lw)[BLK_W + BLK_U] = reinterpret_cast<S (*)[BLK_W + BLK_U]>(lds_all);

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int n0 = xcd_swizzle(blockIdx.x, gridDim.x) * 128 + 16 * wave;
  const bool valid = n0 < n_pad;
  const int node = n0 + q;

  // Staging of weight block m (rows 16m .. 16m + 15) into buffer b:
  // pass 1: U columns of gate n; pass 2: Wi all gates, U gates r, z; units as
  // gru_rev_unit, from the packed reverse region when PK.
  constexpr int U1 = KS * 64;                      // units, pass 1
  constexpr int U2 = 5 * KS * 64;                  // pass 2: 3 KS fragments of Wi, 2 KS of U
  constexpr int R2 = (U2 + NT - 1) / NT;
  u32x4 rr[R2];
  auto load_blk = [&](int pass, int m) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < R2; ++u) {
      const int lin = u * NT + tid;
      if (lin < (pass == 1 ? U1 : U2)) {
        if constexpr (PK)
          rr[u] = *reinterpret_cast<const u32x4*>(pk + ((size_t)GruPack<H>::rev_stage(pass, m) + lin) * 8);
        else
          rr[u] = gru_rev_unit<S, H>(Wi, U, pass, m, lin);
      }
    }
  };
  auto store_blk = [&](int pass, int b) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < R2; ++u) {
      const int lin = u * NT + tid;
      if (lin < (pass == 1 ? U1 : U2)) *reinterpret_cast<u32x4*>(&lw[b][lin * 8]) = rr[u];
    }
  };

  // Pass 1's weights (all blocks of U_n, gate n), staged in rounds of R2
  // units per thread; the first round's loads are in flight during phase 1.
  constexpr int P1U = MTL * U1;
  constexpr int P1R = (P1U + R2 * NT - 1) / (R2 * NT);
  auto load_p1 = [&](int round) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < R2; ++u) {
      const int lin = (round * R2 + u) * NT + tid;
      if (lin < P1U) {
        if constexpr (PK)
          rr[u] = *reinterpret_cast<const u32x4*>(pk + ((size_t)GruPack<H>::rev_stage(1, 0) + lin) * 8);
        else
          rr[u] = gru_rev_unit<S, H>(Wi, U, 1, lin / U1, lin % U1);
      }
    }
  };
  auto store_p1 = [&](int round) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < R2; ++u) {
      const int lin = (round * R2 + u) * NT + tid;
      if (lin < P1U) *reinterpret_cast<u32x4*>(&lds_all[lin * 8]) = rr[u];
    }
  };
  load_p1(0);

  // Phase 1 (elementwise, registers): n^, z^ as operand fragments, the
  // g' z term of dh, and G^'s z, n columns.
  frag_t<S> gf[3][KS];
  f32x4 dacc[MTL];
  const S* sv = saved + (size_t)node * 3 * H;
  S* gh = ghat + (size_t)node * 3 * H;
  if (valid) {
    float zv[8], nv[8];
    u32x2 zp[2], np[2], hp[2];   // tiles m, m + 1 of z, n, h (16-byte loads, load_tiles16)
#pragma unroll
    for (int m = 0; m < MTL; ++m) {
      const int f = 16 * m + 4 * g;
      const f32x4 gg = *reinterpret_cast<const f32x4*>(gin + (size_t)node * H + f);
      if (m % 2 == 0) {
        load_tiles16(sv + H + 16 * m, g, zp);
        load_tiles16(sv + 2 * H + 16 * m, g, np);
        load_tiles16(h + (size_t)node * H + 16 * m, g, hp);
      }
      const f32x4 z4 = unpack4(zp[m % 2]), n4 = unpack4(np[m % 2]);
      const f32x4 h4 = unpack4(hp[m % 2]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float dn = gg[j] * (1.f - z4[j]);
        const float dz = gg[j] * (h4[j] - n4[j]);
        dacc[m][j] = gg[j] * z4[j];
        nv[4 * (m % 2) + j] = dn * (1.f - n4[j] * n4[j]);
        zv[4 * (m % 2) + j] = dz * z4[j] * (1.f - z4[j]);
      }
      if (m % 2 == 1) {
        gf[2][m / 2] = pack8<S>(nv);
        gf[1][m / 2] = pack8<S>(zv);
        // G^'s z, n columns of tiles m - 1, m (the fragments hold them packed as bf16)
        const u32x4 pz = __builtin_bit_cast(u32x4, gf[1][m / 2]), pn = __builtin_bit_cast(u32x4, gf[2][m / 2]);
        store_tiles16(gh + H + 32 * (m / 2), u32x2{pz[0], pz[1]}, u32x2{pz[2], pz[3]}, g);
        store_tiles16(gh + 2 * H + 32 * (m / 2), u32x2{pn[0], pn[1]}, u32x2{pn[2], pn[3]}, g);
      }
    }
  }

#pragma unroll
  for (int round = 0; round < P1R; ++round) {
    store_p1(round);
    if (round + 1 < P1R) load_p1(round + 1);
  }
  __syncthreads();
  // Pass 2's first block, in flight during pass 1.
  load_blk(2, 0);

  // Pass 1: blocks m = 0 .. MTL-1 of U_n (unrolled: static register indices).
  float rv[8];
  u32x2 rp[2], hq[2];   // tiles m, m + 1 of r and h (16-byte loads)
#pragma unroll
  for (int m = 0; m < MTL; ++m) {
    if (valid) {
      if (m % 2 == 0) {
        load_tiles16(sv + 16 * m, g, rp);
        load_tiles16(h + (size_t)node * H + 16 * m, g, hq);
      }
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) mma(acc, load_fragi<S>(lds_all + m * U1 * 8, kk, lane), gf[2][kk]);
      const int f = 16 * m + 4 * g;
      const f32x4 r4 = unpack4(rp[m % 2]), h4 = unpack4(hq[m % 2]);
      float rloc[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        rloc[j] = acc[j] * h4[j] * r4[j] * (1.f - r4[j]);
        dacc[m][j] += acc[j] * r4[j];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) rv[4 * (m % 2) + j] = rloc[j];
      if (m % 2 == 1) {
        gf[0][m / 2] = pack8<S>(rv);
        const u32x4 pr = __builtin_bit_cast(u32x4, gf[0][m / 2]);   // G^'s r columns of tiles m - 1, m
        store_tiles16(gh + 32 * (m / 2), u32x2{pr[0], pr[1]}, u32x2{pr[2], pr[3]}, g);
      }
    }
  }
  // Every wave is done with U_n before pass 2's buffers overwrite it.
  __syncthreads();
  // Pass 2: blocks n = 0 .. MTL-1 of Wi (da) and U_r, U_z (dh).
#pragma unroll
  for (int n = 0; n < MTL; ++n) {
    const int b = n & 1;
    store_blk(2, b);
    __syncthreads();
    if (n + 1 < MTL) load_blk(2, n + 1);
    if (valid) {
      f32x4 da = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int gate = 0; gate < 3; ++gate)
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) mma(da, gf[gate][kk], load_fragi<S>(lw[b], gate * KS + kk, lane));
      store4(daT + (size_t)(16 * n + q) * n_pad + n0 + 4 * g, da[0], da[1], da[2], da[3]);
      f32x4 d = dacc[n];
#pragma unroll
      for (int gate = 0; gate < 2; ++gate)
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) mma(d, load_fragi<S>(lw[b] + BLK_W, gate * KS + kk, lane), gf[gate][kk]);
      store4(dh + (size_t)node * H + 16 * n + 4 * g, d[0], d[1], d[2], d[3]);
    }
  }
}

// ---------------------------------------------------------------------------
// Weight gradients of the GRU over one split of the rows k:
//   P[split][0][i][c] = sum_k a[k][i] G^[k][c]          (dWi)
//   P[split][1][i][c] = sum_k x_c[k][i] G^[k][c]        (dU)
// with x_c = h for the r and z columns and r*h for the n columns, and
//   Pb[split][c] = sum_k G^[k][c]                       (db).
// The rows are the nodes of all T steps at once (K = T * n_pad: a, h, saved
// and G^ stacked over t).  A workgroup owns one split of the rows and a
// slice of IT input features (all of them up to H = 64), every gate column:
// each input row is read once.  Per chunk of KC rows the operands are
// staged node-major in LDS (plain 16-byte copies; a rounded to bf16, r*h
// formed on the way) and read as matrix-core fragments with transposing
// LDS reads; the next chunk's loads are in flight during the products.
// Wave w: matrix w / 4 (dWi or dU) and a quarter of that matrix's tiles.
// ---------------------------------------------------------------------------
#ifndef GGNN_GRU_WGRAD_KC64
#define GGNN_GRU_WGRAD_KC64 64
#endif
#ifndef GGNN_GRU_WGRAD_MAXBUF
#define GGNN_GRU_WGRAD_MAXBUF 2
#endif
template <typename S, int H> struct GruWgradCfg {
  // input features per workgroup: each slice re-reads G^ (3H per row), so
  // slices are as wide as the accumulators allow
  static constexpr int IT = (H >= 256 && sizeof(S) == 2) ? 32 : (H >= 128 ? 4096 / H : H);
  static constexpr int NI = IT / 16, NCT = 3 * H / 16;  // tiles: input, gate columns
  static constexpr int KC = (sizeof(S) == 4 || H >= 256) ? 32 : (H >= 128 ? 64 : (H == 64 ? GGNN_GRU_WGRAD_KC64 : 128));   // rows per chunk
  static constexpr int IW = H == 32 ? 1 : NI;            // input tiles per wave
  static constexpr int CW = H == 32 ? 3 : NCT / 4;       // gate-column tiles per wave
  static constexpr int PA = IT + 16, PG = 3 * H + 16;    // LDS row pitches (elements)
  // LDS buffers: two (the next chunk is written while the current one is
  // read) when they fit in 160 KB.
  static constexpr int NBUF = GGNN_GRU_WGRAD_MAXBUF >= 2 && 2 * KC * (3 * PA + PG) * (int)sizeof(S) <= 160 * 1024 ? 2 : 1;
};

template <typename S, int H>
__global__ __launch_bounds__(512) void gru_wgrad_kernel(const float* __restrict__ a, const S* __restrict__ h,
                                                        const S* __restrict__ saved, const S* __restrict__ ghat,
                                                        float* __restrict__ P, float* __restrict__ Pb, long K,
                                                        int rows_per_split) {
  using C = GruWgradCfg<S, H>;
  constexpr int IT = C::IT, KC = C::KC, IW = C::IW, CW = C::CW, PA = C::PA, PG = C::PG, NBUF = C::NBUF;
  constexpr int NT = 512;
  constexpr int V = 16 / sizeof(S);
  constexpr int NA = KC * IT / V, NG = KC * 3 * H / V;   // 16-byte units per chunk
  constexpr int UA = (NA + NT - 1) / NT, UG = (NG + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) S sa[NBUF][3][KC * PA];   // a, h, r*h
  __shared__ __attribute__((aligned(16))) S sg[NBUF][KC * PG];      // G^

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  constexpr int NSL = H / IT;
  const int bid = xcd_swizzle(blockIdx.x, gridDim.x);
  const int sl = bid % NSL, split = bid / NSL;
  const int i0 = sl * IT;
  const long nlo = (long)split * rows_per_split;
  const long nhi = min(K, nlo + rows_per_split);
  const int mat = wave / 4, sub = wave % 4;
  const int it0 = H == 32 ? sub % 2 : 0;
  const int ct0 = H == 32 ? (sub / 2) * 3 : sub * CW;
  const bool do_bias = mat == 0 && sl == 0 && it0 == 0;

  f32x4 acc[IW][CW];
  float bsum[CW];
#pragma unroll
  for (int i = 0; i < IW; ++i)
#pragma unroll
    for (int c = 0; c < CW; ++c) acc[i][c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < CW; ++c) bsum[c] = 0.f;

  // Register stage of one chunk: per A unit the fp32 a (V values), h and r;
  // per G unit the 16 bytes of G^.
  f32x4 ra[UA][V / 4];
  u32x4 rh[UA], rr[UA], rg[UG];
  auto load_chunk = [&](long c0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < UA; ++u) {
      const int lin = u * NT + tid;
      const long row = c0 + lin / (IT / V);
      const int f = i0 + (lin % (IT / V)) * V;
      if ((NA % NT == 0 || lin < NA) && row < nhi) {
#pragma unroll
        for (int x = 0; x < V / 4; ++x) ra[u][x] = *reinterpret_cast<const f32x4*>(a + (size_t)row * H + f + 4 * x);
        rh[u] = *reinterpret_cast<const u32x4*>(h + (size_t)row * H + f);
        rr[u] = *reinterpret_cast<const u32x4*>(saved + (size_t)row * 3 * H + f);
      } else {   // rows past the split (a ragged last chunk) contribute zeros
#pragma unroll
        for (int x = 0; x < V / 4; ++x) ra[u][x] = f32x4{0.f, 0.f, 0.f, 0.f};
        rh[u] = u32x4{0u, 0u, 0u, 0u};
        rr[u] = u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int u = 0; u < UG; ++u) {
      const int lin = u * NT + tid;
      const long row = c0 + lin / (3 * H / V);
      const int c = (lin % (3 * H / V)) * V;
      rg[u] = ((NG % NT == 0 || lin < NG) && row < nhi)
                  ? *reinterpret_cast<const u32x4*>(ghat + (size_t)row * 3 * H + c)
                  : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_chunk = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < UA; ++u) {
      const int lin = u * NT + tid;
      if (NA % NT == 0 || lin < NA) {
        const int r = lin / (IT / V), f = (lin % (IT / V)) * V;
        const S* ph = reinterpret_cast<const S*>(&rh[u]);
        const S* pr = reinterpret_cast<const S*>(&rr[u]);
        float av[V], rhv[V];
#pragma unroll
        for (int x = 0; x < V; ++x) {
          av[x] = ra[u][x / 4][x % 4];
          rhv[x] = to_f<S>(ph[x]) * to_f<S>(pr[x]);
        }
        u32x4 wa, wr;
        if constexpr (sizeof(S) == 2) {
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            wa[x] = pk2(av[2 * x], av[2 * x + 1]);
            wr[x] = pk2(rhv[2 * x], rhv[2 * x + 1]);
          }
        } else {
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            wa[x] = __float_as_uint(av[x]);
            wr[x] = __float_as_uint(rhv[x]);
          }
        }
        *reinterpret_cast<u32x4*>(&sa[buf][0][r * PA + f]) = wa;
        *reinterpret_cast<u32x4*>(&sa[buf][1][r * PA + f]) = rh[u];
        *reinterpret_cast<u32x4*>(&sa[buf][2][r * PA + f]) = wr;
      }
    }
#pragma unroll
    for (int u = 0; u < UG; ++u) {
      const int lin = u * NT + tid;
      if (NG % NT == 0 || lin < NG) {
        const int r = lin / (3 * H / V), c = (lin % (3 * H / V)) * V;
        *reinterpret_cast<u32x4*>(&sg[buf][r * PG + c]) = rg[u];
      }
    }
  };

  // Splits start at multiples of KC rows; a last chunk that runs past the
  // split is zero-filled.
  if (nlo < nhi) load_chunk(nlo);
  int buf = 0;
  for (long c0 = nlo; c0 < nhi; c0 += KC, buf = NBUF == 2 ? buf ^ 1 : 0) {
    if (NBUF == 1 && c0 > nlo) __syncthreads();   // the previous chunk is fully read
    store_chunk(buf);
    __syncthreads();
    if (c0 + KC < nhi) load_chunk(c0 + KC);
#pragma unroll
    for (int k0 = 0; k0 < KC; k0 += 32) {
      frag_t<S> fa[IW][2];   // [.][0]: a (dWi) or h (dU r, z columns); [.][1]: r*h (dU n columns)
#pragma unroll
      for (int i = 0; i < IW; ++i) {
        const int n0 = 16 * (it0 + i);
        fa[i][0] = tr_frag(sa[buf][mat == 0 ? 0 : 1], PA, k0, n0, lane);
        if (mat == 1 && (ct0 + CW) * 16 > 2 * H) fa[i][1] = tr_frag(sa[buf][2], PA, k0, n0, lane);
      }
#pragma unroll
      for (int c = 0; c < CW; ++c) {
        const int ct = ct0 + c;
        const frag_t<S> fb = tr_frag(sg[buf], PG, k0, 16 * ct, lane);
        if (do_bias) {
#pragma unroll
          for (int x = 0; x < 8; ++x) bsum[c] += static_cast<float>(fb[x]);
        }
        const int src = (mat == 1 && 16 * ct >= 2 * H) ? 1 : 0;
#pragma unroll
        for (int i = 0; i < IW; ++i) mma(acc[i][c], src ? fa[i][1] : fa[i][0], fb);
      }
    }
  }
  // D[i = i0 + 16 (it0 + i) + 4g + j][c = 16 (ct0 + c) + q]
  float* out = P + ((size_t)split * 2 + mat) * H * 3 * H;
#pragma unroll
  for (int i = 0; i < IW; ++i)
#pragma unroll
    for (int c = 0; c < CW; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        out[(size_t)(i0 + 16 * (it0 + i) + 4 * g + j) * 3 * H + 16 * (ct0 + c) + q] = acc[i][c][j];
  if (do_bias) {
#pragma unroll
    for (int c = 0; c < CW; ++c) {
      float v = bsum[c];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g == 0) Pb[(size_t)split * 3 * H + 16 * (ct0 + c) + q] = v;
    }
  }
}

}  // namespace dev

namespace {
// Row split of the weight-gradient contraction: about 256 workgroups (one
// per compute unit, 8 waves each) over splits x input-feature slices;
// splits are multiples of 128 rows.
struct Split {
  int nsplit, per;
};
#ifndef GGNN_GRU_WGRAD_WGS
#define GGNN_GRU_WGRAD_WGS 256
#endif
// At H = 256 in bf16 the contraction of csrc/wgrad_wide.hip runs instead:
// six output tiles per split, 144 KB of LDS per workgroup (one per compute
// unit), so 42 splits (252 workgroups) of a multiple of 32 rows.
#ifndef GGNN_GRU_WGRAD256_LDS
#define GGNN_GRU_WGRAD256_LDS 1
#endif
#ifndef GGNN_GRU_WGRAD_PACE
#define GGNN_GRU_WGRAD_PACE 1
#endif
bool gru_wgrad256(long K, int H, bool f32) { return GGNN_GRU_WGRAD256_LDS && H == 256 && !f32 && K % 32 == 0; }
Split gru_split(long K, int H, bool f32) {
  if (gru_wgrad256(K, H, f32)) {
    const long want = GGNN_GRU_WGRAD_WGS / 6;
    const long per = std::max(32L, ((K + want - 1) / want + 31) / 32 * 32);
    return {(int)((K + per - 1) / per), (int)per};
  }
  const long slices = (H >= 256 && !f32) ? H / 32 : (H >= 128 ? H / (4096 / H) : 1);
  const long want = GGNN_GRU_WGRAD_WGS / slices > 0 ? GGNN_GRU_WGRAD_WGS / slices : 1;
  long per = ((K + want - 1) / want + 127) / 128 * 128;
  return {(int)((K + per - 1) / per), (int)per};
}

template <typename S, int H>
constexpr bool gru_big() {
  return sizeof(S) == 2 && H >= 128;
}

template <typename S, int H>
hipError_t gru_pack_h(const void* Wi, const void* U, void* packed, hipStream_t st) {
  if constexpr (gru_big<S, H>()) {
    const int units = 2 * dev::GruPack<H>::UNITS;
    hipLaunchKernelGGL((dev::gru_pack_kernel<S, H>), dim3((units + 255) / 256), dim3(256), 0, st,
                       static_cast<const S*>(Wi), static_cast<const S*>(U), static_cast<S*>(packed));
    return hipGetLastError();
  }
  return hipSuccess;   // no kernel reads the packed form
}

template <typename S, int H>
hipError_t gru_fwd_h(int n_pad, const float* a, const void* h, const void* Wi, const void* U, const float* b,
                     void* h_out, void* saved, const void* packed, hipStream_t st) {
  if constexpr (gru_big<S, H>()) {
    const S* pk = static_cast<const S*>(packed);
#define GGNN_GRU_FWD_BIG(PK)                                                                                   \
  hipLaunchKernelGGL((dev::gru_fwd_big_kernel<S, H, PK>), dim3((n_pad + 127) / 128), dim3(512), 0, st, a,      \
                     static_cast<const S*>(h), static_cast<const S*>(Wi), static_cast<const S*>(U), pk, b,      \
                     static_cast<S*>(h_out), static_cast<S*>(saved), n_pad)
    if (pk != nullptr)
      GGNN_GRU_FWD_BIG(true);
    else
      GGNN_GRU_FWD_BIG(false);
#undef GGNN_GRU_FWD_BIG
    return hipGetLastError();
  }
  constexpr int WAVES = 4;
  hipLaunchKernelGGL((dev::gru_fwd_kernel<S, H, WAVES>), dim3((n_pad + 16 * WAVES - 1) / (16 * WAVES)),
                     dim3(WAVES * 64), 0, st, a, static_cast<const S*>(h), static_cast<const S*>(Wi),
                     static_cast<const S*>(U), b, static_cast<S*>(h_out), static_cast<S*>(saved), n_pad);
  return hipGetLastError();
}

template <typename S, int H>
hipError_t gru_bwd_nodes_h(int n_pad, const float* dh_out, const void* h, const void* saved, const void* Wi,
                           const void* U, void* da, float* dh, void* ghat, const void* packed, hipStream_t st) {
  if constexpr (gru_big<S, H>()) {
    // the reverse region follows the forward one
    const S* pk = packed ? static_cast<const S*>(packed) + (size_t)dev::GruPack<H>::UNITS * 8 : nullptr;
#define GGNN_GRU_BWD_BIG(PK)                                                                                   \
  hipLaunchKernelGGL((dev::gru_bwd_big_kernel<S, H, PK>), dim3((n_pad + 127) / 128), dim3(512), 0, st, dh_out, \
                     static_cast<const S*>(h), static_cast<const S*>(saved), static_cast<const S*>(Wi),         \
                     static_cast<const S*>(U), pk, static_cast<S*>(da), dh, static_cast<S*>(ghat), n_pad)
    if (pk != nullptr)
      GGNN_GRU_BWD_BIG(true);
    else
      GGNN_GRU_BWD_BIG(false);
#undef GGNN_GRU_BWD_BIG
    return hipGetLastError();
  }
  constexpr int WAVES = 4;
  hipLaunchKernelGGL((dev::gru_bwd_kernel<S, H, WAVES>), dim3((n_pad + 16 * WAVES - 1) / (16 * WAVES)),
                     dim3(WAVES * 64), 0, st, dh_out, static_cast<const S*>(h), static_cast<const S*>(saved),
                     static_cast<const S*>(Wi), static_cast<const S*>(U), static_cast<S*>(da), dh,
                     static_cast<S*>(ghat), n_pad);
  return hipGetLastError();
}

template <typename S, int H>
hipError_t gru_wgrad_h(long K, const float* a, const void* h, const void* saved, const void* ghat, float* dWi,
                       float* dU, float* db, void* ws, ReduceList* defer, hipStream_t st) {
  Split sp = gru_split(K, H, sizeof(S) == 4);
  float* P = static_cast<float*>(ws);
  float* Pb = P + (size_t)sp.nsplit * 2 * H * 3 * H;
  hipError_t err;
  if (sizeof(S) == 2 && H == 256 && gru_wgrad256(K, H, false)) {
    int* prog = reinterpret_cast<int*>(Pb + (size_t)sp.nsplit * 3 * H);   // pacing counters
    err = launch_gru_wgrad256(sp.nsplit, sp.per, K, a, h, saved, ghat, P, Pb, GGNN_GRU_WGRAD_PACE ? prog : nullptr,
                              st);
  } else {
    const int blocks = sp.nsplit * (H / dev::GruWgradCfg<S, H>::IT);
    hipLaunchKernelGGL((dev::gru_wgrad_kernel<S, H>), dim3(blocks), dim3(512), 0, st, a,
                       static_cast<const S*>(h), static_cast<const S*>(saved), static_cast<const S*>(ghat), P, Pb,
                       K, sp.per);
    err = hipGetLastError();
  }
  if (err != hipSuccess) return err;
  const long slice = 2L * H * 3 * H;  // partials are [split][which][H][3H]
  err = reduce_or_defer(P, dWi, sp.nsplit, H * 3 * H, slice, defer, st);
  if (err != hipSuccess) return err;
  err = reduce_or_defer(P + (size_t)H * 3 * H, dU, sp.nsplit, H * 3 * H, slice, defer, st);
  if (err != hipSuccess) return err;
  return reduce_or_defer(Pb, db, sp.nsplit, 3 * H, 3L * H, defer, st);
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
hipError_t gru_pack_t(int H, const void* Wi, const void* U, void* packed, hipStream_t st) {
  GGNN_GRU_SWITCH(return (gru_pack_h<S, HH>(Wi, U, packed, st)))
}
template <typename S>
hipError_t gru_fwd_t(int n_pad, int H, const float* a, const void* h, const void* Wi, const void* U, const float* b,
                     void* h_out, void* saved, const void* packed, hipStream_t st) {
  GGNN_GRU_SWITCH(return (gru_fwd_h<S, HH>(n_pad, a, h, Wi, U, b, h_out, saved, packed, st)))
}
template <typename S>
hipError_t gru_bwd_nodes_t(int n_pad, int H, const float* dh_out, const void* h, const void* saved, const void* Wi,
                           const void* U, void* da, float* dh, void* ghat, const void* packed, hipStream_t st) {
  GGNN_GRU_SWITCH(return (gru_bwd_nodes_h<S, HH>(n_pad, dh_out, h, saved, Wi, U, da, dh, ghat, packed, st)))
}
template <typename S>
hipError_t gru_wgrad_t(long K, int H, const float* a, const void* h, const void* saved, const void* ghat, float* dWi,
                       float* dU, float* db, void* ws, ReduceList* defer, hipStream_t st) {
  GGNN_GRU_SWITCH(return (gru_wgrad_h<S, HH>(K, a, h, saved, ghat, dWi, dU, db, ws, defer, st)))
}
#undef GGNN_GRU_SWITCH
}  // namespace

#if GGNN_DT_BF16   // dtype-independent helpers: built once
size_t ghat_bytes(int dt, long rows, int H) {
  size_t b = (size_t)rows * 3 * H * (dt == GGNN_BF16 ? 2 : 4);
  return (b + 255) / 256 * 256;
}

size_t gru_wgrad_workspace(long K, int H) {
  // large enough for the split of either dtype
  Split sp = gru_split(K, H, false);
  const Split s32 = gru_split(K, H, true);
  if (s32.nsplit > sp.nsplit) sp = s32;
  // partials, bias partials, then 8 pacing counters per split (H = 256 bf16)
  return ((size_t)sp.nsplit * 2 * H * 3 * H + (size_t)sp.nsplit * 3 * H + (size_t)sp.nsplit * 8) * sizeof(float);
}

size_t gru_pack_bytes(int dt, int H) {
  return dt == GGNN_BF16 && H >= 128 ? (size_t)12 * H * H * 2 : 0;
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
hipError_t launch_gru_pack(int H, const void* Wi, const void* U, void* packed, hipStream_t st) {
  return gru_pack_t<dev::dt_t>(H, Wi, U, packed, st);
}

hipError_t launch_gru_fwd(int n_pad, int H, const float* a, const void* h, const void* Wi, const void* U,
                          const float* b, void* h_out, void* saved, const void* packed, hipStream_t st) {
  return gru_fwd_t<dev::dt_t>(n_pad, H, a, h, Wi, U, b, h_out, saved, packed, st);
}

hipError_t launch_gru_bwd_nodes(int n_pad, int H, const float* dh_out, const void* h, const void* saved,
                                const void* Wi, const void* U, void* da, float* dh, void* ghat, const void* packed,
                                hipStream_t st) {
  return gru_bwd_nodes_t<dev::dt_t>(n_pad, H, dh_out, h, saved, Wi, U, da, dh, ghat, packed, st);
}

hipError_t launch_gru_wgrad(long K, int H, const float* a, const void* h, const void* saved, const void* ghat,
                            float* dWi, float* dU, float* db, void* ws, ReduceList* defer, hipStream_t st) {
  return gru_wgrad_t<dev::dt_t>(K, H, a, h, saved, ghat, dWi, dU, db, ws, defer, st);
}
}  // namespace GGNN_IMPL_NS

}  // namespace ggnn
