// Reverse of the GRU node update (Eq. 1's GRU, Cho et al. 2014 form) for
// the 16 nodes of one wave, shared by the stand-alone GRU reverse kernel and
// the fused bit-band reverse step.
//
// Lanes: q = lane % 16 is the node (n0 + q), g = lane / 16.  With
// g' = dL/dh', dn = g'(1-z), dz = g'(h-n), n^ = dn(1-n^2), z^ = dz z(1-z),
// q' = n^ U_n^T, r^ = q' h r(1-r):
//   dh = g' z + q' r + r^ U_r^T + z^ U_z^T,   da = [r^ z^ n^] Wi^T.
// The gate gradients are kept in registers as operand fragments
// (accumulator-compatible order: features 32kk + 4g + {0..3} and
// 32kk + 16 + 4g + {0..3}) and dh as an accumulator across the phases;
// G^ = [r^ z^ n^] is also written to `ghat` (node-major [.][3H]) for the
// weight-gradient pass.
#pragma once

#include "device_common.h"

namespace ggnn {
namespace dev {

// Node-major stores of two consecutive 16-feature tiles of a wave's 16 nodes
// (lane (q, g) holds features 4g .. 4g + 3 of each tile, rounded to bf16 and
// packed: t0 the first tile, t1 the second) as one 16-byte store per lane:
// after one permlane32 and one permlane16 swap per dword, lane group g holds
// features 8g .. 8g + 7 of the 32 (groups 0, 1 the first tile's, 2, 3 the
// second's).  Each node row then gets 64 contiguous bytes per instruction
// instead of 32 from 8-byte stores, which streams ~20% faster on this GPU
// (used for the GRU reverse's G^; in the large-H forward, its h', r, z, n
// stores paired this way measured no gain and cost registers).  All 64 lanes
// must be active.
__device__ __forceinline__ void store_tiles16(bf16s* row32, u32x2 t0, u32x2 t1, int g) {
  uint32_t x[2], y[2];
#pragma unroll
  for (int d = 0; d < 2; ++d) {
    // rows of 16 lanes: (A0 A1 A2 A3), (B0 B1 B2 B3) -> (A0 A1 B0 B1), (A2 A3 B2 B3)
    const auto r32 = __builtin_amdgcn_permlane32_swap(t0[d], t1[d], false, false);
    // -> (A0 A2 B0 B2), (A1 A3 B1 B3): lane group g holds (first, second) half of its 8 features
    const auto r16 = __builtin_amdgcn_permlane16_swap(r32[0], r32[1], false, false);
    x[d] = r16[0];
    y[d] = r16[1];
  }
  *reinterpret_cast<u32x4*>(row32 + 8 * g) = u32x4{x[0], x[1], y[0], y[1]};
}
// The reverse: the 16 bytes a lane loads at features 8g .. 8g + 7 of the 32
// (v), handed out as store_tiles16 takes them (both swaps are their own
// inverse): t[0] = features 4g .. 4g + 3 of the first tile, t[1] of the
// second.  Split from the load so that a load can be issued well ahead.
__device__ __forceinline__ void split_tiles16(const u32x4& v, u32x2 (&t)[2]) {
#pragma unroll
  for (int d = 0; d < 2; ++d) {
    const auto r16 = __builtin_amdgcn_permlane16_swap(v[d], v[2 + d], false, false);
    const auto r32 = __builtin_amdgcn_permlane32_swap(r16[0], r16[1], false, false);
    t[0][d] = r32[0];
    t[1][d] = r32[1];
  }
}
__device__ __forceinline__ void load_tiles16(const bf16s* row32, int g, u32x2 (&t)[2]) {
  split_tiles16(*reinterpret_cast<const u32x4*>(row32 + 8 * g), t);
}
__device__ __forceinline__ f32x4 unpack4(u32x2 v) {
  return f32x4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u), __uint_as_float(v.y << 16),
               __uint_as_float(v.y & 0xFFFF0000u)};
}

// Fragment of a node-major row in accumulator-compatible k order.
template <typename S>
__device__ __forceinline__ frag_t<S> rowfrag(const S* row, int kk, int g) {
  return load4x2(row + 32 * kk + 4 * g, row + 32 * kk + 16 + 4 * g);
}

// The per-node inputs of the GRU reverse, for features 16m + 4g + {0..3}
// of one node: the saved gates r, z, n and the state h (loaded ahead of
// use by the fused reverse step, where the loads cross a barrier).
template <typename S, int H>
struct GruBwdIn {
  f32x4 r[H / 16], z[H / 16], n[H / 16], h[H / 16];
  __device__ __forceinline__ void load(const S* saved, const S* hs, int node, int g) {
    const S* sv = saved + (size_t)node * 3 * H;
#pragma unroll
    for (int m = 0; m < H / 16; ++m) {
      const int f = 16 * m + 4 * g;
      r[m] = load4f(sv + f);
      z[m] = load4f(sv + H + f);
      n[m] = load4f(sv + 2 * H + f);
      h[m] = load4f(hs + (size_t)node * H + f);
    }
  }
  __device__ __forceinline__ void expand(int) const {}
};
// bf16: one 16-byte load per lane and 32 features of each input (features
// 8g .. 8g + 7 of the 32), kept raw until expand() hands them out per
// 16-feature tile (split_tiles16), so that the loads can stay in flight
// across barriers.
template <int H>
struct GruBwdIn<bf16s, H> {
  static constexpr int NP = H / 32;
  u32x4 raw[4][NP];   // r, z, n, h
  f32x4 r[H / 16], z[H / 16], n[H / 16], h[H / 16];
  __device__ __forceinline__ void load(const bf16s* saved, const bf16s* hs, int node, int g) {
    const bf16s* sv = saved + (size_t)node * 3 * H;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      raw[0][p] = *reinterpret_cast<const u32x4*>(sv + 32 * p + 8 * g);
      raw[1][p] = *reinterpret_cast<const u32x4*>(sv + H + 32 * p + 8 * g);
      raw[2][p] = *reinterpret_cast<const u32x4*>(sv + 2 * H + 32 * p + 8 * g);
      raw[3][p] = *reinterpret_cast<const u32x4*>(hs + (size_t)node * H + 32 * p + 8 * g);
    }
  }
  // All 64 lanes active (lane-group swaps).
  __device__ __forceinline__ void expand(int) {
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      u32x2 t[2];
      split_tiles16(raw[0][p], t);
      r[2 * p] = unpack4(t[0]);
      r[2 * p + 1] = unpack4(t[1]);
      split_tiles16(raw[1][p], t);
      z[2 * p] = unpack4(t[0]);
      z[2 * p + 1] = unpack4(t[1]);
      split_tiles16(raw[2][p], t);
      n[2 * p] = unpack4(t[0]);
      n[2 * p + 1] = unpack4(t[1]);
      split_tiles16(raw[3][p], t);
      h[2 * p] = unpack4(t[0]);
      h[2 * p + 1] = unpack4(t[1]);
    }
  }
};

// gg[m]: dL/dh' for features 16m + 4g + {0..3} of node n0 + q; in: the
// gates and state of that node (GruBwdIn::load).
// wfrag(which, row, gate, kk): the weight fragment of input feature `row`
// (row % 16 == q) and gate columns gate*H + 32kk + (accumulator-compatible
// order) of Wi (which = 0) or U (which = 1), from LDS or global memory.
// Writes daT[f][n0 + 4g + j] (feature-major, row pitch ld), dh[node][.]
// (node-major, float) and ghat[node][.] (node-major, 3H).
template <typename S, int H, typename WF>
__device__ __forceinline__ void gru_bwd_wave(const f32x4 (&gg)[H / 16], int n0, int q, int g,
                                             GruBwdIn<S, H>& in, WF wfrag, S* daT, long ld, float* dh,
                                             S* ghat) {
  constexpr int KS = H / 32;
  constexpr int MTL = H / 16;
  const int node = n0 + q;
  in.expand(g);
  // Phase 1: elementwise part, kept in registers.
  frag_t<S> gf[3][KS];          // r^, z^, n^ as operand fragments
  f32x4 dacc[MTL];              // dh accumulator (D layout: features 16m + 4g + j)
  float zv[8], nv[8];
  S* gh = ghat + (size_t)node * 3 * H;
#pragma unroll
  for (int m = 0; m < MTL; ++m) {
    const int f = 16 * m + 4 * g;
    const f32x4 z4 = in.z[m], n4 = in.n[m], h4 = in.h[m];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float dn = gg[m][j] * (1.f - z4[j]);
      const float dz = gg[m][j] * (h4[j] - n4[j]);
      dacc[m][j] = gg[m][j] * z4[j];
      nv[4 * (m % 2) + j] = dn * (1.f - n4[j] * n4[j]);
      zv[4 * (m % 2) + j] = dz * z4[j] * (1.f - z4[j]);
    }
    if (m % 2 == 1) {
      gf[2][m / 2] = pack8<S>(nv);
      gf[1][m / 2] = pack8<S>(zv);
    }
    if constexpr (sizeof(S) == 2) {
      if (m % 2 == 1) {   // G^'s z, n columns of tiles m - 1, m as 16-byte stores
        const u32x4 pz = __builtin_bit_cast(u32x4, gf[1][m / 2]), pn = __builtin_bit_cast(u32x4, gf[2][m / 2]);
        store_tiles16(gh + H + 32 * (m / 2), u32x2{pz[0], pz[1]}, u32x2{pz[2], pz[3]}, g);
        store_tiles16(gh + 2 * H + 32 * (m / 2), u32x2{pn[0], pn[1]}, u32x2{pn[2], pn[3]}, g);
      }
    } else {
      store4(gh + H + f, zv[4 * (m % 2)], zv[4 * (m % 2) + 1], zv[4 * (m % 2) + 2], zv[4 * (m % 2) + 3]);
      store4(gh + 2 * H + f, nv[4 * (m % 2)], nv[4 * (m % 2) + 1], nv[4 * (m % 2) + 2], nv[4 * (m % 2) + 3]);
    }
  }
  // Phase 2: q' = n^ U_n^T (D[f_in][node]); r^ and the q' r term of dh.
  {
    float rv[8];
    f32x4 qacc[MTL];
#pragma unroll
    for (int m = 0; m < MTL; ++m) qacc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
#pragma unroll
      for (int m = 0; m < MTL; ++m) mma(qacc[m], wfrag(1, 16 * m + q, 2, kk), gf[2][kk]);
#pragma unroll
    for (int m = 0; m < MTL; ++m) {
      const f32x4 acc = qacc[m];
      const int f = 16 * m + 4 * g;
      const f32x4 r4 = in.r[m], h4 = in.h[m];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        rv[4 * (m % 2) + j] = acc[j] * h4[j] * r4[j] * (1.f - r4[j]);
        dacc[m][j] += acc[j] * r4[j];
      }
      if (m % 2 == 1) gf[0][m / 2] = pack8<S>(rv);
      if constexpr (sizeof(S) == 2) {
        if (m % 2 == 1) {   // G^'s r columns of tiles m - 1, m
          const u32x4 pr = __builtin_bit_cast(u32x4, gf[0][m / 2]);
          store_tiles16(gh + 32 * (m / 2), u32x2{pr[0], pr[1]}, u32x2{pr[2], pr[3]}, g);
        }
      } else {
        store4(gh + f, rv[4 * (m % 2)], rv[4 * (m % 2) + 1], rv[4 * (m % 2) + 2], rv[4 * (m % 2) + 3]);
      }
    }
  }
  // Phase 3: da = G^ Wi^T, D[node][f_in]: four consecutive nodes per lane;
  // phase 4: dh += r^ U_r^T + z^ U_z^T, D[f_in][node].  The k loops are
  // outermost so that the MTL accumulators of each form independent chains.
  f32x4 dacc2[MTL];
#pragma unroll
  for (int n = 0; n < MTL; ++n) dacc2[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int gate = 0; gate < 3; ++gate)
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
#pragma unroll
      for (int n = 0; n < MTL; ++n) mma(dacc2[n], gf[gate][kk], wfrag(0, 16 * n + q, gate, kk));
#pragma unroll
  for (int gate = 0; gate < 2; ++gate)
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
#pragma unroll
      for (int m = 0; m < MTL; ++m) mma(dacc[m], wfrag(1, 16 * m + q, gate, kk), gf[gate][kk]);
#pragma unroll
  for (int n = 0; n < MTL; ++n)
    store4(daT + (size_t)(16 * n + q) * ld + n0 + 4 * g, dacc2[n][0], dacc2[n][1], dacc2[n][2], dacc2[n][3]);
#pragma unroll
  for (int m = 0; m < MTL; ++m)
    store4(dh + (size_t)node * H + 16 * m + 4 * g, dacc[m][0], dacc[m][1], dacc[m][2], dacc[m][3]);
}

}  // namespace dev
}  // namespace ggnn
