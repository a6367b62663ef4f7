// Wide fused step on a 1-bit block band (bf16 storage, H >= 128, where the
// three node blocks with all features are too large to stage whole; B from
// 32 to 512, one workgroup per block row of up to 256 rows, B / 32 waves
// below that): the products of the fused step of Eq. 3 in the operand order
// of Algorithm 1,
//   forward:  a[k]    = sum_e (sum_s bits[e][k][s] X[k-1+s]) W_e   (+ deg_e b_e)
//   reverse:  dM_e[k] = sum_s bits_t[e][k][s] da[k-1+s]            (stored)
//             dX[k]   = dX_in[k] + sum_e dM_e[k] W_e^T
// arranged so that every operand staged in LDS feeds several matrix-core
// steps and the node blocks are staged once per workgroup, not per edge type.
//
// The transform's contraction over features is split into slices of HQ
// features (64 or 32, chosen per shape below):
//   (A_e X) W_e = sum_q (A_e X[:, q]) W_e[q, :].
// For each slice q the workgroup stages features q of the three node blocks
// (k-1, k, k+1) once; every edge type then reuses them.  Per type a wave
// aggregates its 32 rows over the slice (registers, 32 x HQ), then
// multiplies that into its output accumulators (32 rows x H, registers) with
// rows q of W_e (reverse) or of W_e^T (forward).  The bit rows expanded to
// matrix-core fragments (vector ALU work) feed HQ / 16 products each, so the
// wider slice keeps the matrix cores, not the expansion, the bottleneck.
// The weights pass through LDS in units of 32 features (H rows, fragment
// order), shared by all waves: a ring of NH + 1 unit buffers (NH = HQ / 32),
// the next slice's units loaded while the current ones are used and written
// after each unit's products, one barrier per unit.  The next slice's node
// blocks are prefetched over the type loop into a second buffer where LDS
// allows, otherwise staged at the slice boundary.
//
// LDS layouts of a staged block slice (B nodes x HQ features):
//   forward (X node-major in HBM): node rows of HQ features, read with
//     ds_read_b64_tr_b16, which hands a lane eight consecutive nodes of one
//     feature.  Within a 32-feature group, feature f sits in column
//     16 (f % 8 / 4) + 4 (f / 8) + f % 4, so the aggregate's tiles give a lane
//     eight consecutive features (the weight fragments are 16-byte rows; the
//     reverse stores dM with one 16-byte write).  The 16-column groups of a
//     row are XOR-swizzled by row and lane group so that the four rows one
//     read touches, and the two lane groups served together, hit disjoint
//     banks.
//   reverse (da feature-major in HBM): fragment order (a fragment's 64 lane
//     vectors contiguous, 16-byte copies), features in the same order.
#include "device_common.h"
#include "kernels.h"

namespace ggnn {
namespace dev {

#ifndef GGNN_WIDE_FWD_HQ64
#define GGNN_WIDE_FWD_HQ64 1
#endif
template <int H, int B, bool REV, bool BIAS = false>
struct WideCfg {
  // Features per slice: 64 where the three blocks' slice and the weight ring
  // fit in LDS and the workgroup fills a compute unit anyway (B >= 256),
  // except the forward with a message bias at H = 256 (its registers spill
  // at 64); else 32 (at B = 128 two workgroups then share a compute unit).
  // With empty k steps skipped, fewer, wider slices halve the per-slice
  // fixed work (bit loads and re-ordering, skip tests, barriers): the
  // H = 256 forward on the 1M-node workload went 4.26 -> 3.54 ms at 64.
  static constexpr int HQ =
      (B >= 256 && (REV || H <= 128 || (GGNN_WIDE_FWD_HQ64 && !BIAS)) && (3 * B * 64 + 3 * H * 32) * 2 <= 160 * 1024)
          ? 64
          : 32;
  static constexpr int NQ = H / HQ;             // slices
  static constexpr int NH = HQ / 32;            // 32-feature weight units per slice
  static constexpr int MQ = HQ / 16;            // aggregation tiles per slice
  static constexpr int NWB = NH + 1;            // weight-unit buffers
  static constexpr int RPW = 32, NTW = 2;       // rows per wave, 16-row tiles per wave
  static constexpr int WAVES = B / RPW < 8 ? B / RPW : 8;
  static constexpr int R = WAVES * RPW;         // rows per workgroup
  static constexpr int NT = WAVES * kWave;
  static constexpr int RB = B / 32;             // bit-row bytes per lane and block
  static constexpr int GROW = B / 4;            // block columns per lane group (split k order)
  // k order of a block's B columns over the RB matrix-core k steps:
  //   contiguous (B = 128, 256): step kk covers columns 32 kk .. 32 kk + 31,
  //     lane group g the eight columns 32 kk + 8 g + {0..7};
  //   split (other B): lane group g covers columns g GROW .. g GROW + GROW - 1,
  //     step kk the eight columns g GROW + 8 kk + {0..7}.
  // The contiguous order keeps a step's columns together, so the steps whose
  // columns hold no edge into a wave's rows (most of them in a band much
  // narrower than B) are skipped whole.
  static constexpr bool KCONT = (RB == 4 || RB == 8);
  static constexpr int XS = B * HQ;             // elements per staged block slice
  static constexpr int WS = (H / 16) * kWave * 8;   // elements per weight unit
  static constexpr int NXB = (2 * 3 * XS + NWB * WS) * 2 <= 160 * 1024 ? 2 : 1;   // block-slice buffers
  static constexpr int UNITS = 3 * B * HQ / 8;  // 16-byte units of one slice of the three blocks
  static constexpr int XPT = 2;                 // of which each thread prefetches per (slice, type)
  static constexpr int WPT = (H * 4 + NT - 1) / NT;   // 16-byte vectors per thread per weight unit
};

// Feature f of a slice -> its (tile, row) slot, as 16 * tile + row (tile
// 2j + i of the 32-feature group j holds features 32j + 8r + 4i + {0..3} in
// rows 4r + {0..3}); also its column in a forward node row, before the
// swizzle.
__device__ __forceinline__ int wide_slot(int f) {
  const int w = f % 32;
  return 32 * (f / 32) + 16 * ((w % 8) / 4) + 4 * (w / 8) + w % 4;
}
// Lane group and k step of block column c (a multiple of 8 for the step).
template <bool KCONT, int GROW>
__device__ __forceinline__ int wide_colgroup(int c) {
  return KCONT ? (c >> 3) & 3 : c / GROW;
}
template <bool KCONT, int GROW>
__device__ __forceinline__ int wide_colstep(int c) {
  return KCONT ? c >> 5 : (c % GROW) / 8;
}
// First block column of lane group g at k step kk.
template <bool KCONT, int GROW>
__device__ __forceinline__ int wide_col0(int g, int kk) {
  return KCONT ? 32 * kk + 8 * g : g * GROW + 8 * kk;
}
// Swizzle of the 16-column groups of forward node row c (block-local): the
// lane group's parity (and, at HQ = 64, bit 1 of the row), so that the rows
// two lane groups read in one pass, and the four rows one read touches,
// fall on disjoint banks.
template <int HQ, bool KCONT, int GROW>
__device__ __forceinline__ int wide_sw(int c) {
  const int gp = wide_colgroup<KCONT, GROW>(c) & 1;
  if constexpr (HQ == 64) {
    return ((c >> 1) & 1) | (gp << 1);
  } else {
    return gp;
  }
}

// Transposing fragment read: lane (p, g) addresses a0 (its lane group's row
// p / 4 at column 4 (p % 4)); the lane receives element (row + j, column p)
// for j = 0..7 (rows j >= 4 from the second read, 4 rows further on).
__device__ __forceinline__ bf16x8 tr_read8(const bf16s* a0, int pitch) {
  const tr_v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_tr_v4i16*)(const_cast<bf16s*>(a0)));
  const tr_v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_tr_v4i16*)(const_cast<bf16s*>(a0) + 4 * pitch));
  typedef short v8i16 __attribute__((ext_vector_type(8)));
  const v8i16 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// 8 bits -> 8 bf16 elements equal to 0 or 1 (bit i -> element i); see the
// same expansion in the narrow step kernels.
__device__ __forceinline__ bf16x8 wide_bits_frag(uint32_t byte) {
  const uint32_t x = byte * 0x8001u;
  u32x4 w;
#pragma unroll
  for (int k = 0; k < 4; ++k) w[k] = (x & (0x10001u << (2 * k))) * (0x3F80u >> (2 * k));
  return __builtin_bit_cast(bf16x8, w);
}

// Whether any lane of the wave holds a nonzero x (the same answer in every
// lane, so a branch on it is taken by the whole wave).
__device__ __forceinline__ bool wide_any(uint32_t x) { return __builtin_amdgcn_ballot_w64(x != 0u) != 0; }

template <int NB> struct WideBits {
  static constexpr int NW = NB < 4 ? 1 : NB / 4;
  uint32_t w[NW];
  __device__ __forceinline__ void load(const uint8_t* p) {
    if constexpr (NB == 1) {
      w[0] = *p;
    } else if constexpr (NB == 2) {
      w[0] = *reinterpret_cast<const uint16_t*>(p);
    } else if constexpr (NB == 4) {
      w[0] = *reinterpret_cast<const uint32_t*>(p);
    } else if constexpr (NB == 8) {
      const u32x2 v = *reinterpret_cast<const u32x2*>(p);
      w[0] = v[0];
      w[1] = v[1];
    } else {
      const u32x4 v = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = v[i];
    }
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] = 0u;
  }
  __device__ __forceinline__ uint32_t byte(int i) const { return (w[i / 4] >> (8 * (i % 4))) & 0xFFu; }
  // From the split byte order to the contiguous one (see
  // bytes_to_contiguous).  `odd` is g & 1.
  __device__ __forceinline__ void to_contiguous(uint32_t odd) { bytes_to_contiguous<NB>(w, odd); }
  __device__ __forceinline__ int popc() const {
    int c = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) c += __popc(w[i]);
    return c;
  }
};

// Workgroup: C::R rows of block row k (the workgroup's tile t % (B / R)),
// C::WAVES waves of 32 rows.  V = X (forward, node-major [n_pad][H]) or da
// (reverse, feature-major [H][n_pad]); Wsrc = W_e^T (forward) or W_e
// (reverse), [E][H][H], row o holding the o-th output feature's weights.
template <int H, int B, bool REV, bool BIAS>
__global__ __launch_bounds__((WideCfg<H, B, REV>::NT)) void step_wide_kernel(
    const uint8_t* __restrict__ bits, const bf16s* __restrict__ V, const bf16s* __restrict__ Wsrc,
    const float* __restrict__ bias, float* __restrict__ out, int n_pad, int E, const float* __restrict__ dX_in,
    bf16s* __restrict__ dM, long ldm) {
  using C = WideCfg<H, B, REV, BIAS>;
  constexpr int NT = C::NT, HQ = C::HQ, NQ = C::NQ, NH = C::NH, MQ = C::MQ, NWB = C::NWB;
  constexpr int NTW = C::NTW, RB = C::RB, XS = C::XS, GROW = C::GROW;
  constexpr int MT = H / 16;             // 16-feature output tiles
  constexpr int NP = REV ? 1 : 2;        // forward: the aggregate enters the transform as bf16 hi + lo
  constexpr int ROWB = B / 8;
  constexpr int UB = C::UNITS / 3;       // units per block
  constexpr int TPR = B / C::R;
  __shared__ __attribute__((aligned(16))) bf16s xs[C::NXB][3 * XS];
  __shared__ __attribute__((aligned(16))) bf16s ws[NWB][C::WS];

  const int nb = n_pad / B;
  const int t = xcd_swizzle(blockIdx.x, gridDim.x);
  const int k = t / TPR;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int rw = (t % TPR) * C::R + C::RPW * wave;   // first row (block-local) of this wave
  const int s_lo = (k == 0) ? 1 : 0;
  const int s_hi = (k == nb - 1) ? 1 : 2;
  const int iters = NQ * E;

  // ---- staging units ----------------------------------------------------
  // Unit u of slice qs, block s = u / UB, r = u % UB.  Forward: node
  // c = r / (HQ/8) of the block, features qs*HQ + 8G .. 8G + 7 (G = r %
  // (HQ/8)); reverse: feature f = 16 (r / (16 B/8)) + r % 16 of the slice,
  // nodes 8 c8 .. 8 c8 + 7 (c8 = (r / 16) % (B/8)).  Units of a block
  // outside the matrix are skipped.
  auto unit_ok = [&](int u) __attribute__((always_inline)) {
    const int s = u / UB;
    return u < C::UNITS && s >= s_lo && s <= s_hi;
  };
  auto unit_load = [&](int u, int qs) __attribute__((always_inline)) {
    const int s = u / UB, r = u % UB;
    const bf16s* p;
    if constexpr (!REV) {
      p = V + (size_t)((k - 1 + s) * B + r / (HQ / 8)) * H + qs * HQ + 8 * (r % (HQ / 8));
    } else {
      const int f = 16 * (r / (16 * (B / 8))) + r % 16, c8 = (r / 16) % (B / 8);
      p = V + (size_t)(qs * HQ + f) * n_pad + (k - 1 + s) * B + 8 * c8;
    }
    return *reinterpret_cast<const u32x4*>(p);
  };
  auto unit_store = [&](int u, bf16s* xb, const u32x4& v) __attribute__((always_inline)) {
    const int s = u / UB, r = u % UB;
    bf16s* d = xb + s * XS;
    if constexpr (!REV) {
      const int c = r / (HQ / 8), G = r % (HQ / 8);
      const int sw = wide_sw<HQ, C::KCONT, GROW>(c);
      const int m0 = 2 * (G / 4), w0 = 4 * (G % 4);   // tiles m0, m0 + 1 of the 32-group G / 4
      bf16s* row = d + c * HQ;
      *reinterpret_cast<u32x2*>(row + 16 * (m0 ^ sw) + w0) = u32x2{v[0], v[1]};         // features 8G .. 8G+3
      *reinterpret_cast<u32x2*>(row + 16 * ((m0 + 1) ^ sw) + w0) = u32x2{v[2], v[3]};   // features 8G+4 .. 8G+7
    } else {
      const int f = 16 * (r / (16 * (B / 8))) + r % 16, c = 8 * ((r / 16) % (B / 8));
      // fragment (kk, tile) of the block: lane group c / (B/4), k step (c % (B/4)) / 8
      const int slot = wide_slot(f), gg = wide_colgroup<C::KCONT, GROW>(c), kk = wide_colstep<C::KCONT, GROW>(c);
      *reinterpret_cast<u32x4*>(d + fo<bf16s>(kk * MQ + slot / 16, slot % 16 + 16 * gg, 0)) = v;
    }
  };
  auto stage_x = [&](int qs, bf16s* xb, int u0) __attribute__((always_inline)) {
    for (int u = u0 + tid; u < C::UNITS; u += NT)
      if (unit_ok(u)) unit_store(u, xb, unit_load(u, qs));
  };
  // Weight unit (slice qs, type e, half h2), vector u: output row o = u / 4,
  // features qs*HQ + 32 h2 + 8G .. + 7 (G = u % 4): one fragment vector.
  auto w_load = [&](int u, int qs, int e, int h2) __attribute__((always_inline)) {
    return *reinterpret_cast<const u32x4*>(Wsrc + (size_t)e * H * H + (size_t)(u / 4) * H + qs * HQ + 32 * h2 +
                                           8 * (u % 4));
  };
  auto w_store = [&](int u, bf16s* wb, const u32x4& v) __attribute__((always_inline)) {
    const int o = u / 4, G = u % 4;
    *reinterpret_cast<u32x4*>(wb + fo<bf16s>(o / 16, o % 16 + 16 * G, 0)) = v;
  };

  // ---- bit rows ---------------------------------------------------------
  WideBits<RB> cur[3][NTW], nxt[3][NTW];
  // Byte offset of the lane's part of row 16n + q of block s within one edge
  // type's band (below 2^32: nb * 3 * B * B / 8 bytes per type), and that
  // type's first byte (wave-uniform), so that each load is a uniform base
  // plus a loop-invariant lane offset.
  uint32_t boff[3][NTW];
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int n = 0; n < NTW; ++n)
      boff[s][n] = (uint32_t)(((k * 3 + s) * B + rw + 16 * n + q) * ROWB + g * RB);
  const size_t type_bytes = (size_t)nb * 3 * B * ROWB;
  auto load_bits = [&](int e, WideBits<RB> (&dst)[3][NTW]) __attribute__((always_inline)) {
    const uint8_t* tb = bits + (size_t)e * type_bytes;
#pragma unroll
    for (int s = 0; s < 3; ++s) {
#pragma unroll
      for (int n = 0; n < NTW; ++n) {
        if (s < s_lo || s > s_hi) {
          dst[s][n].zero();
        } else {
          dst[s][n].load(tb + boff[s][n]);
        }
      }
    }
  };

  // Bit rows in the contiguous k order (see WideCfg::KCONT).
  const uint32_t godd = static_cast<uint32_t>(g & 1);
  // Blocks with no edge into the wave's rows stay all zero and are skipped.
  auto reorder_bits = [&](WideBits<RB> (&b)[3][NTW]) __attribute__((always_inline)) {
    if constexpr (C::KCONT) {
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        if (s < s_lo || s > s_hi) continue;
        uint32_t any_bits = 0;
#pragma unroll
        for (int n = 0; n < NTW; ++n)
#pragma unroll
          for (int i = 0; i < WideBits<RB>::NW; ++i) any_bits |= b[s][n].w[i];
        if (!wide_any(any_bits)) continue;
#pragma unroll
        for (int n = 0; n < NTW; ++n) b[s][n].to_contiguous(godd);
      }
    }
  };

  // ---- prologue: slice 0, type 0 ----------------------------------------
  load_bits(0, cur);
  reorder_bits(cur);
#pragma unroll
  for (int h2 = 0; h2 < NH; ++h2)
    for (int u = tid; u < H * 4; u += NT) w_store(u, ws[h2], w_load(u, 0, 0, h2));
  stage_x(0, xs[0], 0);
  __syncthreads();

  f32x4 acc[NTW][MT];
#pragma unroll
  for (int n = 0; n < NTW; ++n)
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[n][m] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Forward tiles: lane (p, g) reads rows 8kk + p/4 (+4) of its group's
  // region; its swizzle is the same for every k step and both reads.
  const int swl = wide_sw<HQ, C::KCONT, GROW>(wide_col0<C::KCONT, GROW>(g, 0) + q / 4);
  int qs = 0, e = 0;     // slice and edge type of iteration it
  int wcur = 0;          // ring buffer of this iteration's first weight unit
  for (int it = 0; it < iters; ++it) {
    const bf16s* xb = xs[C::NXB == 2 ? (qs & 1) : 0];
    const bool more = it + 1 < iters;
    const int en = e + 1 < E ? e + 1 : 0, qn = e + 1 < E ? qs : qs + 1;
    // The next type's bit rows (HBM reads), in flight over this iteration.
    if (more) load_bits(en, nxt);

    // Aggregate of this wave's rows over the slice: P[n][m] = D[feature
    // slot 16m + 4g + j][row 16n + q].
    f32x4 P[NTW][MQ];
#pragma unroll
    for (int n = 0; n < NTW; ++n)
#pragma unroll
      for (int m = 0; m < MQ; ++m) P[n][m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      if (s < s_lo || s > s_hi) continue;
      // A block, or (contiguous k order) a k step, with no edge of this type
      // into the wave's rows adds exact zeros: its expansion and products are
      // skipped (wave-uniform tests; the split order tests whole blocks, in
      // the forward only).
      if constexpr (C::KCONT || !REV) {
        uint32_t any_bits = 0;
#pragma unroll
        for (int n = 0; n < NTW; ++n)
#pragma unroll
          for (int i = 0; i < WideBits<RB>::NW; ++i) any_bits |= cur[s][n].w[i];
        if (!wide_any(any_bits)) continue;
      }
      const bf16s* xsb = xb + s * XS;
#pragma unroll
      for (int kk = 0; kk < RB; ++kk) {
        if constexpr (C::KCONT) {
          uint32_t any_step = 0;
#pragma unroll
          for (int n = 0; n < NTW; ++n) any_step |= cur[s][n].byte(kk);
          if (!wide_any(any_step)) continue;
        }
        bf16x8 bf[NTW];
#pragma unroll
        for (int n = 0; n < NTW; ++n) bf[n] = wide_bits_frag(cur[s][n].byte(kk));
#pragma unroll
        for (int m = 0; m < MQ; ++m) {
          bf16x8 af;
          if constexpr (!REV) {
            af = tr_read8(xsb + (wide_col0<C::KCONT, GROW>(g, kk) + q / 4) * HQ + 16 * (m ^ swl) + 4 * (q % 4), HQ);
          } else {
            af = load_fragi<bf16s>(xsb, kk * MQ + m, lane);
          }
#pragma unroll
          for (int n = 0; n < NTW; ++n) mma(P[n][m], af, bf[n]);
        }
      }
    }

    // A share of the next slice's blocks (double-buffered forms), requested
    // after the aggregation (its LDS reads keep many registers in flight)
    // and in flight during the transform.
    const bool pre_x = C::NXB == 2 && qs + 1 < NQ;
    u32x4 xreg[C::XPT];
    if (pre_x) {
#pragma unroll
      for (int i = 0; i < C::XPT; ++i) {
        const int u = (e * C::XPT + i) * NT + tid;
        if (unit_ok(u)) xreg[i] = unit_load(u, qs + 1);
      }
    }
    // Per-type bias (forward, once per type): deg_e(row) b_e, added with the
    // first unit's products below.
    float fd[NTW];
    if constexpr (BIAS) {
      if (qs == 0) {
#pragma unroll
        for (int n = 0; n < NTW; ++n) {
          int d = cur[0][n].popc() + cur[1][n].popc() + cur[2][n].popc();
          d += __shfl_xor(d, 16);
          d += __shfl_xor(d, 32);
          fd[n] = static_cast<float>(d);
        }
      }
    }

#pragma unroll
    for (int h2 = 0; h2 < NH; ++h2) {
      // The next slice's weight unit h2, in flight during this unit's
      // products.
      u32x4 wreg[C::WPT];
      if (more) {
#pragma unroll
        for (int i = 0; i < C::WPT; ++i) {
          const int u = i * NT + tid;
          if ((H * 4) % NT == 0 || u < H * 4) wreg[i] = w_load(u, qn, en, h2);
        }
      }
      // The lane's eight consecutive features 32 h2 + 8g .. + 7 of the slice,
      // row 16n + q.
      bf16x8 pf[NP][NTW];
#pragma unroll
      for (int n = 0; n < NTW; ++n) {
        float v8[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v8[j] = P[n][2 * h2][j];
          v8[4 + j] = P[n][2 * h2 + 1][j];
        }
        if constexpr (NP == 2) {
          split8(v8, pf[0][n], pf[NP - 1][n]);
        } else {
          pf[0][n] = pack8<bf16s>(v8);
        }
      }
      if constexpr (REV) {
#pragma unroll
        for (int n = 0; n < NTW; ++n)
          *reinterpret_cast<u32x4*>(dM + ((size_t)e * ldm + (size_t)k * B + rw + 16 * n + q) * H + qs * HQ +
                                    32 * h2 + 8 * g) = __builtin_bit_cast(u32x4, pf[0][n]);
      }
      // Transform: acc[n][mo] += (W^T rows 16mo.., features of the unit) x aggregate.
      const int wb = (wcur + h2) % NWB;
#pragma unroll
      for (int mo = 0; mo < MT; ++mo) {
        const bf16x8 wf = load_fragi<bf16s>(ws[wb], mo, lane);
#pragma unroll
        for (int n = 0; n < NTW; ++n)
#pragma unroll
          for (int part = 0; part < NP; ++part) mma(acc[n][mo], wf, pf[part][n]);
        if constexpr (BIAS) {
          if (qs == 0 && h2 == 0) {
            const f32x4 b4 = *reinterpret_cast<const f32x4*>(bias + (size_t)e * H + 16 * mo + 4 * g);
#pragma unroll
            for (int n = 0; n < NTW; ++n)
#pragma unroll
              for (int j = 0; j < 4; ++j) acc[n][mo][j] += fd[n] * b4[j];
          }
        }
      }
      // The next slice's unit h2 goes to the buffer the previous unit used
      // (every wave is past that unit's barrier).
      if (more) {
        bf16s* wn = ws[(wcur + NH + h2) % NWB];
#pragma unroll
        for (int i = 0; i < C::WPT; ++i) {
          const int u = i * NT + tid;
          if ((H * 4) % NT == 0 || u < H * 4) w_store(u, wn, wreg[i]);
        }
      }
      if (h2 == NH - 1 && pre_x) {
#pragma unroll
        for (int i = 0; i < C::XPT; ++i) {
          const int u = (e * C::XPT + i) * NT + tid;
          if (unit_ok(u)) unit_store(u, xs[(qs + 1) & 1], xreg[i]);
        }
      }
      __syncthreads();
    }
    if (e == E - 1 && qs + 1 < NQ) {
      // Units of the next slice not prefetched above (all of them with a
      // single buffer): staged now that every wave is done with this slice.
      const int done = C::NXB == 2 ? E * C::XPT * NT : 0;
      if (done < C::UNITS) {
        stage_x(qs + 1, xs[C::NXB == 2 ? ((qs + 1) & 1) : 0], done);
        __syncthreads();
      }
    }
    if (more) {
#pragma unroll
      for (int s = 0; s < 3; ++s)
#pragma unroll
        for (int n = 0; n < NTW; ++n) cur[s][n] = nxt[s][n];
      reorder_bits(cur);
    }
    qs = qn;
    e = en;
    wcur = (wcur + NH) % NWB;
  }

  // Output rows: lane (q, g) holds features 16m + 4g .. + 3 of row 16n + q.
#pragma unroll
  for (int n = 0; n < NTW; ++n) {
    const size_t row = ((size_t)k * B + rw + 16 * n + q) * H + 4 * g;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      f32x4 v = acc[n][m];
      if (REV && dX_in != nullptr) {
        const f32x4 b = *reinterpret_cast<const f32x4*>(dX_in + row + 16 * m);
        v = f32x4{b[0] + v[0], b[1] + v[1], b[2] + v[2], b[3] + v[3]};
      }
      *reinterpret_cast<f32x4*>(out + row + 16 * m) = v;
    }
  }
}

}  // namespace dev

namespace {
template <int H, int B>
hipError_t wide_launch(bool rev, int n_pad, int E, const void* bits, const void* V, const void* Wsrc,
                       const float* bias, float* out, const float* dX_in, void* dM, long ldm, hipStream_t st) {
  using C = dev::WideCfg<H, B, false>;   // R and NT do not depend on the direction
  const int blocks = (n_pad / B) * (B / C::R);
  const uint8_t* bp = static_cast<const uint8_t*>(bits);
  const dev::bf16s* vp = static_cast<const dev::bf16s*>(V);
  const dev::bf16s* wp = static_cast<const dev::bf16s*>(Wsrc);
  dev::bf16s* mp = static_cast<dev::bf16s*>(dM);
  if (rev)
    hipLaunchKernelGGL((dev::step_wide_kernel<H, B, true, false>), dim3(blocks), dim3(C::NT), 0, st, bp, vp, wp,
                       nullptr, out, n_pad, E, dX_in, mp, ldm);
  else if (bias != nullptr)
    hipLaunchKernelGGL((dev::step_wide_kernel<H, B, false, true>), dim3(blocks), dim3(C::NT), 0, st, bp, vp, wp,
                       bias, out, n_pad, E, nullptr, nullptr, 0L);
  else
    hipLaunchKernelGGL((dev::step_wide_kernel<H, B, false, false>), dim3(blocks), dim3(C::NT), 0, st, bp, vp, wp,
                       nullptr, out, n_pad, E, nullptr, nullptr, 0L);
  return hipGetLastError();
}

template <int H>
hipError_t wide_h(bool rev, int n_pad, int B, int E, const void* bits, const void* V, const void* Wsrc,
                  const float* bias, float* out, const float* dX_in, void* dM, long ldm, hipStream_t st) {
  switch (B) {
    case 32: return wide_launch<H, 32>(rev, n_pad, E, bits, V, Wsrc, bias, out, dX_in, dM, ldm, st);
    case 64: return wide_launch<H, 64>(rev, n_pad, E, bits, V, Wsrc, bias, out, dX_in, dM, ldm, st);
    case 128: return wide_launch<H, 128>(rev, n_pad, E, bits, V, Wsrc, bias, out, dX_in, dM, ldm, st);
    case 256: return wide_launch<H, 256>(rev, n_pad, E, bits, V, Wsrc, bias, out, dX_in, dM, ldm, st);
    case 512: return wide_launch<H, 512>(rev, n_pad, E, bits, V, Wsrc, bias, out, dX_in, dM, ldm, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace

namespace GGNN_IMPL_NS {
bool step_wide_applies(int B, int H) {
#if GGNN_DT_BF16
  return (H == 128 || H == 256) && (B == 32 || B == 64 || B == 128 || B == 256 || B == 512);
#else
  (void)B;
  (void)H;
  return false;
#endif
}

hipError_t launch_step_wide(bool rev, int n_pad, int B, int H, int E, const void* bits, const void* V,
                            const void* Wsrc, const float* bias, float* out, const float* dX_in, void* dM, long ldm,
                            hipStream_t st) {
#if GGNN_DT_BF16
  switch (H) {
    case 128: return wide_h<128>(rev, n_pad, B, E, bits, V, Wsrc, bias, out, dX_in, dM, ldm, st);
    case 256: return wide_h<256>(rev, n_pad, B, E, bits, V, Wsrc, bias, out, dX_in, dM, ldm, st);
  }
#else
  (void)rev, (void)n_pad, (void)B, (void)H, (void)E, (void)bits, (void)V, (void)Wsrc, (void)bias, (void)out;
  (void)dX_in, (void)dM, (void)ldm, (void)st;
#endif
  return hipErrorInvalidValue;
}
}  // namespace GGNN_IMPL_NS

}  // namespace ggnn
