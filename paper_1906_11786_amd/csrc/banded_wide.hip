// Wide fused step on a 1-bit block band (bf16 storage, H >= 128, blocks too
// large to stage whole): the products of the fused step of Eq. 3 in the
// operand order of Algorithm 1,
//   forward:  a[k]    = sum_e (sum_s bits[e][k][s] X[k-1+s]) W_e   (+ deg_e b_e)
//   reverse:  dM_e[k] = sum_s bits_t[e][k][s] da[k-1+s]            (stored)
//             dX[k]   = dX_in[k] + sum_e dM_e[k] W_e^T
// arranged so that every operand staged in LDS feeds several matrix-core
// steps and the node blocks are staged once per workgroup, not per edge type.
//
// The transform's contraction over features is split into slices of
// HQ = 32 features:  (A_e X) W_e = sum_q (A_e X[:, q]) W_e[q, :].
// For each slice q the workgroup stages features q of the three node blocks
// (k-1, k, k+1) once; every edge type then reuses them.  Per type a wave
// aggregates its 32 rows over the slice (registers, 32 x 32), and multiplies
// that into its output accumulators (32 rows x H, registers) with rows q of
// W_e (reverse) or of W_e^T (forward), which the workgroup stages per
// (slice, type) in LDS in fragment order.  The next (slice, type)'s weights
// and a share of the next slice's node blocks are loaded at the top of each
// (slice, type) and written to the other LDS buffer at its end: one barrier
// per (slice, type), none inside the products.
//
// LDS layouts of a staged block slice (B nodes x 32 features):
//   forward (X node-major in HBM): node rows of 32 features, the node range
//     split into four lane-group regions (lane group g owns block columns
//     [gB/4, (g+1)B/4) in the k order of the aggregation) separated by 32
//     bytes, so the two 16-lane halves of a transposing read hit disjoint
//     banks; read with ds_read_b64_tr_b16, which hands a lane eight
//     consecutive nodes of one feature.  Feature f of the slice sits in
//     column 16 (f % 8 / 4) + 4 (f / 8) + f % 4: the aggregate's tiles 0 and
//     1 then give a lane eight consecutive features (the weight fragments are
//     16-byte rows; the reverse stores dM with one 16-byte write).
//   reverse (da feature-major in HBM): fragment order (a fragment's 64 lane
//     vectors contiguous, 16-byte copies), features in the same permuted
//     order.
#include "device_common.h"
#include "kernels.h"

namespace ggnn {
namespace dev {

template <int H, int B>
struct WideCfg {
  static constexpr int HQ = 32;                  // features per slice
  static constexpr int NQ = H / HQ;
  static constexpr int RPW = 32, NTW = 2;        // rows per wave, 16-row tiles per wave
  static constexpr int WAVES = B / RPW < 8 ? B / RPW : 8;
  static constexpr int R = WAVES * RPW;          // rows per workgroup
  static constexpr int NT = WAVES * kWave;
  static constexpr int RB = B / 32;              // bit-row bytes per lane and block
  static constexpr int GROW = B / 4;             // block columns per lane group
  static constexpr int PADG = 16;                // elements between lane-group regions (forward)
  static constexpr int GS = GROW * HQ + PADG;    // elements per lane-group region (forward)
  static constexpr int XS = B * HQ + 4 * PADG;   // elements per staged block slice
  static constexpr int WS = (H / 16) * kWave * 8;   // elements per staged weight slice
  static constexpr int NXB = (2 * 3 * XS + 2 * WS) * 2 <= 160 * 1024 ? 2 : 1;   // block-slice buffers
  static constexpr int UNITS = 3 * B * HQ / 8;   // 16-byte units of one slice of the three blocks
  static constexpr int XPT = 2;                  // of which each thread prefetches per (slice, type)
  static constexpr int WPT = (H * 4 + NT - 1) / NT;   // weight units per thread per (slice, type)
};

// Feature f (0..31) of a slice -> its column in a forward node row.
__device__ __forceinline__ int wide_col(int f) { return 16 * ((f % 8) / 4) + 4 * (f / 8) + f % 4; }
// Feature f of a slice -> its (tile, row) slot, as 16 * tile + row.
__device__ __forceinline__ int wide_slot(int f) { return wide_col(f); }

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

template <int NB> struct WideBits {
  static constexpr int NW = NB / 4;
  uint32_t w[NW];
  __device__ __forceinline__ void load(const uint8_t* p) {
    if constexpr (NB == 4) {
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
__global__ __launch_bounds__((WideCfg<H, B>::NT)) void step_wide_kernel(
    const uint8_t* __restrict__ bits, const bf16s* __restrict__ V, const bf16s* __restrict__ Wsrc,
    const float* __restrict__ bias, float* __restrict__ out, int n_pad, int E, const float* __restrict__ dX_in,
    bf16s* __restrict__ dM, long ldm) {
  using C = WideCfg<H, B>;
  constexpr int NT = C::NT, HQ = C::HQ, NQ = C::NQ, NTW = C::NTW, RB = C::RB, XS = C::XS, GS = C::GS;
  constexpr int MT = H / 16;             // 16-feature output tiles
  constexpr int NP = REV ? 1 : 2;        // forward: the aggregate enters the transform as bf16 hi + lo
  constexpr int ROWB = B / 8;
  constexpr int UB = C::UNITS / 3;       // units per block
  constexpr int TPR = B / C::R;
  __shared__ __attribute__((aligned(16))) bf16s xs[C::NXB][3 * XS];
  __shared__ __attribute__((aligned(16))) bf16s ws[2][C::WS];

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
  // Unit u of slice qs, block s = u / UB.  Forward: node c = r / 4 of the
  // block, features qs*HQ + 8G .. 8G + 7 (G = r % 4); reverse: feature
  // f = 16 (r / (16 B/8)) + r % 16, nodes 8 c8 .. 8 c8 + 7 (c8 = (r / 16) %
  // (B/8)).  Units of a block outside the matrix are skipped.
  auto unit_ok = [&](int u) __attribute__((always_inline)) {
    const int s = u / UB;
    return u < C::UNITS && s >= s_lo && s <= s_hi;
  };
  auto unit_load = [&](int u, int qs) __attribute__((always_inline)) {
    const int s = u / UB, r = u % UB;
    const bf16s* p;
    if constexpr (!REV) {
      p = V + (size_t)((k - 1 + s) * B + r / 4) * H + qs * HQ + 8 * (r % 4);
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
      const int c = r / 4, G = r % 4;
      bf16s* row = d + (c / C::GROW) * GS + (c % C::GROW) * HQ;
      *reinterpret_cast<u32x2*>(row + 4 * G) = u32x2{v[0], v[1]};        // features 8G .. 8G+3
      *reinterpret_cast<u32x2*>(row + 16 + 4 * G) = u32x2{v[2], v[3]};   // features 8G+4 .. 8G+7
    } else {
      const int f = 16 * (r / (16 * (B / 8))) + r % 16, c = 8 * ((r / 16) % (B / 8));
      // fragment (kk, tile) of the block: lane group c / (B/4), k step (c % (B/4)) / 8
      const int slot = wide_slot(f), gg = c / C::GROW, kk = (c % C::GROW) / 8;
      *reinterpret_cast<u32x4*>(d + fo<bf16s>(kk * 2 + slot / 16, slot % 16 + 16 * gg, 0)) = v;
    }
  };
  auto stage_x = [&](int qs, bf16s* xb, int u0) __attribute__((always_inline)) {
    for (int u = u0 + tid; u < C::UNITS; u += NT)
      if (unit_ok(u)) unit_store(u, xb, unit_load(u, qs));
  };
  // Weight unit u of (slice qs, type e): output row o = u / 4, slice
  // features 8G .. 8G + 7 (G = u % 4): one fragment vector.
  auto w_load = [&](int u, int qs, int e) __attribute__((always_inline)) {
    return *reinterpret_cast<const u32x4*>(Wsrc + (size_t)e * H * H + (size_t)(u / 4) * H + qs * HQ + 8 * (u % 4));
  };
  auto w_store = [&](int u, bf16s* wb, const u32x4& v) __attribute__((always_inline)) {
    const int o = u / 4, G = u % 4;
    *reinterpret_cast<u32x4*>(wb + fo<bf16s>(o / 16, o % 16 + 16 * G, 0)) = v;
  };

  // ---- bit rows ---------------------------------------------------------
  WideBits<RB> cur[3][NTW], nxt[3][NTW];
  auto load_bits = [&](int e, WideBits<RB> (&dst)[3][NTW]) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < 3; ++s) {
#pragma unroll
      for (int n = 0; n < NTW; ++n) {
        if (s < s_lo || s > s_hi) {
          dst[s][n].zero();
        } else {
          dst[s][n].load(bits + ((((size_t)e * nb + k) * 3 + s) * B + rw + 16 * n + q) * ROWB + g * RB);
        }
      }
    }
  };

  // ---- prologue: slice 0, type 0 ----------------------------------------
  load_bits(0, cur);
  for (int u = tid; u < H * 4; u += NT) w_store(u, ws[0], w_load(u, 0, 0));
  stage_x(0, xs[0], 0);
  __syncthreads();

  f32x4 acc[NTW][MT];
#pragma unroll
  for (int n = 0; n < NTW; ++n)
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[n][m] = f32x4{0.f, 0.f, 0.f, 0.f};

  int qs = 0, e = 0;   // slice and edge type of iteration it
  for (int it = 0; it < iters; ++it) {
    const bf16s* xb = xs[C::NXB == 2 ? (qs & 1) : 0];
    const bf16s* wb = ws[it & 1];
    const bool more = it + 1 < iters;
    const int en = e + 1 < E ? e + 1 : 0, qn = e + 1 < E ? qs : qs + 1;
    // Aggregate of this wave's rows over the slice: P[n][m] = D[feature
    // slot 16m + 4g + j][row 16n + q].
    f32x4 P[NTW][2];
#pragma unroll
    for (int n = 0; n < NTW; ++n)
#pragma unroll
      for (int m = 0; m < 2; ++m) P[n][m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      if (s < s_lo || s > s_hi) continue;
      const bf16s* xsb = xb + s * XS;
#pragma unroll
      for (int kk = 0; kk < RB; ++kk) {
        bf16x8 bf[NTW];
#pragma unroll
        for (int n = 0; n < NTW; ++n) bf[n] = wide_bits_frag(cur[s][n].byte(kk));
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          bf16x8 af;
          if constexpr (!REV) {
            af = tr_read8(xsb + g * GS + (8 * kk + q / 4) * HQ + 16 * m + 4 * (q % 4), HQ);
          } else {
            af = load_fragi<bf16s>(xsb, kk * 2 + m, lane);
          }
#pragma unroll
          for (int n = 0; n < NTW; ++n) mma(P[n][m], af, bf[n]);
        }
      }
    }
    // Next (slice, type): weights and bit rows; a share of the next slice's
    // blocks (double-buffered forms).  Requested after the aggregation (its
    // LDS reads keep many registers in flight), in flight during the
    // transform.
    u32x4 wreg[C::WPT];
    if (more) {
#pragma unroll
      for (int i = 0; i < C::WPT; ++i) {
        const int u = i * NT + tid;
        if ((H * 4) % NT == 0 || u < H * 4) wreg[i] = w_load(u, qn, en);
      }
      load_bits(en, nxt);
    }
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
    // slice-0 transform below.
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
    // The lane's eight consecutive slice features 8g .. 8g + 7 of row 16n + q.
    bf16x8 pf[NP][NTW];
#pragma unroll
    for (int n = 0; n < NTW; ++n) {
      float v8[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v8[j] = P[n][0][j];
        v8[4 + j] = P[n][1][j];
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
        *reinterpret_cast<u32x4*>(dM + ((size_t)e * ldm + (size_t)k * B + rw + 16 * n + q) * H + qs * HQ + 8 * g) =
            __builtin_bit_cast(u32x4, pf[0][n]);
    }
    // Transform: acc[n][mo] += W^T rows 16mo.. (slice features) x aggregate.
#pragma unroll
    for (int mo = 0; mo < MT; ++mo) {
      const bf16x8 wf = load_fragi<bf16s>(wb, mo, lane);
#pragma unroll
      for (int n = 0; n < NTW; ++n)
#pragma unroll
        for (int part = 0; part < NP; ++part) mma(acc[n][mo], wf, pf[part][n]);
      if constexpr (BIAS) {
        if (qs == 0) {
          const f32x4 b4 = *reinterpret_cast<const f32x4*>(bias + (size_t)e * H + 16 * mo + 4 * g);
#pragma unroll
          for (int n = 0; n < NTW; ++n)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[n][mo][j] += fd[n] * b4[j];
        }
      }
    }

    // Hand the prefetched operands to the other buffers.
    if (more) {
#pragma unroll
      for (int i = 0; i < C::WPT; ++i) {
        const int u = i * NT + tid;
        if ((H * 4) % NT == 0 || u < H * 4) w_store(u, ws[(it + 1) & 1], wreg[i]);
      }
    }
    if (pre_x) {
#pragma unroll
      for (int i = 0; i < C::XPT; ++i) {
        const int u = (e * C::XPT + i) * NT + tid;
        if (unit_ok(u)) unit_store(u, xs[(qs + 1) & 1], xreg[i]);
      }
    }
    __syncthreads();
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
    }
    qs = qn;
    e = en;
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
  using C = dev::WideCfg<H, B>;
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
  return (H == 128 || H == 256) && (B == 128 || B == 256 || B == 512);
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
