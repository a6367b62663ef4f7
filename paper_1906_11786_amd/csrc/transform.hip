// Message transform M_e = X W_e (+ b_e) and its reverse on gfx950 matrix
// cores (typed form of Eq. 1: one H x H map per edge type).
//
// Layouts: X [n_pad][H] node-major, W [E][H][H] (W[e][h_in][h_out]),
// M [E][H][n_pad] float and dM [E][H][ld] dt (ld >= n_pad), both
// feature-major, dX [n_pad][H] float.
#include "device_common.h"
#include "kernels.h"

#include <type_traits>

namespace ggnn {
namespace dev {

// ---------------------------------------------------------------------------
// Forward.  A workgroup owns 32*WAVES nodes (wave w: 32 of them) for every
// edge type.  D[node][h_out]: A operand = X rows (contiguous in h_in, read
// once from HBM and kept in registers for all E types), B operand = W_e^T
// rows, staged per (e, 64-column chunk) in LDS with the transpose done on
// the LDS write.  Lanes then hold four consecutive nodes of one feature, the
// feature-major store unit of M.  M is kept in fp32 (16-byte stores): it is
// summed over many edges next, and a bf16 copy would add a rounding of the
// same size as the bf16 state itself at every step.
// ---------------------------------------------------------------------------
template <typename S, int H, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void transform_fwd_kernel(const S* __restrict__ X,
                                                                       const S* __restrict__ W,
                                                                       const float* __restrict__ bias,
                                                                       float* __restrict__ M, int n_pad, int E) {
  constexpr int NT = WAVES * kWave;
  constexpr int V = 16 / sizeof(S);
  constexpr int FC = H < 64 ? H : 64;   // output features per LDS chunk
  constexpr int PW = H + V;             // W^T tile pitch
  constexpr int KS = H / 32;
  constexpr int NTL = FC / 16;
  __shared__ __attribute__((aligned(16))) S wt[FC * PW];

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int node0 = xcd_swizzle(blockIdx.x, gridDim.x) * (32 * WAVES) + 32 * wave;
  const bool valid = node0 < n_pad;

  frag_t<S> af[2][KS];
  if (valid) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) af[mt][kk] = load8(X + (size_t)(node0 + 16 * mt + q) * H + 32 * kk + 8 * g);
  }
  for (int e = 0; e < E; ++e) {
    for (int oc = 0; oc < H; oc += FC) {
      __syncthreads();
      const S* wsrc = W + (size_t)e * H * H + oc;
      for (int lin = tid; lin < H * FC / V; lin += NT) {
        int i = lin / (FC / V), o8 = (lin % (FC / V)) * V;
        u32x4 v = *reinterpret_cast<const u32x4*>(wsrc + (size_t)i * H + o8);
        const S* pv = reinterpret_cast<const S*>(&v);
#pragma unroll
        for (int x = 0; x < V; ++x) wt[(o8 + x) * PW + i] = pv[x];
      }
      __syncthreads();
      if (!valid) continue;
      f32x4 acc[2][NTL];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTL; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
#pragma unroll
        for (int nt = 0; nt < NTL; ++nt) {
          frag_t<S> bf = load8(&wt[(16 * nt + q) * PW + 32 * kk + 8 * g]);
          mma(acc[0][nt], af[0][kk], bf);
          mma(acc[1][nt], af[1][kk], bf);
        }
      // D[node = node0 + 16mt + 4g + j][o = oc + 16nt + q]
#pragma unroll
      for (int nt = 0; nt < NTL; ++nt) {
        const int o = oc + 16 * nt + q;
        const float bb = bias ? bias[e * H + o] : 0.f;
        float* out = M + ((size_t)e * H + o) * n_pad + node0 + 4 * g;
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
          store4(out + 16 * mt, acc[mt][nt][0] + bb, acc[mt][nt][1] + bb, acc[mt][nt][2] + bb, acc[mt][nt][3] + bb);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Backward, input gradient: dX_out = dX_in + sum_e dM_e W_e^T (dM rows of
// length ld >= n_pad: one step's slice of a multi-step buffer).
// A workgroup owns 16*WAVES nodes; wave w: 16 nodes, all H input features.
// D[h_in][node]: A operand = W_e rows (contiguous in h_out, tiny, cached),
// B operand = dM_e rows of one node: feature-major dM is staged per type in
// LDS and read with a stride.  Lanes hold four consecutive features of one
// node: 16-byte float stores into node-major dX.
// ---------------------------------------------------------------------------
template <typename S, int H, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void transform_bwd_dx_kernel(const S* __restrict__ W,
                                                                          const S* __restrict__ dM,
                                                                          const float* dX_in, float* dX_out,
                                                                          int n_pad, int E, long ld) {
  constexpr int NT = WAVES * kWave;
  constexpr int V = 16 / sizeof(S);
  constexpr int NW = 16 * WAVES;
  constexpr int PM = NW + 4 / sizeof(S);
  constexpr int KS = H / 32;
  constexpr int MTL = H / 16;
  __shared__ __attribute__((aligned(16))) S tile[H * PM];

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int n0 = xcd_swizzle(blockIdx.x, gridDim.x) * NW;
  const bool valid = n0 + 16 * wave < n_pad;

  f32x4 acc[MTL];
#pragma unroll
  for (int m = 0; m < MTL; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
  constexpr int TU = H * NW / V;                 // 16-byte units of one dM tile
  constexpr int UN = (TU + NT - 1) / NT;
  u32x4 reg[UN];
  auto load_tile = [&](int e) __attribute__((always_inline)) {
    const S* src = dM + (size_t)e * H * ld + n0;
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      const int lin = u * NT + tid;
      const int h = lin / (NW / V), c = (lin % (NW / V)) * V;
      if ((TU % NT == 0 || lin < TU) && n0 + c < n_pad)
        reg[u] = *reinterpret_cast<const u32x4*>(src + (size_t)h * ld + c);
    }
  };
  load_tile(0);
  for (int e = 0; e < E; ++e) {
    __syncthreads();
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      const int lin = u * NT + tid;
      const int h = lin / (NW / V), c = (lin % (NW / V)) * V;
      if ((TU % NT == 0 || lin < TU) && n0 + c < n_pad) {
        uint32_t* p = reinterpret_cast<uint32_t*>(&tile[h * PM + c]);
        p[0] = reg[u].x; p[1] = reg[u].y; p[2] = reg[u].z; p[3] = reg[u].w;
      }
    }
    __syncthreads();
    if (e + 1 < E) load_tile(e + 1);    // in flight during this type's products
    if (!valid) continue;
    const S* we = W + (size_t)e * H * H;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      frag_t<S> bf = load8_strided(&tile[(32 * kk + 8 * g) * PM + 16 * wave + q], PM);
#pragma unroll
      for (int m = 0; m < MTL; ++m) {
        frag_t<S> afr = load8(we + (size_t)(16 * m + q) * H + 32 * kk + 8 * g);
        mma(acc[m], afr, bf);
      }
    }
  }
  if (!valid) return;
  // D[h_in = 16m + 4g + j][node = n0 + 16*wave + q]
  const size_t row = (size_t)(n0 + 16 * wave + q) * H + 4 * g;
#pragma unroll
  for (int m = 0; m < MTL; ++m) {
    f32x4 base = dX_in ? *reinterpret_cast<const f32x4*>(dX_in + row + 16 * m) : f32x4{0.f, 0.f, 0.f, 0.f};
    store4(dX_out + row + 16 * m, base.x + acc[m][0], base.y + acc[m][1], base.z + acc[m][2], base.w + acc[m][3]);
  }
}

// ---------------------------------------------------------------------------
// Backward, weight gradient, one split of the contraction: P[split][e][h_in]
// [h_out] = sum over the split's rows k of X[k][h_in] * dM[e][h_out][k], and
// the bias partial Pb[split][e][h_out] = sum over k of dM[e][h_out][k].  The
// contraction runs over K rows: K = n_pad for one step, or T * n_pad for all
// steps at once (X[t] stacked, dM rows of length ld = T * n_pad holding step
// t at offset t * n_pad).  Workgroup tile TI x TI (TI = min(H, 64)), TI/16
// waves; rows are taken in chunks of 64: X (node-major) is staged in LDS and
// read with a stride, dM (feature-major, contiguous in k) is read directly.
// The tile index runs fastest over the logical workgroup index, so the tiles
// of one split share their X chunks in one XCD's L2.
// ---------------------------------------------------------------------------
template <typename S, int H>
__global__ __launch_bounds__((H < 64 ? H : 64) / 16 * kWave) void transform_wgrad_kernel(
    const S* __restrict__ X, const S* __restrict__ dM, long ld, float* __restrict__ P, float* __restrict__ Pb,
    long K, int E, int rows_per_split) {
  constexpr int TI = H < 64 ? H : 64;
  constexpr int WAVES = TI / 16;
  constexpr int NT = WAVES * kWave;
  constexpr int V = 16 / sizeof(S);
  constexpr int KN = 64;                  // rows per LDS chunk
  constexpr int PX = TI + 4 / sizeof(S);
  constexpr int NTL = TI / 16;
  constexpr int TPD = H / TI;             // tiles per dimension
  __shared__ __attribute__((aligned(16))) S tile[KN * PX];

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  int bid = xcd_swizzle(blockIdx.x, gridDim.x);
  const int to = bid % TPD; bid /= TPD;
  const int ti = bid % TPD; bid /= TPD;
  const int e = bid % E;
  const int split = bid / E;
  const long nlo = (long)split * rows_per_split;
  const long nhi = min(K, nlo + rows_per_split);

  f32x4 acc[NTL];
  float bsum[NTL];
#pragma unroll
  for (int n = 0; n < NTL; ++n) {
    acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    bsum[n] = 0.f;
  }
  const bool do_bias = (ti == 0 && wave == 0 && Pb != nullptr);
  // Software pipeline: the next chunk's X tile and dM fragments are loaded
  // into registers while the current chunk is multiplied.
  constexpr int TU = KN * TI / V;
  constexpr int UN = (TU + NT - 1) / NT;
  u32x4 xr[UN];
  frag_t<S> br[KN / 32][NTL];
  auto load_chunk = [&](long c0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      const int lin = u * NT + tid;
      const int r = lin / (TI / V), c = (lin % (TI / V)) * V;
      if ((TU % NT == 0 || lin < TU) && c0 + r < nhi)
        xr[u] = *reinterpret_cast<const u32x4*>(X + (size_t)(c0 + r) * H + ti * TI + c);
    }
#pragma unroll
    for (int kk = 0; kk < KN / 32; ++kk) {
      if (c0 + 32 * kk >= nhi) break;
#pragma unroll
      for (int n = 0; n < NTL; ++n)
        br[kk][n] = load8(dM + ((size_t)e * H + to * TI + 16 * n + q) * ld + c0 + 32 * kk + 8 * g);
    }
  };
  if (nlo < nhi) load_chunk(nlo);
  for (long c0 = nlo; c0 < nhi; c0 += KN) {
    __syncthreads();
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      const int lin = u * NT + tid;
      const int r = lin / (TI / V), c = (lin % (TI / V)) * V;
      if ((TU % NT == 0 || lin < TU) && c0 + r < nhi) {
        uint32_t* p = reinterpret_cast<uint32_t*>(&tile[r * PX + c]);
        p[0] = xr[u].x; p[1] = xr[u].y; p[2] = xr[u].z; p[3] = xr[u].w;
      }
    }
    frag_t<S> bcur[KN / 32][NTL];
#pragma unroll
    for (int kk = 0; kk < KN / 32; ++kk)
#pragma unroll
      for (int n = 0; n < NTL; ++n) bcur[kk][n] = br[kk][n];
    __syncthreads();
    if (c0 + KN < nhi) load_chunk(c0 + KN);
#pragma unroll
    for (int kk = 0; kk < KN / 32; ++kk) {
      if (c0 + 32 * kk >= nhi) break;    // K and the split length are multiples of 32
      frag_t<S> afr = load8_strided(&tile[(32 * kk + 8 * g) * PX + 16 * wave + q], PX);
#pragma unroll
      for (int n = 0; n < NTL; ++n) {
        mma(acc[n], afr, bcur[kk][n]);
        if (do_bias) {
#pragma unroll
          for (int x = 0; x < 8; ++x) bsum[n] += static_cast<float>(bcur[kk][n][x]);
        }
      }
    }
  }
  // D[h_in = ti*TI + 16*wave + 4g + j][h_out = to*TI + 16n + q]
  float* out = P + ((size_t)split * E + e) * H * H;
#pragma unroll
  for (int n = 0; n < NTL; ++n) {
    const int o = to * TI + 16 * n + q;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      out[(size_t)(ti * TI + 16 * wave + 4 * g + j) * H + o] = acc[n][j];
    }
  }
  if (do_bias) {
#pragma unroll
    for (int n = 0; n < NTL; ++n) {
      float v = bsum[n];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g == 0) Pb[((size_t)split * E + e) * H + to * TI + 16 * n + q] = v;
    }
  }
}

// ---------------------------------------------------------------------------
// Backward, weight gradient with node-major dM (the fused bit-band reverse
// step writes dM_e rows node by node): one split of the rows,
//   P[split][e][h_in][h_out] = sum_k X[k][h_in] * dM[e][k][h_out],
//   Pb[split][e][h_out]      = sum_k dM[e][k][h_out],
// rows k of type e at dM + (e * ldk + k) * H.  A workgroup (NWV waves) owns one
// split of the rows, a group of TE edge types and a slice of IT input
// features: per chunk of KC rows it stages X and the group's dM rows
// node-major in LDS (plain 16-byte copies) and reads them as matrix-core
// fragments with transposing LDS reads, the next chunk's loads in flight.
// Wave w owns the (type, output tile) pairs w, w + NWV, ... of its workgroup,
// each over all IT/16 input tiles.
// ---------------------------------------------------------------------------
#ifndef GGNN_WGRAD_TE64
#define GGNN_WGRAD_TE64 4
#endif
#ifndef GGNN_WGRAD_KC64
#define GGNN_WGRAD_KC64 128
#endif
#ifndef GGNN_WGRAD_WAVES64
#define GGNN_WGRAD_WAVES64 8
#endif
// Edge types per workgroup of the node-major form.
constexpr int wgrad_nm_types(int H, bool f32) {
  return H <= 32 ? 10 : (H == 64 ? GGNN_WGRAD_TE64 : (H == 128 && !f32 ? 2 : 1));
}
template <typename S, int H> struct WgradNmCfg {
  // All input features per workgroup: the stored dM (the large operand) is
  // then read once; the H = 256 fp32 form keeps 64-feature slices.
  static constexpr int IT = (H >= 256 && sizeof(S) == 4) ? 64 : H;   // input features per workgroup
  static constexpr int TE = wgrad_nm_types(H, sizeof(S) == 4);   // types per workgroup
  static constexpr int KC = (sizeof(S) == 4 || H >= 256) ? 64 : (H == 64 ? GGNN_WGRAD_KC64 : 128);   // rows per chunk
  static constexpr int PX = IT + 16, PD = H + 16;                // LDS row pitches (elements)
  static constexpr int NPAIR = TE * H / 16;                      // (type, output tile) pairs
  static constexpr int NWV = (H == 64 && sizeof(S) == 2) ? GGNN_WGRAD_WAVES64 : 8;   // waves per workgroup
  static constexpr int PW = (NPAIR + NWV - 1) / NWV;             // pairs per wave (at most)
  static constexpr int NBUF = 2 * KC * (PX + TE * PD) * (int)sizeof(S) <= 160 * 1024 ? 2 : 1;
};

template <typename S, int H>
__global__ __launch_bounds__(64 * (WgradNmCfg<S, H>::NWV)) void transform_wgrad_nm_kernel(const S* __restrict__ X, const S* __restrict__ dM,
                                                                 long ldk, float* __restrict__ P,
                                                                 float* __restrict__ Pb, long K, int E,
                                                                 int rows_per_split) {
  using C = WgradNmCfg<S, H>;
  constexpr int IT = C::IT, TE = C::TE, KC = C::KC, PX = C::PX, PD = C::PD, PW = C::PW, NBUF = C::NBUF;
  constexpr int NWV = C::NWV, NT = 64 * NWV, NI = IT / 16;
  constexpr int V = 16 / sizeof(S);
  constexpr int NX = KC * IT / V, ND = TE * KC * H / V;   // 16-byte units per chunk
  constexpr int UX = (NX + NT - 1) / NT, UD = (ND + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) S sx[NBUF][KC * PX];
  __shared__ __attribute__((aligned(16))) S sd[NBUF][TE * KC * PD];

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  constexpr int NSL = H / IT;
  const int ngroups = (E + TE - 1) / TE;
  int bid = xcd_swizzle(blockIdx.x, gridDim.x);
  const int sl = bid % NSL; bid /= NSL;
  const int grp = bid % ngroups;
  const int split = bid / ngroups;
  const int e0 = grp * TE, ne = min(TE, E - e0);
  const int i0 = sl * IT;
  const long nlo = (long)split * rows_per_split;
  const long nhi = min(K, nlo + rows_per_split);

  f32x4 acc[PW][NI];
  float bsum[PW];
#pragma unroll
  for (int p = 0; p < PW; ++p) {
    bsum[p] = 0.f;
#pragma unroll
    for (int i = 0; i < NI; ++i) acc[p][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  u32x4 rx[UX], rd[UD];
  auto load_chunk = [&](long c0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < UX; ++u) {
      const int lin = u * NT + tid;
      const long row = c0 + lin / (IT / V);
      const int f = i0 + (lin % (IT / V)) * V;
      rx[u] = ((NX % NT == 0 || lin < NX) && row < nhi) ? *reinterpret_cast<const u32x4*>(X + (size_t)row * H + f)
                                                        : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < UD; ++u) {
      const int lin = u * NT + tid;
      const int te = lin / (KC * H / V), rem = lin % (KC * H / V);
      const long row = c0 + rem / (H / V);
      const int c = (rem % (H / V)) * V;
      rd[u] = ((ND % NT == 0 || lin < ND) && te < ne && row < nhi)
                  ? *reinterpret_cast<const u32x4*>(dM + ((size_t)(e0 + te) * ldk + row) * H + c)
                  : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_chunk = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < UX; ++u) {
      const int lin = u * NT + tid;
      if (NX % NT == 0 || lin < NX)
        *reinterpret_cast<u32x4*>(&sx[buf][(lin / (IT / V)) * PX + (lin % (IT / V)) * V]) = rx[u];
    }
#pragma unroll
    for (int u = 0; u < UD; ++u) {
      const int lin = u * NT + tid;
      if (ND % NT == 0 || lin < ND) {
        const int te = lin / (KC * H / V), rem = lin % (KC * H / V);
        *reinterpret_cast<u32x4*>(&sd[buf][(te * KC + rem / (H / V)) * PD + (rem % (H / V)) * V]) = rd[u];
      }
    }
  };

  // Splits start at multiples of KC rows; a chunk that runs past the split
  // (or a type past E) is zero-filled.
  if (nlo < nhi) load_chunk(nlo);
  int buf = 0;
  for (long c0 = nlo; c0 < nhi; c0 += KC, buf = NBUF == 2 ? buf ^ 1 : 0) {
    if (NBUF == 1 && c0 > nlo) __syncthreads();
    store_chunk(buf);
    __syncthreads();
    if (c0 + KC < nhi) load_chunk(c0 + KC);
#pragma unroll
    for (int k0 = 0; k0 < KC; k0 += 32) {
      if constexpr (NI <= 8) {
        // all X fragments of the k step held, each dM fragment in turn
        frag_t<S> fa[NI];
#pragma unroll
        for (int i = 0; i < NI; ++i) fa[i] = tr_frag(sx[buf], PX, k0, 16 * i, lane);
#pragma unroll
        for (int p = 0; p < PW; ++p) {
          const int pr = wave + NWV * p;
          if (PW * NWV == C::NPAIR || pr < C::NPAIR) {
            const int te = pr / (H / 16), ot = pr % (H / 16);
            const frag_t<S> fb = tr_frag(sd[buf] + te * KC * PD, PD, k0, 16 * ot, lane);
#pragma unroll
            for (int x = 0; x < 8; ++x) bsum[p] += static_cast<float>(fb[x]);
#pragma unroll
            for (int i = 0; i < NI; ++i) mma(acc[p][i], fa[i], fb);
          }
        }
        continue;
      }
      // wide slices: the wave's dM fragments first (few), then each X
      // fragment in turn (holding all X fragments would spill)
      frag_t<S> fb[PW];
#pragma unroll
      for (int p = 0; p < PW; ++p) {
        const int pr = wave + NWV * p;
        if (PW * NWV == C::NPAIR || pr < C::NPAIR) {
          const int te = pr / (H / 16), ot = pr % (H / 16);
          fb[p] = tr_frag(sd[buf] + te * KC * PD, PD, k0, 16 * ot, lane);
#pragma unroll
          for (int x = 0; x < 8; ++x) bsum[p] += static_cast<float>(fb[p][x]);
        }
      }
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const frag_t<S> fa = tr_frag(sx[buf], PX, k0, 16 * i, lane);
#pragma unroll
        for (int p = 0; p < PW; ++p) {
          const int pr = wave + NWV * p;
          if (PW * NWV == C::NPAIR || pr < C::NPAIR) mma(acc[p][i], fa, fb[p]);
        }
      }
    }
  }
  // D[h_in = i0 + 16 i + 4g + j][h_out = 16 ot + q] of type e0 + te
#pragma unroll
  for (int p = 0; p < PW; ++p) {
    const int pr = wave + NWV * p;
    if (!(PW * NWV == C::NPAIR || pr < C::NPAIR)) continue;
    const int te = pr / (H / 16), ot = pr % (H / 16);
    if (te >= ne) continue;
    float* out = P + ((size_t)split * E + e0 + te) * H * H;
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) out[(size_t)(i0 + 16 * i + 4 * g + j) * H + 16 * ot + q] = acc[p][i][j];
    if (Pb != nullptr && sl == 0) {
      float v = bsum[p];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g == 0) Pb[((size_t)split * E + e0 + te) * H + 16 * ot + q] = v;
    }
  }
}

}  // namespace dev

#if GGNN_DT_BF16   // dtype-independent kernels: built once
// out[i] += sum_{s < nsplit} part[s * stride + i] for i < count.  A
// workgroup of 64 x RW threads owns 64 V consecutive outputs: thread (x, y)
// sums, for its V outputs, the splits s = y, y + RW, y + 2RW, ... in
// increasing order (eight loads in flight), then thread (x, 0) adds the RW
// sums in order y = 0..RW-1.  The order depends only on nsplit, so results do
// not depend on scheduling, and V = 4 (16-byte loads; count, stride and both
// pointers must be multiples of four floats) gives the same bits as V = 1.
constexpr int kReduceRW = 16;
template <int V>
__device__ __forceinline__ void reduce_block(const float* __restrict__ part, float* __restrict__ out, int nsplit,
                                             int count, long stride, int blk) {
  using T = std::conditional_t<V == 4, dev::f32x4, float>;
  constexpr int RW = kReduceRW;
  __shared__ T red[RW][64];
  const int x = threadIdx.x % 64, y = threadIdx.x / 64;
  const int i = (blk * 64 + x) * V;
  T s = {};
  if (i < count) {
    int k = y;
    for (; k + 7 * RW < nsplit; k += 8 * RW) {
      T v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = *reinterpret_cast<const T*>(part + (size_t)(k + j * RW) * stride + i);
#pragma unroll
      for (int j = 0; j < 8; ++j) s += v[j];
    }
    for (; k < nsplit; k += RW) s += *reinterpret_cast<const T*>(part + (size_t)k * stride + i);
  }
  red[y][x] = s;
  __syncthreads();
  if (y == 0 && i < count) {
    T t = {};
#pragma unroll
    for (int w = 0; w < RW; ++w) t += red[w][x];
    T* o = reinterpret_cast<T*>(out + i);
    *o = *o + t;
  }
}

__global__ __launch_bounds__(64 * kReduceRW) void reduce_partials_kernel(const float* __restrict__ part,
                                                                         float* __restrict__ out, int nsplit,
                                                                         int count, long stride) {
  reduce_block<1>(part, out, nsplit, count, stride, blockIdx.x);
}

// Several reductions in one launch (the weight-gradient partials of one
// reverse pass): block b works for the segment whose block range holds it.
struct ReduceMulti {
  ReduceSeg seg[ReduceList::kMax];
  int first[ReduceList::kMax + 1];
  int vec[ReduceList::kMax];   // 4: the segment meets the 16-byte conditions of reduce_block<4>
  int n;
};
__global__ __launch_bounds__(64 * kReduceRW) void reduce_multi_kernel(ReduceMulti m) {
  const int b = blockIdx.x;
  int si = 0;
  while (si + 1 < m.n && b >= m.first[si + 1]) ++si;
  const ReduceSeg sg = m.seg[si];
  if (m.vec[si] == 4) {
    reduce_block<4>(sg.part, sg.out, sg.nsplit, sg.count, sg.stride, b - m.first[si]);
  } else {
    reduce_block<1>(sg.part, sg.out, sg.nsplit, sg.count, sg.stride, b - m.first[si]);
  }
}

hipError_t launch_reduce_multi(const ReduceList& l, hipStream_t st) {
  if (l.n == 0) return hipSuccess;
  ReduceMulti m{};
  m.n = l.n;
  m.first[0] = 0;
  for (int i = 0; i < l.n; ++i) {
    const ReduceSeg& sg = l.seg[i];
    m.seg[i] = sg;
    const bool v4 = sg.count % 4 == 0 && sg.stride % 4 == 0 && reinterpret_cast<uintptr_t>(sg.part) % 16 == 0 &&
                    reinterpret_cast<uintptr_t>(sg.out) % 16 == 0;
    m.vec[i] = v4 ? 4 : 1;
    m.first[i + 1] = m.first[i] + (sg.count + 64 * m.vec[i] - 1) / (64 * m.vec[i]);
  }
  hipLaunchKernelGGL(reduce_multi_kernel, dim3(m.first[l.n]), dim3(64 * kReduceRW), 0, st, m);
  return hipGetLastError();
}

hipError_t reduce_or_defer(const float* part, float* out, int nsplit, int count, long stride, ReduceList* defer,
                           hipStream_t st) {
  if (count <= 0) return hipSuccess;
  if (defer != nullptr && defer->n < ReduceList::kMax) {
    defer->seg[defer->n++] = ReduceSeg{part, out, nsplit, count, stride};
    return hipSuccess;
  }
  return launch_reduce_partials(part, out, nsplit, count, stride, st);
}

// Zero-fill with a kernel (not hipMemsetAsync, so the launch can sit inside a
// captured HIP graph).  p is 16-byte aligned.
__global__ void fill_zero_kernel(float* __restrict__ p, size_t count) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (4 * i + 3 < count) {
    reinterpret_cast<float4*>(p)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  } else {
    for (size_t k = 4 * i; k < count; ++k) p[k] = 0.f;
  }
}

hipError_t launch_fill_zero(float* p, size_t count, hipStream_t st) {
  if (count == 0) return hipSuccess;
  const size_t n4 = (count + 3) / 4;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, st, p, count);
  return hipGetLastError();
}

hipError_t launch_reduce_partials(const float* part, float* out, int nsplit, int count, long stride,
                                  hipStream_t st) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(reduce_partials_kernel, dim3((count + 63) / 64), dim3(64 * kReduceRW), 0, st, part, out, nsplit,
                     count, stride);
  return hipGetLastError();
}

#endif

namespace {
// Row split of the weight-gradient contraction: about 2048 workgroups over
// all tiles (several waves per SIMD to hide the memory latency of the chunk
// loop), each split a multiple of 64 rows and at least GGNN_WGRAD_MIN_ROWS,
// so the partial slices stay small next to the rows they summarise.
#ifndef GGNN_WGRAD_MIN_ROWS
#define GGNN_WGRAD_MIN_ROWS 1024
#endif
struct Split {
  int nsplit, per;
};
Split transform_split(long K, int H, int E) {
  const long TI = H < 64 ? H : 64;
  const long tiles = E * (H / TI) * (H / TI);
  const long want = (2048 + tiles - 1) / tiles;
  long per = ((K + want - 1) / want + 63) / 64 * 64;
  if (per < GGNN_WGRAD_MIN_ROWS) per = GGNN_WGRAD_MIN_ROWS;
  return {(int)((K + per - 1) / per), (int)per};
}

// Node-major form: about 256 workgroups (one per compute unit, 8 waves
// each) over splits x type groups x input slices (fp32 at H = 256 only);
// splits are multiples of 128 rows.
#ifndef GGNN_WGRAD_NM_WGS
#define GGNN_WGRAD_NM_WGS 256
#endif
Split transform_nm_split(long K, int H, int E, int te, bool f32) {
  const long per_split = ((E + te - 1) / te) * (H >= 256 && f32 ? H / 64 : 1);
  const long want = GGNN_WGRAD_NM_WGS / per_split > 0 ? GGNN_WGRAD_NM_WGS / per_split : 1;
  long per = ((K + want - 1) / want + 127) / 128 * 128;
  return {(int)((K + per - 1) / per), (int)per};
}

template <typename S, int H>
hipError_t transform_fwd_h(int n_pad, int E, const void* X, const void* W, const float* bias, float* M,
                           hipStream_t st) {
  const S* xp = static_cast<const S*>(X);
  const S* wp = static_cast<const S*>(W);
  float* mp = M;
  const int tiles4 = (n_pad + 127) / 128;
  if (tiles4 >= 1024) {
    hipLaunchKernelGGL((dev::transform_fwd_kernel<S, H, 4>), dim3(tiles4), dim3(256), 0, st, xp, wp, bias, mp, n_pad, E);
  } else {
    hipLaunchKernelGGL((dev::transform_fwd_kernel<S, H, 2>), dim3((n_pad + 63) / 64), dim3(128), 0, st, xp, wp, bias,
                       mp, n_pad, E);
  }
  return hipGetLastError();
}

template <typename S, int H>
hipError_t transform_dx_h(int n_pad, int E, const void* W, const void* dM, long ld, const float* dX_in,
                          float* dX_out, hipStream_t st) {
  hipLaunchKernelGGL((dev::transform_bwd_dx_kernel<S, H, 4>), dim3((n_pad + 63) / 64), dim3(256), 0, st,
                     static_cast<const S*>(W), static_cast<const S*>(dM), dX_in, dX_out, n_pad, E, ld);
  return hipGetLastError();
}

template <typename S, int H>
hipError_t transform_wgrad_h(long K, int E, const void* X, const void* dM, long ld, float* dW, float* dbias, void* ws,
                             hipStream_t st) {
  Split sp = transform_split(K, H, E);
  constexpr int TI = H < 64 ? H : 64;
  float* P = static_cast<float*>(ws);
  float* Pb = dbias ? P + (size_t)sp.nsplit * E * H * H : nullptr;
  const int blocks = sp.nsplit * E * (H / TI) * (H / TI);
  hipLaunchKernelGGL((dev::transform_wgrad_kernel<S, H>), dim3(blocks), dim3(TI / 16 * 64), 0, st,
                     static_cast<const S*>(X), static_cast<const S*>(dM), ld, P, Pb, K, E, sp.per);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  err = launch_reduce_partials(P, dW, sp.nsplit, E * H * H, (long)E * H * H, st);
  if (err != hipSuccess || !dbias) return err;
  return launch_reduce_partials(Pb, dbias, sp.nsplit, E * H, (long)E * H, st);
}

#ifndef GGNN_WGRAD256_WIDE
#define GGNN_WGRAD256_WIDE 1
#endif
template <typename S, int H>
hipError_t transform_wgrad_nm_h(long K, int E, const void* X, const void* dM, long ldk, float* dW, float* dbias,
                                void* ws, ReduceList* defer, hipStream_t st) {
  using C = dev::WgradNmCfg<S, H>;
  Split sp = transform_nm_split(K, H, E, C::TE, sizeof(S) == 4);
  float* P = static_cast<float*>(ws);
  float* Pb = dbias ? P + (size_t)sp.nsplit * E * H * H : nullptr;
  hipError_t err;
  if (GGNN_WGRAD256_WIDE && H == 256 && sizeof(S) == 2 && C::TE == 1) {
    err = launch_transform_wgrad_nm256(sp.nsplit, sp.per, K, E, X, dM, ldk, P, Pb, st);   // same split
  } else {
    const int blocks = sp.nsplit * ((E + C::TE - 1) / C::TE) * (H / C::IT);
    hipLaunchKernelGGL((dev::transform_wgrad_nm_kernel<S, H>), dim3(blocks), dim3(64 * C::NWV), 0, st,
                       static_cast<const S*>(X), static_cast<const S*>(dM), ldk, P, Pb, K, E, sp.per);
    err = hipGetLastError();
  }
  if (err != hipSuccess) return err;
  err = reduce_or_defer(P, dW, sp.nsplit, E * H * H, (long)E * H * H, defer, st);
  if (err != hipSuccess || !dbias) return err;
  return reduce_or_defer(Pb, dbias, sp.nsplit, E * H, (long)E * H, defer, st);
}

template <typename S>
hipError_t transform_wgrad_nm_t(long K, int H, int E, const void* X, const void* dM, long ldk, float* dW,
                                float* dbias, void* ws, ReduceList* defer, hipStream_t st) {
  switch (H) {
    case 32: return transform_wgrad_nm_h<S, 32>(K, E, X, dM, ldk, dW, dbias, ws, defer, st);
    case 64: return transform_wgrad_nm_h<S, 64>(K, E, X, dM, ldk, dW, dbias, ws, defer, st);
    case 128: return transform_wgrad_nm_h<S, 128>(K, E, X, dM, ldk, dW, dbias, ws, defer, st);
    case 256: return transform_wgrad_nm_h<S, 256>(K, E, X, dM, ldk, dW, dbias, ws, defer, st);
  }
  return hipErrorInvalidValue;
}

template <typename S>
hipError_t transform_fwd_t(int n_pad, int H, int E, const void* X, const void* W, const float* bias, float* M,
                           hipStream_t st) {
  switch (H) {
    case 32: return transform_fwd_h<S, 32>(n_pad, E, X, W, bias, M, st);
    case 64: return transform_fwd_h<S, 64>(n_pad, E, X, W, bias, M, st);
    case 128: return transform_fwd_h<S, 128>(n_pad, E, X, W, bias, M, st);
    case 256: return transform_fwd_h<S, 256>(n_pad, E, X, W, bias, M, st);
  }
  return hipErrorInvalidValue;
}
template <typename S>
hipError_t transform_dx_t(int n_pad, int H, int E, const void* W, const void* dM, long ld, const float* dX_in,
                          float* dX_out, hipStream_t st) {
  switch (H) {
    case 32: return transform_dx_h<S, 32>(n_pad, E, W, dM, ld, dX_in, dX_out, st);
    case 64: return transform_dx_h<S, 64>(n_pad, E, W, dM, ld, dX_in, dX_out, st);
    case 128: return transform_dx_h<S, 128>(n_pad, E, W, dM, ld, dX_in, dX_out, st);
    case 256: return transform_dx_h<S, 256>(n_pad, E, W, dM, ld, dX_in, dX_out, st);
  }
  return hipErrorInvalidValue;
}
template <typename S>
hipError_t transform_wgrad_t(long K, int H, int E, const void* X, const void* dM, long ld, float* dW, float* dbias,
                             void* ws, hipStream_t st) {
  switch (H) {
    case 32: return transform_wgrad_h<S, 32>(K, E, X, dM, ld, dW, dbias, ws, st);
    case 64: return transform_wgrad_h<S, 64>(K, E, X, dM, ld, dW, dbias, ws, st);
    case 128: return transform_wgrad_h<S, 128>(K, E, X, dM, ld, dW, dbias, ws, st);
    case 256: return transform_wgrad_h<S, 256>(K, E, X, dM, ld, dW, dbias, ws, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace

#if GGNN_DT_BF16
size_t transform_wgrad_workspace(long K, int H, int E) {
  // large enough for both forms (feature-major and node-major dM)
  const Split a = transform_split(K, H, E), b = transform_nm_split(K, H, E, dev::wgrad_nm_types(H, false), false),
              c = transform_nm_split(K, H, E, dev::wgrad_nm_types(H, true), true);
  size_t n = (size_t)(a.nsplit > b.nsplit ? a.nsplit : b.nsplit);
  if ((size_t)c.nsplit > n) n = (size_t)c.nsplit;
  return (n * E * H * H + n * E * H) * sizeof(float);
}
#endif

namespace GGNN_IMPL_NS {
hipError_t launch_transform_fwd(int n_pad, int H, int E, const void* X, const void* W, const float* bias, float* M,
                                hipStream_t st) {
  return transform_fwd_t<dev::dt_t>(n_pad, H, E, X, W, bias, M, st);
}

hipError_t launch_transform_bwd_dx(int n_pad, int H, int E, const void* W, const void* dM, long ld,
                                   const float* dX_in, float* dX_out, hipStream_t st) {
  return transform_dx_t<dev::dt_t>(n_pad, H, E, W, dM, ld, dX_in, dX_out, st);
}

hipError_t launch_transform_wgrad(long K, int H, int E, const void* X, const void* dM, long ld, float* dW,
                                  float* dbias, void* ws, hipStream_t st) {
  return transform_wgrad_t<dev::dt_t>(K, H, E, X, dM, ld, dW, dbias, ws, st);
}

hipError_t launch_transform_wgrad_nm(long K, int H, int E, const void* X, const void* dM, long ldk, float* dW,
                                     float* dbias, void* ws, ReduceList* defer, hipStream_t st) {
  return transform_wgrad_nm_t<dev::dt_t>(K, H, E, X, dM, ldk, dW, dbias, ws, defer, st);
}
}  // namespace GGNN_IMPL_NS

}  // namespace ggnn
