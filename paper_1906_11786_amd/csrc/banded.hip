// Banded block contraction on gfx950 matrix cores: the three batched block
// products of Eq. 3 (Algorithm 1's three einsums over Cks, Uks, Lks) and
// their transpose.
//
// Layouts: band[e][k][s][r][c] (s = 0: block column k-1, 1: k, 2: k+1; r the
// receiver row, c the sender column), M feature-major [E][H][n_pad] float,
// dM feature-major [E][H][n_pad] dt, a node-major [n_pad][H] float, da
// feature-major [H][n_pad] dt.
#include "device_common.h"
#include "kernels.h"

namespace ggnn {
namespace dev {

// ---------------------------------------------------------------------------
// Forward: a[k*B + r][h] = sum_e sum_s sum_c band[e][k][s][r][c] * M[e][h][(k-1+s)*B + c]
//
// One workgroup owns NW = 32*WAVES consecutive rows of one block row k and
// all H features; wave w owns 32 rows.  Tile orientation D[h][r]: the A
// operand is M (rows h, from LDS; in bf16 mode each float is staged as a
// bf16 pair hi + lo with hi + lo = M to 16 bits, and both parts go through
// the matrix cores, so the products keep fp32-level accuracy while the band
// stays bf16), the B operand is the band (rows r, loaded
// straight from HBM into registers: the band is streamed exactly once and
// never shared between waves).  Each lane then holds four consecutive
// features of one node, so `a` is written with 16-byte stores.
// The contraction runs over chunks (e, s, c0..c0+KC); inside a chunk lane
// group g owns the contiguous columns [g*KC/4, (g+1)*KC/4), so every lane
// reads one contiguous run of its band row.
// ---------------------------------------------------------------------------
template <typename S, int H, int WAVES, int KC>
__global__ __launch_bounds__(WAVES * kWave) void banded_fwd_kernel(const S* __restrict__ band,
                                                                    const float* __restrict__ M,
                                                                    float* __restrict__ a, int n_pad, int B,
                                                                    int E) {
  constexpr int NT = WAVES * kWave;          // threads
  constexpr int V = 16 / sizeof(S);          // elements of S per 16-byte unit
  constexpr int LDP = KC + V;                // LDS row pitch (elements), 16-byte aligned, staggered banks
  constexpr int TU = H * KC / 4;             // 16-byte (4 float) units of one M chunk
  constexpr int UNITS = (TU + NT - 1) / NT;  // per thread
  constexpr int KS = KC / 32;                // 32-wide k steps per chunk
  constexpr int MT = H / 16;                 // feature tiles
  constexpr int RUN = KC / 4;                // band elements per lane per chunk and row
  constexpr int NP = sizeof(S) == 2 ? 2 : 1; // bf16: M enters the matrix cores as hi + lo parts
  __shared__ __attribute__((aligned(16))) S lds[2][NP][H * LDP];

  const int nb = n_pad / B;
  const int NW = 32 * WAVES;
  const int tiles_per_row = B / NW;
  const int t = xcd_swizzle(blockIdx.x, gridDim.x);
  const int k = t / tiles_per_row;
  const int r0 = (t % tiles_per_row) * NW;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int rw = r0 + 32 * wave;             // first row of this wave

  const int s_lo = (k == 0) ? 1 : 0;
  const int s_hi = (k == nb - 1) ? 1 : 2;
  const int ns = s_hi - s_lo + 1;
  const int cpb = B / KC;                    // chunks per block
  const int nq = E * ns * cpb;

  auto chunk = [&](int qi, int& e, int& s, int& c0) __attribute__((always_inline)) {
    e = qi / (ns * cpb);
    int rem = qi % (ns * cpb);
    s = s_lo + rem / cpb;
    c0 = (rem % cpb) * KC;
  };

  f32x4 mreg[UNITS];
  frag_t<S> bcur[2][KS], bnext[2][KS];

  auto load_m = [&](int qi) __attribute__((always_inline)) {
    int e, s, c0;
    chunk(qi, e, s, c0);
    const float* base = M + (size_t)e * H * n_pad + (size_t)(k - 1 + s) * B + c0;
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
      int lin = u * NT + tid;
      if (TU % NT == 0 || lin < TU) {
        int h = lin / (KC / 4), col = (lin % (KC / 4)) * 4;
        mreg[u] = *reinterpret_cast<const f32x4*>(base + (size_t)h * n_pad + col);
      }
    }
  };
  auto store_m = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
      int lin = u * NT + tid;
      if (TU % NT == 0 || lin < TU) {
        int h = lin / (KC / 4), col = (lin % (KC / 4)) * 4;
        split_store4(&lds[buf][0][h * LDP + col], &lds[buf][NP - 1][h * LDP + col], mreg[u]);
      }
    }
  };
  auto load_band = [&](int qi, frag_t<S> (&dst)[2][KS]) {
    int e, s, c0;
    chunk(qi, e, s, c0);
    const S* base = band + ((((size_t)e * nb + k) * 3 + s) * B) * (size_t)B + c0 + g * RUN;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const S* row = base + (size_t)(rw + 16 * nt + q) * B;
#pragma unroll
      for (int j = 0; j < KS; ++j) dst[nt][j] = load8(row + 8 * j);
    }
  };

  f32x4 acc[MT][2];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) acc[m][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  load_m(0);
  load_band(0, bcur);
  store_m(0);
  __syncthreads();
  for (int qi = 0; qi < nq; ++qi) {
    const int buf = qi & 1;
    const bool more = qi + 1 < nq;
    if (more) {
      load_m(qi + 1);
      load_band(qi + 1, bnext);
    }
#pragma unroll
    for (int j = 0; j < KS; ++j) {
#pragma unroll
      for (int m = 0; m < MT; ++m) {
#pragma unroll
        for (int part = 0; part < NP; ++part) {
          frag_t<S> af = load8(&lds[buf][part][(16 * m + q) * LDP + g * RUN + 8 * j]);
          mma(acc[m][0], af, bcur[0][j]);
          mma(acc[m][1], af, bcur[1][j]);
        }
      }
    }
    if (more) store_m(buf ^ 1);
    __syncthreads();
    if (more) {
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int j = 0; j < KS; ++j) bcur[nt][j] = bnext[nt][j];
    }
  }
  // D[h = 16m + 4g + i][r = rw + 16nt + q]
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    float* out = a + (size_t)(k * B + rw + 16 * nt + q) * H + 4 * g;
#pragma unroll
    for (int m = 0; m < MT; ++m) store4(out + 16 * m, acc[m][nt][0], acc[m][nt][1], acc[m][nt][2], acc[m][nt][3]);
  }
}

// ---------------------------------------------------------------------------
// Backward: dM[e][h][j*B + c] = sum_{kr = j-1, j, j+1} sum_r band[e][kr][j-kr+1][r][c] * da[h][kr*B + r]
// i.e. A_e^T da: the transposed blocks, with block row kr = j+1 read through
// its sub-diagonal slot and kr = j-1 through its super-diagonal slot.
//
// One workgroup owns (e, block j, NW = 32*WAVES sender columns); wave w owns
// 32 columns.  Tile orientation D[c][h]: A operand = band^T (rows c, the k
// index r runs down the stored band rows, so it is staged in LDS and read
// with a stride), B operand = da (rows h, contiguous in r, from LDS).  Each
// lane holds four consecutive nodes of one feature: dM is feature-major, so
// it is written with 8-byte (bf16) stores.  k order inside a 32-step is the
// plain r = 32*j + 8*g + i, which keeps the strided LDS reads conflict-free.
// ---------------------------------------------------------------------------
template <typename S, int H, int WAVES, int KC>
__global__ __launch_bounds__(WAVES * kWave) void banded_bwd_kernel(const S* __restrict__ band,
                                                                    const S* __restrict__ da,
                                                                    S* __restrict__ dM, int n_pad, int B, int E,
                                                                    long ldm) {
  constexpr int NT = WAVES * kWave;
  constexpr int V = 16 / sizeof(S);
  constexpr int NW = 32 * WAVES;             // sender columns per workgroup
  constexpr int PB = NW + 4 / sizeof(S);     // band tile pitch: 4-byte pad, conflict-free strided reads
  constexpr int PD = KC + V;                 // da tile pitch
  constexpr int TB = KC * NW / V, TD = H * KC / V;   // 16-byte units of the band and da tiles
  constexpr int UB = (TB + NT - 1) / NT;     // per thread
  constexpr int UD = (TD + NT - 1) / NT;
  constexpr int KS = KC / 32;
  constexpr int NTL = H / 16;                // feature tiles
  __shared__ __attribute__((aligned(16))) S lb[2][KC * PB];
  __shared__ __attribute__((aligned(16))) S ld[2][H * PD];

  const int nb = n_pad / B;
  const int tiles_per_blk = B / NW;
  const int t = xcd_swizzle(blockIdx.x, gridDim.x);
  const int e = t / (nb * tiles_per_blk);
  const int rem = t % (nb * tiles_per_blk);
  const int j = rem / tiles_per_blk;
  const int c0 = (rem % tiles_per_blk) * NW;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int cw = 32 * wave;                  // first column of this wave inside the tile

  const int kr_lo = (j == 0) ? j : j - 1;
  const int kr_hi = (j == nb - 1) ? j : j + 1;
  const int cpb = B / KC;
  const int nq = (kr_hi - kr_lo + 1) * cpb;

  u32x4 breg[UB], dreg[UD];
  auto load = [&](int qi) __attribute__((always_inline)) {
    int kr = kr_lo + qi / cpb;
    int rr0 = (qi % cpb) * KC;
    int s = j - kr + 1;
    const S* bsrc = band + ((((size_t)e * nb + kr) * 3 + s) * B + rr0) * (size_t)B + c0;
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      int lin = u * NT + tid;
      if (TB % NT == 0 || lin < TB) {
        int r = lin / (NW / V), col = (lin % (NW / V)) * V;
        breg[u] = *reinterpret_cast<const u32x4*>(bsrc + (size_t)r * B + col);
      }
    }
    const S* dsrc = da + (size_t)kr * B + rr0;
#pragma unroll
    for (int u = 0; u < UD; ++u) {
      int lin = u * NT + tid;
      if (TD % NT == 0 || lin < TD) {
        int h = lin / (KC / V), col = (lin % (KC / V)) * V;
        dreg[u] = *reinterpret_cast<const u32x4*>(dsrc + (size_t)h * n_pad + col);
      }
    }
  };
  auto store = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      int lin = u * NT + tid;
      if (TB % NT == 0 || lin < TB) {
        int r = lin / (NW / V), col = (lin % (NW / V)) * V;
        uint32_t* p = reinterpret_cast<uint32_t*>(&lb[buf][r * PB + col]);  // rows are only 4-byte aligned
        p[0] = breg[u].x; p[1] = breg[u].y; p[2] = breg[u].z; p[3] = breg[u].w;
      }
    }
#pragma unroll
    for (int u = 0; u < UD; ++u) {
      int lin = u * NT + tid;
      if (TD % NT == 0 || lin < TD) {
        int h = lin / (KC / V), col = (lin % (KC / V)) * V;
        *reinterpret_cast<u32x4*>(&ld[buf][h * PD + col]) = dreg[u];
      }
    }
  };

  f32x4 acc[2][NTL];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int n = 0; n < NTL; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};

  load(0);
  store(0);
  __syncthreads();
  for (int qi = 0; qi < nq; ++qi) {
    const int buf = qi & 1;
    const bool more = qi + 1 < nq;
    if (more) load(qi + 1);
#pragma unroll
    for (int jj = 0; jj < KS; ++jj) {
      frag_t<S> af[2];
#pragma unroll
      for (int m = 0; m < 2; ++m) af[m] = load8_strided(&lb[buf][(32 * jj + 8 * g) * PB + cw + 16 * m + q], PB);
#pragma unroll
      for (int n = 0; n < NTL; ++n) {
        frag_t<S> bf = load8(&ld[buf][(16 * n + q) * PD + 32 * jj + 8 * g]);
        mma(acc[0][n], af[0], bf);
        mma(acc[1][n], af[1], bf);
      }
    }
    if (more) store(buf ^ 1);
    __syncthreads();
  }
  // D[c = cw + 16m + 4g + i][h = 16n + q]
  S* out = dM + (size_t)e * H * ldm + (size_t)j * B + c0 + cw + 4 * g;
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int n = 0; n < NTL; ++n)
      store4(out + (size_t)(16 * n + q) * ldm + 16 * m, acc[m][n][0], acc[m][n][1], acc[m][n][2], acc[m][n][3]);
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
// Launch shape: the largest workgroup (up to four waves, never more rows than
// a block holds) that still gives at least this many workgroups.
#ifndef GGNN_FWD_MIN_BLOCKS
#define GGNN_FWD_MIN_BLOCKS 256
#endif
#ifndef GGNN_BWD_MIN_BLOCKS
#define GGNN_BWD_MIN_BLOCKS 1024
#endif
namespace {
inline int pick_waves(int B, int nb, int E_or_1, int min_blocks) {
  int waves = B >= 128 ? 4 : B / 32;
  while (waves > 1 && (long)nb * E_or_1 * (B / (32 * waves)) < min_blocks) waves /= 2;
  return waves;
}
}  // namespace

template <typename S, int H>
static hipError_t fwd_dispatch(const void* band, const float* M, float* a, int n_pad, int B, int E, hipStream_t st) {
  const int nb = n_pad / B;
  const int waves = pick_waves(B, nb, 1, GGNN_FWD_MIN_BLOCKS);
  const int blocks = nb * (B / (32 * waves));
  constexpr int KCW = (H >= 256 || sizeof(S) == 4) ? 32 : 64;   // chunk width when B allows it
  const S* bp = static_cast<const S*>(band);
  const float* mp = M;
  if (B < KCW) {  // B == 32
    hipLaunchKernelGGL((banded_fwd_kernel<S, H, 1, 32>), dim3(blocks), dim3(64), 0, st, bp, mp, a, n_pad, B, E);
    return hipGetLastError();
  }
  switch (waves) {
    case 4: hipLaunchKernelGGL((banded_fwd_kernel<S, H, 4, KCW>), dim3(blocks), dim3(256), 0, st, bp, mp, a, n_pad, B, E); break;
    case 2: hipLaunchKernelGGL((banded_fwd_kernel<S, H, 2, KCW>), dim3(blocks), dim3(128), 0, st, bp, mp, a, n_pad, B, E); break;
    default: hipLaunchKernelGGL((banded_fwd_kernel<S, H, 1, KCW>), dim3(blocks), dim3(64), 0, st, bp, mp, a, n_pad, B, E); break;
  }
  return hipGetLastError();
}

template <typename S, int H>
static hipError_t bwd_dispatch(const void* band, const void* da, void* dM, long ldm, int n_pad, int B, int E,
                               hipStream_t st) {
  const int nb = n_pad / B;
  const int waves = pick_waves(B, nb, E, GGNN_BWD_MIN_BLOCKS);
  const int blocks = E * nb * (B / (32 * waves));
  constexpr int KC = 32;
  const S* bp = static_cast<const S*>(band);
  const S* dp = static_cast<const S*>(da);
  S* op = static_cast<S*>(dM);
  switch (waves) {
    case 4: hipLaunchKernelGGL((banded_bwd_kernel<S, H, 4, KC>), dim3(blocks), dim3(256), 0, st, bp, dp, op, n_pad, B, E, ldm); break;
    case 2: hipLaunchKernelGGL((banded_bwd_kernel<S, H, 2, KC>), dim3(blocks), dim3(128), 0, st, bp, dp, op, n_pad, B, E, ldm); break;
    default: hipLaunchKernelGGL((banded_bwd_kernel<S, H, 1, KC>), dim3(blocks), dim3(64), 0, st, bp, dp, op, n_pad, B, E, ldm); break;
  }
  return hipGetLastError();
}

template <typename S>
static hipError_t fwd_h(int H, const void* band, const float* M, float* a, int n_pad, int B, int E, hipStream_t st) {
  switch (H) {
    case 32: return fwd_dispatch<S, 32>(band, M, a, n_pad, B, E, st);
    case 64: return fwd_dispatch<S, 64>(band, M, a, n_pad, B, E, st);
    case 128: return fwd_dispatch<S, 128>(band, M, a, n_pad, B, E, st);
    case 256: return fwd_dispatch<S, 256>(band, M, a, n_pad, B, E, st);
  }
  return hipErrorInvalidValue;
}
template <typename S>
static hipError_t bwd_h(int H, const void* band, const void* da, void* dM, long ldm, int n_pad, int B, int E,
                        hipStream_t st) {
  switch (H) {
    case 32: return bwd_dispatch<S, 32>(band, da, dM, ldm, n_pad, B, E, st);
    case 64: return bwd_dispatch<S, 64>(band, da, dM, ldm, n_pad, B, E, st);
    case 128: return bwd_dispatch<S, 128>(band, da, dM, ldm, n_pad, B, E, st);
    case 256: return bwd_dispatch<S, 256>(band, da, dM, ldm, n_pad, B, E, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace dev

namespace GGNN_IMPL_NS {
hipError_t launch_banded_fwd(int n_pad, int B, int H, int E, const void* band, const float* M, float* a,
                             hipStream_t st) {
  return dev::fwd_h<dev::dt_t>(H, band, M, a, n_pad, B, E, st);
}

hipError_t launch_banded_bwd(int n_pad, int B, int H, int E, const void* band, const void* da, void* dM, long ldm,
                             hipStream_t st) {
  return dev::bwd_h<dev::dt_t>(H, band, da, dM, ldm, n_pad, B, E, st);
}
}  // namespace GGNN_IMPL_NS

}  // namespace ggnn
