// "Supernode" propagation next to the block band (Discussion section: nodes
// allowed to communicate with all nodes, implemented with dense slices of the
// first rows and columns of the adjacency matrix).  Supernodes are the nodes
// 0 .. s-1.  Per edge type, 1-bit dense slices:
//   rows  R_e [s][n_pad]:  edges j -> i with i < s (into a supernode, from anywhere)
//   cols  C_e [n_pad][s]:  edges j -> i with i >= s, j < s (out of a supernode)
// (every other edge belongs to the band), and their transposes for the
// reverse pass.  With M_e = X W_e (+ b_e):
//   a[i]   += sum_e (R_e X)[i] W_e + deg_R,e(i) b_e          (i < s; aggregate first, long contraction)
//   a[i]   += sum_e sum_{j<s} C_e[i][j] (X_s W_e + b_e)[j]   (all i; transform first: X_s W_e is s x H)
// Reverse for the upstream gradient da:
//   P_e = R_e X,  dP_e = da_s W_e^T,  dX += sum_e R_e^T dP_e,  dW_e += P_e^T da_s,  dbias_e += deg_R,e^T da_s
//   dM_e = C_e^T da (s x H),  dX_s += sum_e dM_e W_e^T,  dW_e += X_s^T dM_e,  dbias_e += column sums of dM_e
//
// Kernels: a bits x dense product with a long contraction and a short output
// (the row slice, split over node chunks with fixed-order partial sums), one
// with a short contraction and a long output (the column slice), both on the
// matrix cores; the small dense products (s x H x H per type) on the vector
// ALUs.
#include "device_common.h"
#include "kernels.h"

namespace ggnn {
namespace dev {

template <typename S> __device__ __forceinline__ frag_t<S> sn_bits_frag(uint32_t byte);
template <> __device__ __forceinline__ bf16x8 sn_bits_frag<bf16s>(uint32_t byte) {
  // bit 2k at position 2k and bit 2k+1 at 16 + 2k of byte * 0x8001; masked and
  // scaled onto bf16 1.0 (0x3F80) in the low and high half of word k
  const uint32_t x = byte * 0x8001u;
  u32x4 w;
#pragma unroll
  for (int k = 0; k < 4; ++k) w[k] = (x & (0x10001u << (2 * k))) * (0x3F80u >> (2 * k));
  return __builtin_bit_cast(bf16x8, w);
}
template <> __device__ __forceinline__ f32x8 sn_bits_frag<float>(uint32_t byte) {
  f32x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<float>((byte >> i) & 1u);
  return r;
}

constexpr int kSnKC = 64;   // nodes staged per sub-chunk of the long contraction

// LDS row pitch (elements) of node-major staging read with transposing
// reads: 2P bytes = 160 mod 256 puts the four rows of one read on disjoint
// banks.
template <typename S, int H> constexpr int sn_pitch() {
  return sizeof(S) == 2 ? H + ((80 - H) % 128 + 128) % 128 : H + 4;
}

// Long contraction over the nodes of one chunk:
//   part[c][e][i][h] = sum_{j in chunk c} bits[e][i][j] Z(j, h),  i < s.
// bits [E][s][n_pad/8] (row i, bit j).  Z node-major [n_pad][H] (ZFM =
// false) or feature-major [H][n_pad] (ZFM = true), storage type S.
// Workgroup (4 waves): one chunk and one edge type; wave w owns the row
// tiles w, w + 4 (s <= 128) and every feature tile.
template <typename S, int H, bool ZFM>
__global__ __launch_bounds__(256) void super_rows_kernel(const uint8_t* __restrict__ bits, const S* __restrict__ Z,
                                                         float* __restrict__ part, int n_pad, int E, int s,
                                                         int chunk) {
  constexpr int MT = H / 16, P = sn_pitch<S, H>(), PF = kSnKC + 16 / (int)sizeof(S);
  constexpr int V = 16 / sizeof(S);
  __shared__ __attribute__((aligned(16))) S zs[ZFM ? H * PF : kSnKC * P];
  const int c = blockIdx.x / E, e = blockIdx.x % E;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int nrt = s / 16;
  const int j_lo = c * chunk, j_hi = min(n_pad, j_lo + chunk);
  const size_t rowb = (size_t)n_pad / 8;
  f32x4 acc[2][MT];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[r][m] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int j0 = j_lo; j0 < j_hi; j0 += kSnKC) {
    __syncthreads();   // the previous sub-chunk is fully read
    if constexpr (!ZFM) {
      for (int u = tid; u < kSnKC * (H / V); u += 256) {
        const int k = u / (H / V), h = (u % (H / V)) * V;
        *reinterpret_cast<u32x4*>(&zs[k * P + h]) = *reinterpret_cast<const u32x4*>(Z + (size_t)(j0 + k) * H + h);
      }
    } else {
      for (int u = tid; u < H * (kSnKC / V); u += 256) {
        const int h = u / (kSnKC / V), k = (u % (kSnKC / V)) * V;
        *reinterpret_cast<u32x4*>(&zs[h * PF + k]) = *reinterpret_cast<const u32x4*>(Z + (size_t)h * n_pad + j0 + k);
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kSnKC / 32; ++kk) {
      frag_t<S> bf[2];
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int rt = wave + 4 * r;
        const uint32_t byte =
            rt < nrt ? bits[((size_t)e * s + 16 * rt + q) * rowb + (j0 + 32 * kk) / 8 + g] : 0u;
        bf[r] = sn_bits_frag<S>(byte);
      }
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        frag_t<S> af;
        if constexpr (!ZFM) {
          af = tr_frag(zs, P, 32 * kk, 16 * m, lane);
        } else {
          af = load8(&zs[(16 * m + q) * PF + 32 * kk + 8 * g]);
        }
#pragma unroll
        for (int r = 0; r < 2; ++r)
          if (wave + 4 * r < nrt) mma(acc[r][m], af, bf[r]);
      }
    }
  }
  // D[feature 16m + 4g + j][row 16 rt + q]
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int rt = wave + 4 * r;
    if (rt >= nrt) continue;
    float* o = part + (((size_t)c * E + e) * s + 16 * rt + q) * H + 4 * g;
#pragma unroll
    for (int m = 0; m < MT; ++m) *reinterpret_cast<f32x4*>(o + 16 * m) = acc[r][m];
  }
}

// Short contraction, long output, summed over edge types:
//   out[i][h] += sum_e sum_{j < s} bits[e][i][j] Y[e][j][h],  all rows i.
// bits [E][n_pad][s/8] (row i, bit j); Y float [E][s][H].  Workgroup (4
// waves, 64 rows): per type, Y_e is staged in LDS in fragment order (bf16 hi
// + lo pairs in bf16 mode, float otherwise) and every wave multiplies it by
// the bit rows of its 16 rows.
template <typename S, int H>
__global__ __launch_bounds__(256) void super_cols_kernel(const uint8_t* __restrict__ bits,
                                                         const float* __restrict__ Y, float* __restrict__ out,
                                                         int n_pad, int E, int s) {
  constexpr int MT = H / 16;
  constexpr int NP = sizeof(S) == 2 ? 2 : 1;
  constexpr int SMAX = 128;
  constexpr int FR = 64 * 8;   // elements of one fragment
  __shared__ __attribute__((aligned(16))) S ys[NP][(SMAX / 32) * MT * FR];
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int i0 = blockIdx.x * 64 + 16 * wave;
  const int ks = s / 32;
  const size_t rowb = (size_t)s / 8;
  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int e = 0; e < E; ++e) {
    __syncthreads();
    // fragment (kk, m), lane (qq, gg): Y[e][32kk + 8gg + x][16m + qq], x = 0..7
    for (int u = tid; u < ks * MT * 64; u += 256) {
      const int l = u % 64, fm = u / 64, m = fm % MT, kk = fm / MT;
      const int qq = l % 16, gg = l / 16;
      const float* src = Y + ((size_t)e * s + 32 * kk + 8 * gg) * H + 16 * m + qq;
      float v[8];
#pragma unroll
      for (int x = 0; x < 8; ++x) v[x] = src[(size_t)x * H];
      if constexpr (NP == 2) {
        bf16x8 hi, lo;
        split8(v, hi, lo);
        *reinterpret_cast<bf16x8*>(&ys[0][(size_t)fm * FR + l * 8]) = hi;
        *reinterpret_cast<bf16x8*>(&ys[NP - 1][(size_t)fm * FR + l * 8]) = lo;
      } else {
#pragma unroll
        for (int x = 0; x < 8; ++x) ys[0][(size_t)fm * FR + fo<S>(0, l, x)] = v[x];
      }
    }
    __syncthreads();
    for (int kk = 0; kk < ks; ++kk) {
      const frag_t<S> bf = sn_bits_frag<S>(bits[((size_t)e * n_pad + i0 + q) * rowb + 4 * kk + g]);
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int part = 0; part < NP; ++part)
          mma(acc[m], load_fragi<S>(ys[part] + (size_t)(kk * MT + m) * FR, 0, lane), bf);
    }
  }
  // D[feature 16m + 4g + j][row i0 + q]
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    float* o = out + (size_t)(i0 + q) * H + 16 * m + 4 * g;
    const f32x4 b = *reinterpret_cast<const f32x4*>(o);
    *reinterpret_cast<f32x4*>(o) = f32x4{b[0] + acc[m][0], b[1] + acc[m][1], b[2] + acc[m][2], b[3] + acc[m][3]};
  }
}

// Row degrees of the row slice: deg[e][i] = number of bits set in row i
// (one instance per storage-type build).
template <typename S>
__global__ __launch_bounds__(256) void super_deg_kernel(const uint8_t* __restrict__ bits, float* __restrict__ deg,
                                                        int n_pad, int rows) {
  const int r = blockIdx.x;
  const size_t rowb = (size_t)n_pad / 8;
  int c = 0;
  for (size_t w = threadIdx.x; w < rowb / 4; w += 256)
    c += __popc(reinterpret_cast<const uint32_t*>(bits + (size_t)r * rowb)[w]);
  __shared__ int red[256];
  red[threadIdx.x] = c;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0 && r < rows) deg[r] = static_cast<float>(red[0]);
}

// Small dense products on the vector ALUs, one thread per output element:
//   C[b][m][n] (= or +=) sum_{b' in batches of b} ( sum_k A(b', m, k) B(b', k, n)
//                                                  + scale(b', m) bias(b', n) )
// A, B: strided views (element strides for batch, row and column) of storage
// type TA / TB (A NULL: all ones); with `reduce`, every b' in [0, nb) feeds
// the single output batch 0, else b' = b.  bias (float [nb][N]) and scale
// (float [nb][M]) optional.  Fixed summation order.
struct SmallGemm {
  int M, N, K, nb, reduce, accumulate;
  const void* A;
  long a_b, a_m, a_k;
  const void* B;
  long b_b, b_k, b_n;
  float* C;
  long c_b, c_m, c_n;
  const float* bias;
  const float* scale;
};
// kSgG threads per output, thread t summing k = t, t + kSgG, ... of every
// batch in order (the bias of batch bb on thread 0 after its terms); the kSgG
// partial sums are combined by a fixed butterfly, so the result does not
// depend on scheduling.
constexpr int kSgG = 8;
template <typename TA, typename TB>
__global__ __launch_bounds__(256) void small_gemm_kernel(SmallGemm p) {
  const long idx = ((long)blockIdx.x * blockDim.x + threadIdx.x) / kSgG;
  const int t = threadIdx.x % kSgG;
  const long outs = (long)(p.reduce ? 1 : p.nb) * p.M * p.N;
  const bool active = idx < outs;   // the same for the kSgG threads of an output
  const int n = (int)(idx % p.N), m = (int)((idx / p.N) % p.M), b = (int)(idx / ((long)p.N * p.M));
  const TA* A = static_cast<const TA*>(p.A);
  const TB* B = static_cast<const TB*>(p.B);
  float s = 0.f;
  if (active) {
    const int b_lo = p.reduce ? 0 : b, b_hi = p.reduce ? p.nb : b + 1;
    for (int bb = b_lo; bb < b_hi; ++bb) {
      for (int k = t; k < p.K; k += kSgG) {
        const float a = A ? to_f<TA>(A[bb * p.a_b + m * p.a_m + k * p.a_k]) : 1.f;
        s += a * to_f<TB>(B[bb * p.b_b + k * p.b_k + n * p.b_n]);
      }
      if (p.bias && t == 0) s += (p.scale ? p.scale[(long)bb * p.M + m] : 1.f) * p.bias[(long)bb * p.N + n];
    }
  }
#pragma unroll
  for (int d = kSgG / 2; d > 0; d /= 2) s += __shfl_xor(s, d);
  if (active && t == 0) {
    float* c = p.C + b * p.c_b + m * p.c_m + n * p.c_n;
    *c = p.accumulate ? *c + s : s;
  }
}

}  // namespace dev

namespace {
using dev::SmallGemm;

template <typename TA, typename TB>
hipError_t small_gemm(const SmallGemm& p, hipStream_t st) {
  const long outs = (long)(p.reduce ? 1 : p.nb) * p.M * p.N;
  const long threads = outs * dev::kSgG;
  hipLaunchKernelGGL((dev::small_gemm_kernel<TA, TB>), dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, p);
  return hipGetLastError();
}

// Row-slice chunking: about 256 workgroups over chunks x types, chunks a
// multiple of the staging sub-chunk.
int sn_chunk(int n_pad, int E) {
  const long want = (256 + E - 1) / E;
  long ch = ((n_pad + want - 1) / want + dev::kSnKC - 1) / dev::kSnKC * dev::kSnKC;
  return (int)(ch < dev::kSnKC ? dev::kSnKC : ch);
}

// Workspace (floats): row-slice partials [nch][E][s][H], then three [E][s][H]
// buffers (P, the second product, the third) and deg [E][s].
struct SnLayout {
  size_t part, p0, p1, p2, deg, total;
  int nch, chunk;
};
SnLayout sn_layout(int n_pad, int H, int E, int s) {
  auto up = [](size_t x) { return (x + 63) / 64 * 64; };
  SnLayout l;
  l.chunk = sn_chunk(n_pad, E);
  l.nch = (n_pad + l.chunk - 1) / l.chunk;
  const size_t esh = (size_t)E * s * H;
  l.part = 0;
  l.p0 = up((size_t)l.nch * esh);
  l.p1 = l.p0 + up(esh);
  l.p2 = l.p1 + up(esh);
  l.deg = l.p2 + up(esh);
  l.total = (l.deg + up((size_t)E * s)) * sizeof(float);
  return l;
}

template <typename S, int H>
hipError_t rows_product(const uint8_t* bits, const S* Z, bool zfm, float* out, float* part, const SnLayout& L,
                        int n_pad, int E, int s, hipStream_t st) {
  if (zfm)
    hipLaunchKernelGGL((dev::super_rows_kernel<S, H, true>), dim3(L.nch * E), dim3(256), 0, st, bits, Z, part, n_pad,
                       E, s, L.chunk);
  else
    hipLaunchKernelGGL((dev::super_rows_kernel<S, H, false>), dim3(L.nch * E), dim3(256), 0, st, bits, Z, part,
                       n_pad, E, s, L.chunk);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const long cnt = (long)E * s * H;
  err = launch_fill_zero(out, (size_t)cnt, st);
  if (err != hipSuccess) return err;
  return launch_reduce_partials(part, out, L.nch, (int)cnt, cnt, st);
}

template <typename S, int H>
hipError_t super_fwd_h(int n_pad, int E, int s, const uint8_t* rows, const uint8_t* cols, const S* X, const S* W,
                       const float* bias, float* a, float* ws, hipStream_t st) {
  const SnLayout L = sn_layout(n_pad, H, E, s);
  float *P = ws + L.p0, *Ms = ws + L.p1, *deg = ws + L.deg;
  // P_e = R_e X, deg_R
  hipError_t err = rows_product<S, H>(rows, X, false, P, ws + L.part, L, n_pad, E, s, st);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((dev::super_deg_kernel<S>), dim3(E * s), dim3(256), 0, st, rows, deg, n_pad, E * s);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  // a[0:s] += sum_e P_e W_e + deg_R,e b_e
  SmallGemm g1{s, H, H, E, 1, 1, P, (long)s * H, H, 1, W, (long)H * H, H, 1, a, 0, H, 1, bias, deg};
  if ((err = small_gemm<float, S>(g1, st)) != hipSuccess) return err;
  // M_s,e = X_s W_e + b_e;  a += sum_e C_e M_s,e
  SmallGemm g2{s, H, H, E, 0, 0, X, 0, H, 1, W, (long)H * H, H, 1, Ms, (long)s * H, H, 1, bias, nullptr};
  if ((err = small_gemm<S, S>(g2, st)) != hipSuccess) return err;
  hipLaunchKernelGGL((dev::super_cols_kernel<S, H>), dim3(n_pad / 64), dim3(256), 0, st, cols, Ms, a, n_pad, E, s);
  return hipGetLastError();
}

template <typename S, int H>
hipError_t super_bwd_h(int n_pad, int E, int s, const uint8_t* rows, const uint8_t* rows_t, const uint8_t* cols_t,
                       const S* X, const S* W, const S* da, float* dX, float* dW, float* dbias, float* ws,
                       hipStream_t st) {
  const SnLayout L = sn_layout(n_pad, H, E, s);
  float *P = ws + L.p0, *dP = ws + L.p1, *dMs = ws + L.p2, *deg = ws + L.deg;
  const long np = n_pad;
  // recompute P_e = R_e X and deg_R; dM_s,e = C_e^T da
  hipError_t err = rows_product<S, H>(rows, X, false, P, ws + L.part, L, n_pad, E, s, st);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((dev::super_deg_kernel<S>), dim3(E * s), dim3(256), 0, st, rows, deg, n_pad, E * s);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  if ((err = rows_product<S, H>(cols_t, da, true, dMs, ws + L.part, L, n_pad, E, s, st)) != hipSuccess) return err;
  // dP_e = da_s W_e^T  (da feature-major: element (i, h) at h * n_pad + i)
  SmallGemm g1{s, H, H, E, 0, 0, da, 0, 1, np, W, (long)H * H, 1, H, dP, (long)s * H, H, 1, nullptr, nullptr};
  if ((err = small_gemm<S, S>(g1, st)) != hipSuccess) return err;
  // dX += sum_e R_e^T dP_e
  hipLaunchKernelGGL((dev::super_cols_kernel<S, H>), dim3(n_pad / 64), dim3(256), 0, st, rows_t, dP, dX, n_pad, E, s);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  // dX_s += sum_e dM_s,e W_e^T
  SmallGemm g2{s, H, H, E, 1, 1, dMs, (long)s * H, H, 1, W, (long)H * H, 1, H, dX, 0, H, 1, nullptr, nullptr};
  if ((err = small_gemm<float, S>(g2, st)) != hipSuccess) return err;
  // dW_e += P_e^T da_s + X_s^T dM_s,e
  SmallGemm g3{H, H, s, E, 0, 1, P, (long)s * H, 1, H, da, 0, 1, np, dW, (long)H * H, H, 1, nullptr, nullptr};
  if ((err = small_gemm<float, S>(g3, st)) != hipSuccess) return err;
  SmallGemm g4{H, H, s, E, 0, 1, X, 0, 1, H, dMs, (long)s * H, H, 1, dW, (long)H * H, H, 1, nullptr, nullptr};
  if ((err = small_gemm<S, float>(g4, st)) != hipSuccess) return err;
  if (dbias == nullptr) return hipSuccess;
  // dbias_e += deg_R,e^T da_s + column sums of dM_s,e
  SmallGemm g5{1, H, s, E, 0, 1, deg, s, 0, 1, da, 0, 1, np, dbias, H, 0, 1, nullptr, nullptr};
  if ((err = small_gemm<float, S>(g5, st)) != hipSuccess) return err;
  SmallGemm g6{1, H, s, E, 0, 1, nullptr, 0, 0, 0, dMs, (long)s * H, H, 1, dbias, H, 0, 1, nullptr, nullptr};
  return small_gemm<float, float>(g6, st);
}
}  // namespace

namespace GGNN_IMPL_NS {
hipError_t launch_super_fwd(int n_pad, int H, int E, int s, const void* rows, const void* cols, const void* X,
                            const void* W, const float* bias, float* a, void* ws, hipStream_t st) {
  using S = dev::dt_t;
  const uint8_t *r = static_cast<const uint8_t*>(rows), *c = static_cast<const uint8_t*>(cols);
  const S *x = static_cast<const S*>(X), *w = static_cast<const S*>(W);
  float* f = static_cast<float*>(ws);
  switch (H) {
    case 32: return super_fwd_h<S, 32>(n_pad, E, s, r, c, x, w, bias, a, f, st);
    case 64: return super_fwd_h<S, 64>(n_pad, E, s, r, c, x, w, bias, a, f, st);
    case 128: return super_fwd_h<S, 128>(n_pad, E, s, r, c, x, w, bias, a, f, st);
    case 256: return super_fwd_h<S, 256>(n_pad, E, s, r, c, x, w, bias, a, f, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_super_bwd(int n_pad, int H, int E, int s, const void* rows, const void* rows_t,
                            const void* cols_t, const void* X, const void* W, const void* da, float* dX, float* dW,
                            float* dbias, void* ws, hipStream_t st) {
  using S = dev::dt_t;
  const uint8_t *r = static_cast<const uint8_t*>(rows), *rt = static_cast<const uint8_t*>(rows_t),
                *ct = static_cast<const uint8_t*>(cols_t);
  const S *x = static_cast<const S*>(X), *w = static_cast<const S*>(W), *d = static_cast<const S*>(da);
  float* f = static_cast<float*>(ws);
  switch (H) {
    case 32: return super_bwd_h<S, 32>(n_pad, E, s, r, rt, ct, x, w, d, dX, dW, dbias, f, st);
    case 64: return super_bwd_h<S, 64>(n_pad, E, s, r, rt, ct, x, w, d, dX, dW, dbias, f, st);
    case 128: return super_bwd_h<S, 128>(n_pad, E, s, r, rt, ct, x, w, d, dX, dW, dbias, f, st);
    case 256: return super_bwd_h<S, 256>(n_pad, E, s, r, rt, ct, x, w, d, dX, dW, dbias, f, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace GGNN_IMPL_NS

#if GGNN_DT_BF16
size_t super_workspace(int n_pad, int H, int E, int s) { return sn_layout(n_pad, H, E, s).total; }
#endif

}  // namespace ggnn
