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

// LDS row pitch (elements) of node-major staging read with transposing
// reads: 2P bytes = 160 mod 256 puts the four rows of one read on disjoint
// banks.
template <typename S, int H> constexpr int sn_pitch() {
  return sizeof(S) == 2 ? H + ((80 - H) % 128 + 128) % 128 : H + 4;
}
// Nodes per chunk of the long contraction: the whole chunk of Z is staged in
// LDS at once (at most 96 KB), a multiple of 64 nodes.
template <typename S, int H, bool ZFM> constexpr int sn_chunk_nodes() {
  constexpr int per = ZFM ? 98304 / (H * (int)sizeof(S)) - 16 : 98304 / (sn_pitch<S, H>() * (int)sizeof(S));
  constexpr int c = per / 64 * 64;
  return c > 576 ? 576 : c;
}

// Long contraction over the nodes of one chunk, for the active supernode
// rows i < sa and the edge types of one group:
//   part[c][e][i][h] = sum_{j in chunk c} bits[e][i][j] Z(j, h)
//   part[c][E sa H + e sa + i] = number of those bits set (row degree)
// bits [E][s][n_pad/8] (row i, bit j).  Z node-major [n_pad][H] (ZFM =
// false) or feature-major [H][n_pad] (ZFM = true), storage type S.
// Workgroup (4 waves): chunk c, types [e0, e1); the chunk of Z is staged in
// LDS once (all of a thread's loads issued before its writes, one memory
// latency), then every (type, 16-row tile) pair of the group goes to a wave;
// a wave loads its rows' bit bytes for the whole chunk in one go (the first
// pair's before the staging) and skips every 32-node k step where none of
// its 16 rows has an edge (wave-uniform test).
template <typename S, int H, bool ZFM>
__global__ __launch_bounds__(256) void super_long_kernel(const uint8_t* __restrict__ bits, const S* __restrict__ Z,
                                                         float* __restrict__ part, long pstride, int n_pad, int E,
                                                         int s, int sa, int chunk, int tpg) {
  constexpr int MT = H / 16, CN = sn_chunk_nodes<S, H, ZFM>(), V = 16 / (int)sizeof(S);
  constexpr int P = sn_pitch<S, H>(), PF = CN + 16 / (int)sizeof(S);
  constexpr int NKS = CN / 32;   // k steps (and bit dwords per row) of a full chunk
  __shared__ __attribute__((aligned(16))) S zs[ZFM ? H * PF : CN * P];
  const int ntg = (E + tpg - 1) / tpg;
  // the type groups of one chunk on one XCD (they stage the same rows)
  const int lid = xcd_swizzle(blockIdx.x, gridDim.x);
  const int c = lid / ntg, tgi = lid % ntg;
  const int e0 = tgi * tpg, e1 = min(E, e0 + tpg);
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int j_lo = c * chunk, len = min(n_pad - j_lo, chunk);   // a multiple of 64
  const int nks = len / 32;
  const size_t rowb = (size_t)n_pad / 8;
  const int nrt = sa / 16;
  const int npairs = (e1 - e0) * nrt;
  // this lane's bit row of pair pr, whole chunk: dword ks holds the bytes of
  // k step ks for the four lane groups (byte g: nodes 32 ks + 8 g .. + 7)
  uint32_t bw[NKS];
  auto load_bits = [&](int pr) __attribute__((always_inline)) {
    const int e = e0 + pr / nrt, rt = pr % nrt;
    const uint8_t* brow = bits + ((size_t)e * s + 16 * rt + q) * rowb + j_lo / 8;
#pragma unroll
    for (int d = 0; d < NKS; d += 2) {
      if (d < nks) {
        const u32x2 v = *reinterpret_cast<const u32x2*>(brow + 4 * d);
        bw[d] = v[0];
        bw[d + 1] = v[1];
      } else {
        bw[d] = 0u;
        bw[d + 1] = 0u;
      }
    }
  };
  if (wave < npairs) load_bits(wave);
  // stage the chunk: every 16-byte unit of a thread in flight at once
  {
    constexpr int UPT = ((ZFM ? H * (CN / V) : CN * (H / V)) + 255) / 256;
    const int units = ZFM ? H * (len / V) : len * (H / V);
    u32x4 r[UPT];
#pragma unroll
    for (int u = 0; u < UPT; ++u) {
      const int lin = u * 256 + tid;
      if (lin < units) {
        if constexpr (ZFM) {
          const int h = lin / (len / V), k = (lin % (len / V)) * V;
          r[u] = *reinterpret_cast<const u32x4*>(Z + (size_t)h * n_pad + j_lo + k);
        } else {
          const int k = lin / (H / V), h = (lin % (H / V)) * V;
          r[u] = *reinterpret_cast<const u32x4*>(Z + (size_t)(j_lo + k) * H + h);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < UPT; ++u) {
      const int lin = u * 256 + tid;
      if (lin < units) {
        if constexpr (ZFM) {
          const int h = lin / (len / V), k = (lin % (len / V)) * V;
          *reinterpret_cast<u32x4*>(&zs[h * PF + k]) = r[u];
        } else {
          const int k = lin / (H / V), h = (lin % (H / V)) * V;
          *reinterpret_cast<u32x4*>(&zs[k * P + h]) = r[u];
        }
      }
    }
  }
  __syncthreads();
  for (int pr = wave; pr < npairs; pr += 4) {
    const int e = e0 + pr / nrt, rt = pr % nrt;
    if (pr != wave) load_bits(pr);
    f32x4 acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
    int deg = 0;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const uint32_t byte = (bw[ks] >> (8 * g)) & 0xFFu;
      if (__builtin_amdgcn_ballot_w64(byte != 0u) == 0) continue;
      deg += __popc(byte);
      const frag_t<S> bf = sn_bits_frag<S>(byte);
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        frag_t<S> af;
        if constexpr (!ZFM) {
          af = tr_frag(zs, P, 32 * ks, 16 * m, lane);
        } else {
          af = load8(&zs[(16 * m + q) * PF + 32 * ks + 8 * g]);
        }
        mma(acc[m], af, bf);
      }
    }
    // D[feature 16m + 4g + j][row 16 rt + q]
    float* o = part + (size_t)c * pstride + ((size_t)e * sa + 16 * rt + q) * H + 4 * g;
#pragma unroll
    for (int m = 0; m < MT; ++m) *reinterpret_cast<f32x4*>(o + 16 * m) = acc[m];
    deg += __shfl_xor(deg, 16);
    deg += __shfl_xor(deg, 32);
    if (g == 0) part[(size_t)c * pstride + (size_t)E * sa * H + (size_t)e * sa + 16 * rt + q] = static_cast<float>(deg);
  }
}

// out[i] = sum_{c < nch} part[c * stride + i] for i < count (a multiple of
// four).  A workgroup of 64 x 16 threads owns 256 consecutive outputs:
// thread (x, y) sums, for its four outputs, the chunks c = y, y + 16, ... in
// increasing order (all its loads in flight), then thread (x, 0) adds the 16
// sums in order y = 0..15.  The order depends only on nch: results do not
// depend on scheduling.
constexpr int kSnRW = 16;
static __global__ __launch_bounds__(64 * kSnRW) void sn_reduce_kernel(const float* __restrict__ part,
                                                                      float* __restrict__ out, int nch, int count,
                                                                      long stride) {
  __shared__ f32x4 red[kSnRW][64];
  const int x = threadIdx.x % 64, y = threadIdx.x / 64;
  const int i = 4 * (blockIdx.x * 64 + x);
  f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
  if (i < count) {
    int c = y;
    for (; c + 3 * kSnRW < nch; c += 4 * kSnRW) {
      f32x4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const f32x4*>(part + (size_t)(c + u * kSnRW) * stride + i);
#pragma unroll
      for (int u = 0; u < 4; ++u) s += v[u];
    }
    for (; c < nch; c += kSnRW) s += *reinterpret_cast<const f32x4*>(part + (size_t)c * stride + i);
  }
  red[y][x] = s;
  __syncthreads();
  if (y == 0 && i < count) {
    f32x4 t = red[0][x];
#pragma unroll
    for (int w = 1; w < kSnRW; ++w) t += red[w][x];
    *reinterpret_cast<f32x4*>(out + i) = t;
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


#if GGNN_DT_BF16
// The supernode rows' per-type aggregate for the fused forward step, as a gather:
//   rec[e][i][h] = sum_{j : bits[e][i] has bit j} X[j][h],   rec[E sr H + e sr + i] = that count
// for the first sr rows of the row slice R_e (X node-major [n_pad][H]).  The slice rows are sparse
// (hub edges), so rather than a contraction over all n_pad nodes, a workgroup (e, i) lists the row's
// set bits and sums the listed nodes' states: each of its sixteen waves takes a sixteenth of the row
// (at the 20k-node workload one dword per lane, so a call is three dependent memory rounds: bits,
// list, rows), compacts the set bits of 2048 columns at a time into an LDS list in column order (a
// prefix count over the lanes), and adds the listed rows in that order in fp32, lane (r, c) taking 8
// features of entries r, r + R, ... (R rows per load instruction); the waves' partial sums are then
// combined in wave order, so the result depends only on the row (no float atomics).  The reverse
// record is gathered from the gate gradients G^ instead of da (super_gather_rev_kernel below): da is
// feature-major, so a gather of it costs one scattered element per feature row and listed node, and
// every layout of those loads tried (one node of all features per instruction, 16 nodes of 4
// features, the row split over 8 workgroups) ran slower than the long contraction's staging.
constexpr int kSnGatherWaves = 16;
template <int H>
__global__ __launch_bounds__(64 * kSnGatherWaves) void super_gather_kernel(const uint8_t* __restrict__ bits,
                                                                           const bf16s* __restrict__ X,
                                                                           float* __restrict__ rec, int n_pad, int E,
                                                                           int s, int sr) {
  constexpr int NW = kSnGatherWaves, SLAB = 64 * 32;
  __shared__ int lst[NW][SLAB];
  __shared__ float part[NW][H + 1];
  const int e = blockIdx.x / sr, i = blockIdx.x % sr;
  const int tid = threadIdx.x, w = tid / kWave, lane = tid % kWave;
  const uint32_t* row = reinterpret_cast<const uint32_t*>(bits + ((size_t)e * s + i) * (size_t)(n_pad / 8));
  const int ndw = n_pad / 32;
  const int d0 = w * ndw / NW, d1 = (w + 1) * ndw / NW;
  constexpr int CPR = H / 8;      // lanes per listed row
  constexpr int R = 64 / CPR;     // listed rows per load instruction
  constexpr int UB = 8;           // load instructions in flight
  const int r = lane / CPR, c = lane % CPR;
  float acc[8];
#pragma unroll
  for (int x = 0; x < 8; ++x) acc[x] = 0.f;
  int deg = 0;
  for (int base = d0; base < d1; base += kWave) {
    const int d = base + lane;
    uint32_t wd = d < d1 ? row[d] : 0u;
    const int cnt = __popc(wd);
    int incl = cnt;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int v = __shfl_up(incl, off);
      if (lane >= off) incl += v;
    }
    const int total = __shfl(incl, kWave - 1);
    int pos = incl - cnt;
    while (wd != 0u) {
      const int b = __ffs(wd) - 1;
      wd &= wd - 1u;
      lst[w][pos++] = d * 32 + b;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    deg += total;
    for (int k0 = 0; k0 < total; k0 += R * UB) {
      u32x4 v[UB];
#pragma unroll
      for (int u = 0; u < UB; ++u) {
        const int k = k0 + u * R + r;
        v[u] = k < total ? *reinterpret_cast<const u32x4*>(X + (size_t)lst[w][k] * H + 8 * c) : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int u = 0; u < UB; ++u)
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          acc[2 * x] += lo_f(v[u][x]);
          acc[2 * x + 1] += hi_f(v[u][x]);
        }
    }
    __builtin_amdgcn_wave_barrier();   // this slab's list is read before the next one is written
  }
  // entries r = 0 .. R-1 of the wave, then the waves in order
#pragma unroll
  for (int x = 0; x < 8; ++x)
#pragma unroll
    for (int off = CPR; off < kWave; off <<= 1) acc[x] += __shfl_xor(acc[x], off);
  if (r == 0) {
#pragma unroll
    for (int x = 0; x < 8; ++x) part[w][8 * c + x] = acc[x];
  }
  if (lane == 0) part[w][H] = static_cast<float>(deg);
  __syncthreads();
  if (tid <= H) {
    float t = part[0][tid];
#pragma unroll
    for (int ww = 1; ww < NW; ++ww) t += part[ww][tid];
    if (tid < H)
      rec[((size_t)e * sr + i) * H + tid] = t;
    else
      rec[(size_t)E * sr * H + (size_t)e * sr + i] = t;
  }
}

// The supernode rows' record of the fused reverse step from the GRU reverse's gate gradients: the
// message gradient of supernode j is sum_i C_e[i][j] da[i] over its out-edges, and da = G^ Wi^T row
// by row, so the record is (sum_i C_e[i][j] G^[i]) Wi^T: the listed rows of G^ (node-major [n][3H],
// contiguous 3H-element rows, where da is stored feature-major and its gathers touch one line per
// feature) are summed in fp32 in column order as above, then multiplied by Wi once per (e, j).  The
// sum skips da's bf16 rounding; it is otherwise the same linear map.  Lane (r, c) adds 8 gate columns
// of entries r, r + R, ... (R = 64 / (3H/8) rows per load); a wave's R partial sums are added in
// order, then the waves' sums in a fixed order.  For the product, thread (f, p) of 16 per output
// feature f holds gate columns 3H/16 p .. of row f of Wi (loaded at the start, in flight during the
// gathers) and the 16 partial dot products are added by a fixed butterfly over the lanes.
template <int H>
__global__ __launch_bounds__(64 * kSnGatherWaves) void super_gather_rev_kernel(const uint8_t* __restrict__ bits,
                                                                               const bf16s* __restrict__ ghat,
                                                                               const bf16s* __restrict__ Wi,
                                                                               float* __restrict__ rec, int n_pad,
                                                                               int E, int s, int sr) {
  constexpr int NW = kSnGatherWaves, SLAB = 64 * 32, G3 = 3 * H;
  constexpr int CPR = G3 / 8, R = 64 / CPR;   // lanes per listed row, rows per load instruction
  constexpr int UB = 8;
  __shared__ int lst[NW][SLAB];
  __shared__ float part[NW][G3];
  __shared__ float gsum[G3];
  __shared__ int degs[NW];
  const int e = blockIdx.x / sr, j = blockIdx.x % sr;
  const int tid = threadIdx.x, w = tid / kWave, lane = tid % kWave;
  const uint32_t* row = reinterpret_cast<const uint32_t*>(bits + ((size_t)e * s + j) * (size_t)(n_pad / 8));
  const int ndw = n_pad / 32;
  const int d0 = w * ndw / NW, d1 = (w + 1) * ndw / NW;
  const int r = lane / CPR, c = lane % CPR;
  const bool active = r < R;
  // Wi row f = tid / 16, gate columns CW p .. CW p + CW - 1 (p = tid % 16), as CW / 2 dwords
  constexpr int CW = G3 / 16;
  const int wf = tid / 16, wp = tid % 16;
  uint32_t wreg[CW / 2];
  if (wf < H) {
    const uint32_t* wsrc = reinterpret_cast<const uint32_t*>(Wi + (size_t)wf * G3 + CW * wp);
#pragma unroll
    for (int x = 0; x < CW / 2; ++x) wreg[x] = wsrc[x];
  }
  float acc[8];
#pragma unroll
  for (int x = 0; x < 8; ++x) acc[x] = 0.f;
  int deg = 0;
  for (int base = d0; base < d1; base += kWave) {
    const int d = base + lane;
    uint32_t wd = d < d1 ? row[d] : 0u;
    const int cnt = __popc(wd);
    int incl = cnt;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int v = __shfl_up(incl, off);
      if (lane >= off) incl += v;
    }
    const int total = __shfl(incl, kWave - 1);
    int pos = incl - cnt;
    while (wd != 0u) {
      const int b = __ffs(wd) - 1;
      wd &= wd - 1u;
      lst[w][pos++] = d * 32 + b;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    deg += total;
    for (int k0 = 0; k0 < total; k0 += R * UB) {
      u32x4 v[UB];
#pragma unroll
      for (int u = 0; u < UB; ++u) {
        const int k = k0 + u * R + r;
        v[u] = active && k < total ? *reinterpret_cast<const u32x4*>(ghat + (size_t)lst[w][k] * G3 + 8 * c)
                                   : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int u = 0; u < UB; ++u)
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          acc[2 * x] += lo_f(v[u][x]);
          acc[2 * x + 1] += hi_f(v[u][x]);
        }
    }
    __builtin_amdgcn_wave_barrier();   // this slab's list is read before the next one is written
  }
  // entries r = 0 .. R-1 of the wave (lanes c + CPR r) added in order into the lanes of r = 0, then the
  // waves' sums in order: four threads per column add four waves each, combined by a fixed butterfly
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    float t = acc[x];
#pragma unroll
    for (int rr = 1; rr < R; ++rr) t += __shfl(acc[x], c + CPR * rr);
    acc[x] = t;
  }
  if (r == 0) {
#pragma unroll
    for (int x = 0; x < 8; ++x) part[w][8 * c + x] = acc[x];
  }
  if (lane == 0) degs[w] = deg;
  __syncthreads();
  static_assert(NW % 4 == 0 && (4 * G3) % kWave == 0, "whole waves per column group");
  if (tid < 4 * G3) {
    const int col = tid / 4, qp = tid % 4;
    float t = 0.f;
#pragma unroll
    for (int ww = qp * (NW / 4); ww < (qp + 1) * (NW / 4); ++ww) t += part[ww][col];
    t += __shfl_xor(t, 1);
    t += __shfl_xor(t, 2);
    if (qp == 0) gsum[col] = t;
  }
  __syncthreads();
  if (wf < H) {
    // da feature wf of the summed rows: the gate columns of G^'s sum times Wi[wf][.]
    float t = 0.f;
#pragma unroll
    for (int x = 0; x < CW / 2; ++x)
      t += gsum[CW * wp + 2 * x] * lo_f(wreg[x]) + gsum[CW * wp + 2 * x + 1] * hi_f(wreg[x]);
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) t += __shfl_xor(t, off);
    if (wp == 0) rec[((size_t)e * sr + j) * H + wf] = t;
  }
  if (tid == 0) {
    int dsum = 0;
    for (int ww = 0; ww < NW; ++ww) dsum += degs[ww];
    rec[(size_t)E * sr * H + (size_t)e * sr + j] = static_cast<float>(dsum);
  }
}
#endif
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

// Long contraction plan: chunks of the LDS capacity, and edge-type groups so
// that the grid has about 256 workgroups.  Partial and result records hold
// E sa H products then E sa row degrees.
struct SnLong {
  int chunk, nch, tpg;
  long pstride;   // floats per record (a multiple of 64)
  int count;      // floats used per record
};
template <typename S, int H, bool ZFM>
SnLong sn_long_plan(int n_pad, int E, int sa) {
  constexpr int CN = dev::sn_chunk_nodes<S, H, ZFM>();
  SnLong p;
  p.chunk = CN;
  p.nch = (n_pad + CN - 1) / CN;
  // type groups: about 256 workgroups, and at least one (type, row tile)
  // pair for each of the four waves where the types allow
  const int want = (256 + p.nch - 1) / p.nch;
  int ntg = want < 1 ? 1 : (want > E ? E : want);
  const int nrt = sa / 16, tpg4 = (4 + nrt - 1) / nrt;
  if ((E + ntg - 1) / ntg < tpg4) ntg = (E + tpg4 - 1) / tpg4;
  p.tpg = (E + ntg - 1) / ntg;
  p.count = E * sa * (H + 1);
  p.pstride = ((long)p.count + 63) / 64 * 64;
  return p;
}
// Partial records needed by either long contraction (node-major or
// feature-major Z) of this size.
template <typename S, int H>
size_t sn_long_part_floats(int n_pad, int E, int sa) {
  const SnLong a = sn_long_plan<S, H, false>(n_pad, E, sa), b = sn_long_plan<S, H, true>(n_pad, E, sa);
  const int nch = a.nch > b.nch ? a.nch : b.nch;
  return nch > 1 ? (size_t)nch * a.pstride : 0;
}

// out = [P_e (sa x H) for every e | deg_e (sa) for every e], P_e = (bits_e Z)
// over all nodes, for the first sa rows of the slice.
template <typename S, int H, bool ZFM>
hipError_t super_long(const uint8_t* bits, const S* Z, float* part, float* out, int n_pad, int E, int s, int sa,
                      hipStream_t st) {
  const SnLong p = sn_long_plan<S, H, ZFM>(n_pad, E, sa);
  const int ntg = (E + p.tpg - 1) / p.tpg;
  float* dst = p.nch == 1 ? out : part;
  hipLaunchKernelGGL((dev::super_long_kernel<S, H, ZFM>), dim3(p.nch * ntg), dim3(256), 0, st, bits, Z, dst,
                     p.pstride, n_pad, E, s, sa, p.chunk, p.tpg);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || p.nch == 1) return err;
  hipLaunchKernelGGL(dev::sn_reduce_kernel, dim3((p.count / 4 + 63) / 64), dim3(64 * dev::kSnRW), 0, st, part, out,
                     p.nch, p.count, p.pstride);
  return hipGetLastError();
}

// Workspace (floats) of the stand-alone slice calls: long-contraction
// partials, then the records P (R_e X, deg_R), dP (E s H) and dM_s (C_e^T da).
struct SnLayout {
  size_t part, p0, p1, p2, total;
};
template <typename S, int H>
SnLayout sn_layout(int n_pad, int E, int s) {
  auto up = [](size_t x) { return (x + 63) / 64 * 64; };
  SnLayout l;
  const size_t rec = (size_t)sn_long_plan<S, H, false>(n_pad, E, s).pstride;
  l.part = 0;
  l.p0 = up(sn_long_part_floats<S, H>(n_pad, E, s));
  l.p1 = l.p0 + rec;
  l.p2 = l.p1 + up((size_t)E * s * H);
  l.total = (l.p2 + rec) * sizeof(float);
  return l;
}

template <typename S, int H>
hipError_t super_fwd_h(int n_pad, int E, int s, const uint8_t* rows, const uint8_t* cols, const S* X, const S* W,
                       const float* bias, float* a, float* ws, hipStream_t st) {
  const SnLayout L = sn_layout<S, H>(n_pad, E, s);
  float *P = ws + L.p0, *Ms = ws + L.p1, *deg = P + (size_t)E * s * H;
  // P_e = R_e X, deg_R
  hipError_t err = super_long<S, H, false>(rows, X, ws + L.part, P, n_pad, E, s, s, st);
  if (err != hipSuccess) return err;
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
  const SnLayout L = sn_layout<S, H>(n_pad, E, s);
  float *P = ws + L.p0, *dP = ws + L.p1, *dMs = ws + L.p2, *deg = P + (size_t)E * s * H;
  const long np = n_pad;
  // recompute P_e = R_e X and deg_R; dM_s,e = C_e^T da
  hipError_t err = super_long<S, H, false>(rows, X, ws + L.part, P, n_pad, E, s, s, st);
  if (err != hipSuccess) return err;
  if ((err = super_long<S, H, true>(cols_t, da, ws + L.part, dMs, n_pad, E, s, s, st)) != hipSuccess) return err;
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

#if GGNN_DT_BF16
// The record of the fused supernode steps (bf16, H = 32 or 64): rec =
// [P_e (sr x H) | deg_e (sr)] for the first sr rows of the slice, from the
// forward gather (Z = X node-major) where it applies, else from the long
// contraction with its per-chunk partials in ws (the reverse takes
// launch_super_gather_rev where that applies).

#ifndef GGNN_SUPER_GATHER
#define GGNN_SUPER_GATHER 1
#endif
hipError_t launch_super_long_fused(int n_pad, int H, int E, int s, int sr, const void* bits, const void* Z, bool zfm,
                                   float* ws, float* rec, hipStream_t st) {
  if (sr != 16 && sr != 32) return hipErrorInvalidValue;
  const uint8_t* b = static_cast<const uint8_t*>(bits);
  const dev::bf16s* z = static_cast<const dev::bf16s*>(Z);
  using S = dev::bf16s;
  if (GGNN_SUPER_GATHER && !zfm && (H == 32 || H == 64) && n_pad % 64 == 0) {
    // forward: the row slice's sums as a gather (one workgroup of 16 waves per row)
    if (H == 32)
      hipLaunchKernelGGL((dev::super_gather_kernel<32>), dim3(E * sr), dim3(64 * dev::kSnGatherWaves), 0, st, b, z,
                         rec, n_pad, E, s, sr);
    else
      hipLaunchKernelGGL((dev::super_gather_kernel<64>), dim3(E * sr), dim3(64 * dev::kSnGatherWaves), 0, st, b, z,
                         rec, n_pad, E, s, sr);
    return hipGetLastError();
  }
  if (H == 32)
    return zfm ? super_long<S, 32, true>(b, z, ws, rec, n_pad, E, s, sr, st)
               : super_long<S, 32, false>(b, z, ws, rec, n_pad, E, s, sr, st);
  if (H == 64)
    return zfm ? super_long<S, 64, true>(b, z, ws, rec, n_pad, E, s, sr, st)
               : super_long<S, 64, false>(b, z, ws, rec, n_pad, E, s, sr, st);
  return hipErrorInvalidValue;
}
bool super_gather_rev_applies(int n_pad, int H) {
  return GGNN_SUPER_GATHER && (H == 32 || H == 64) && n_pad % 64 == 0;
}
hipError_t launch_super_gather_rev(int n_pad, int H, int E, int s, int sr, const void* bits, const void* ghat,
                                   const void* Wi, float* rec, hipStream_t st) {
  if ((sr != 16 && sr != 32) || !super_gather_rev_applies(n_pad, H)) return hipErrorInvalidValue;
  const uint8_t* b = static_cast<const uint8_t*>(bits);
  const dev::bf16s* g = static_cast<const dev::bf16s*>(ghat);
  const dev::bf16s* w = static_cast<const dev::bf16s*>(Wi);
  if (H == 32)
    hipLaunchKernelGGL((dev::super_gather_rev_kernel<32>), dim3(E * sr), dim3(64 * dev::kSnGatherWaves), 0, st, b, g,
                       w, rec, n_pad, E, s, sr);
  else
    hipLaunchKernelGGL((dev::super_gather_rev_kernel<64>), dim3(E * sr), dim3(64 * dev::kSnGatherWaves), 0, st, b, g,
                       w, rec, n_pad, E, s, sr);
  return hipGetLastError();
}
#endif

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
namespace {
template <int H>
size_t super_ws_h(int n_pad, int E, int s) {
  const size_t a = sn_layout<dev::bf16s, H>(n_pad, E, s).total, b = sn_layout<float, H>(n_pad, E, s).total;
  return a > b ? a : b;
}
// Fused form: the record (super_fused_record_floats, room for 32 rows a
// type), then the long contraction's partials.
template <int H>
size_t super_fused_ws_h(int n_pad, int E) {
  return (((size_t)E * 32 * (H + 1) + 63) / 64 * 64 + sn_long_part_floats<dev::bf16s, H>(n_pad, E, 32)) *
         sizeof(float);
}
}  // namespace

size_t super_workspace(int n_pad, int H, int E, int s) {
  switch (H) {
    case 32: return super_ws_h<32>(n_pad, E, s);
    case 64: return super_ws_h<64>(n_pad, E, s);
    case 128: return super_ws_h<128>(n_pad, E, s);
    case 256: return super_ws_h<256>(n_pad, E, s);
  }
  return 0;
}
size_t super_fused_record_floats(int H, int E) { return ((size_t)E * 32 * (H + 1) + 63) / 64 * 64; }
size_t super_fused_workspace(int n_pad, int H, int E) {
  switch (H) {
    case 32: return super_fused_ws_h<32>(n_pad, E);
    case 64: return super_fused_ws_h<64>(n_pad, E);
  }
  return 0;
}
#endif

}  // namespace ggnn
