// Banded propagation on a 1-bit block band (lossless: A_e has entries in
// {0,1}), in the operand order of Algorithm 1.
//
// Forward (fused): a[k] = sum_e ( sum_s C/U/L_e[k][s] X[k-1+s] ) W_e  (+ deg_e b_e)
//   the three block products of Eq. 3 aggregate the node states first
//   (pre_e = A_e X, kept in registers), then the per-type transform follows
//   in the same workgroup, so the messages never go to HBM.
// Reverse: dM_e[j] = sum_s bits_t[e][j][s] da[j-1+s] = A_e^T da, where the
//   transposed bit band holds the transposed blocks with the sub- and
//   super-diagonal roles swapped (bits_t[e][j][s] = band[e][j-1+s][2-s]^T).
//
// Bit layout (both bands): bits[e][k][s][r][B/8]: row r of block (e, k, s),
// byte c/8 holds columns c..c+7, bit c%8.  A lane expands 8 bits to an
// 8-element matrix-core fragment in registers.
//
// k order of the aggregation: inside a chunk of KC nodes, lane group g owns
// the contiguous columns [g*KC/4, (g+1)*KC/4), so each lane reads KC/32
// consecutive bytes of its bit row.  The staged node tile is kept in LDS in
// fragment order (frag_off below), so every fragment read of a wave covers
// 1 KB of consecutive bytes.
#include "device_common.h"
#include "gru_wave.h"
#include "kernels.h"
#include "lds_dma.h"

namespace ggnn {
namespace dev {

// 8 bits -> 8 elements equal to 0 or 1 (bit i -> element i).
template <typename S> __device__ __forceinline__ frag_t<S> bits_frag(uint32_t byte);
template <> __device__ __forceinline__ bf16x8 bits_frag<bf16s>(uint32_t byte) {
  // byte * 0x8001 holds bit i at position i and again at i + 15, so bit 2k
  // sits at 2k and bit 2k+1 at 16 + 2k.  Masking those two and multiplying
  // by 0x3F80 >> 2k (bf16 1.0 shifted down; exact for 2k <= 6) gives the
  // word of elements 2k and 2k+1 without a shift.
  const uint32_t x = byte * 0x8001u;
  u32x4 w;
#pragma unroll
  for (int k = 0; k < 4; ++k) w[k] = (x & (0x10001u << (2 * k))) * (0x3F80u >> (2 * k));
  return __builtin_bit_cast(bf16x8, w);
}
template <> __device__ __forceinline__ f32x8 bits_frag<float>(uint32_t byte) {
  f32x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<float>((byte >> i) & 1u);
  return r;
}

// NB consecutive bytes (NB in {1, 2, 4, 8, 16}, naturally aligned) as words.
template <int NB> struct RowBytes {
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
      u32x2 v = *reinterpret_cast<const u32x2*>(p);
      w[0] = v[0];
      w[1] = v[1];
    } else {
      u32x4 v = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = v[i];
    }
  }
  __device__ __forceinline__ uint32_t byte(int i) const { return (w[i / 4] >> (8 * (i % 4))) & 0xFFu; }
  __device__ __forceinline__ int popc() const {
    int c = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) c += __popc(w[i]);
    return c;
  }
};

// Two storage elements at p (p 4-byte aligned for bf16, 8-byte for fp32).
__device__ __forceinline__ void store_pair(bf16s* p, uint32_t lo16, uint32_t hi16) {
  *reinterpret_cast<uint32_t*>(p) = (lo16 & 0xFFFFu) | (hi16 << 16);
}

// Fragment order of a staged chunk (KC nodes x H features) in LDS.  The
// eight elements a lane feeds to one matrix-core step (feature h, nodes
// g*KC/4 + 8kk + 0..7 of the chunk) are NV = 8/V 16-byte vectors; for each
// (k step kk, feature tile h/16, vector) the 64 lanes' vectors are
// contiguous.  The LDS serves 16 lanes' 16-byte reads per pass from 64
// four-byte banks, so a fragment read (16 consecutive lanes on 256
// consecutive bytes) never conflicts; reading feature rows at a padded
// pitch instead took two passes per read.
// Staged node chunk: fragment (kk, feature tile h/16).  Split k order: lane
// group g holds nodes g KC/4 + 8 kk + 0..7 of the chunk; contiguous order
// (KCONT): nodes 32 kk + 8 g + 0..7, so that a k step covers 32 consecutive
// nodes.
template <typename S, int H, int KC, bool KCONT = false>
__device__ __forceinline__ int frag_off(int h, int c) {
  const int g = KCONT ? (c / 8) % 4 : c / (KC / 4), kk = KCONT ? c / 32 : (c % (KC / 4)) / 8;
  return fo<S>(kk * (H / 16) + h / 16, h % 16 + 16 * g, c % 8);
}
template <typename S, int H>
__device__ __forceinline__ frag_t<S> load_frag(const S* v, int kk, int m, int lane) {
  return load_fragi<S>(v, kk * (H / 16) + m, lane);
}

// Fused steps: the staged window (X forward, da reverse) has its features
// permuted so that tile m, row i of the aggregation holds feature
//   32 (m / 2) + 8 (i / 4) + 4 (m % 2) + i % 4.
// A lane's accumulators of tiles 2kk and 2kk + 1 then hold eight
// consecutive features, 32kk + 8g .. 32kk + 8g + 7, of its node, so the
// aggregate enters the transform as fragments whose weight operand is eight
// consecutive elements of a row of W_e (reverse) or of W_e^T (forward, when
// the transposed weights are given), one 16-byte load, and the reverse
// stores dM_e with one 16-byte write per pair of tiles.  perm_row(h) is the
// (tile, row) slot of feature h, as 16 * tile + row.
__device__ __forceinline__ int perm_row(int h) {
  const int w = h % 32;
  return 16 * (2 * (h / 32) + (w % 8) / 4) + 4 * (w / 8) + w % 4;
}
// Staging of a chunk of KC nodes x H features for the streamed (large-H)
// forms, in one of two LDS layouts: fragment order (frag_off) or feature
// rows dst[h * VP + c].  The fragment order makes every fragment read a
// single pass, but its writes from node-major rows conflict; feature rows
// are written without conflicts and read in two passes.  Measured on the
// two streamed shapes: fragment order wins at H = 128, feature rows at
// H = 256 (each chunk there is read by fewer waves per byte written).
//
// Nodes [n0, n0 + KC) of a node-major [n][H] array: each thread moves a pair
// of consecutive nodes for eight features and writes 2-element words.
template <typename S, int H, int KC, int VP, int NT, bool ROWS>
__device__ __forceinline__ void stage_nodes_T(S* dst, const S* src, int n0, int tid) {
  constexpr int PAIRS = KC / 2;
  auto at = [&](int h, int c) __attribute__((always_inline)) {   // feature h goes to slot perm_row(h)
    return ROWS ? perm_row(h) * VP + c : frag_off<S, H, KC>(perm_row(h), c);
  };
  for (int lin = tid; lin < PAIRS * (H / 8); lin += NT) {
    const int cp = lin % PAIRS, f0 = (lin / PAIRS) * 8;
    const S* p0 = src + (size_t)(n0 + 2 * cp) * H + f0;
    if constexpr (sizeof(S) == 2) {
      u32x4 x0 = *reinterpret_cast<const u32x4*>(p0);
      u32x4 x1 = *reinterpret_cast<const u32x4*>(p0 + H);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        store_pair(&dst[at(f0 + 2 * i, 2 * cp)], x0[i] & 0xFFFFu, x1[i] & 0xFFFFu);
        store_pair(&dst[at(f0 + 2 * i + 1, 2 * cp)], x0[i] >> 16, x1[i] >> 16);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        typedef float f32x2 __attribute__((ext_vector_type(2)));
        *reinterpret_cast<f32x2*>(&dst[at(f0 + i, 2 * cp)]) = f32x2{p0[i], p0[H + i]};
      }
    }
  }
}

// Columns [n0, n0 + KC) of a feature-major [H][n_pad] array (16-byte
// copies: a unit is one fragment vector).  In fragment order the feature
// runs fastest over the threads, so the 16 lanes of one LDS pass write 16
// different fragment rows (distinct banks).
// PERM: feature h goes to the (tile, row) slot perm_row(h) (reverse step).
template <typename S, int H, int KC, int VP, int NT, bool ROWS, bool PERM>
__device__ __forceinline__ void stage_cols(S* dst, const S* src, int n_pad, int n0, int tid) {
  constexpr int V = 16 / sizeof(S);
  for (int lin = tid; lin < H * (KC / V); lin += NT) {
    const int h = ROWS ? lin / (KC / V) : lin % H;
    const int c = ROWS ? (lin % (KC / V)) * V : (lin / H) * V;
    const int hs = PERM ? perm_row(h) : h;
    *reinterpret_cast<u32x4*>(&dst[ROWS ? hs * VP + c : frag_off<S, H, KC>(hs, c)]) =
        *reinterpret_cast<const u32x4*>(src + (size_t)h * n_pad + n0 + c);
  }
}

template <typename S, int H, int B>
struct BitsCfg {
  static constexpr int V = 16 / sizeof(S);
  // Stage the three neighbouring node blocks once per workgroup when they fit
  // in 64 KB; otherwise stream KC-node chunks per edge type.
  static constexpr bool ALL = 3 * H * (B + V) * (int)sizeof(S) <= 65536;
  static constexpr int KC = ALL ? B : (B < 64 ? B : 64);
  static constexpr int NBUF = ALL ? 3 : 1;
  static constexpr int VP = KC + V;
  static constexpr bool ROWS = !ALL && H >= 256;   // streamed chunks kept as feature rows
  static constexpr int RB = KC / 32;        // bit-row bytes per lane per chunk (= k steps per chunk)
  // k order of the staged blocks (ALL): contiguous at RB = 4, 8 (B = 128,
  // 256), the bit bytes re-ordered in registers after each type's load; a
  // k step then covers 32 consecutive block columns, and in a band much
  // narrower than B most steps hold no edge into a wave's rows and are
  // skipped whole.  Split otherwise (a lane's bytes as loaded).
  static constexpr bool KCONT = ALL && (RB == 4 || RB == 8);
  static constexpr int RPW = H >= 256 ? 16 : 32;   // rows per wave
  static constexpr int NTW = RPW / 16;      // 16-row tiles per wave
  // Smallest workgroup (waves) launched; the fp32 forms with H >= 128 and
  // the bf16 forms with H = 256 keep at least two waves (their one-wave
  // forms are not built: the code generator fails on them).
  static constexpr int MINW = ((sizeof(S) == 4 && H >= 128) || H >= 256) && B / RPW >= 2 ? 2 : 1;
  // Forward, H <= 64 with the blocks staged: the transform's weight
  // fragments are read straight from global memory (L1/L2 resident, issued
  // at the top of each type and used at its end), so no weight staging sits
  // in the prologue and the type loop has no barrier.
  static constexpr bool WDIR = ALL && H <= 64;
  static constexpr int WP = H + V;          // W^T row pitch (LDS chunks otherwise)
};

// ---------------------------------------------------------------------------
// Fused step on a bit band, forward (REV = false) or reverse (REV = true).
// Workgroup: RPW*WAVES rows of block row k (columns of block column k in
// the reverse).
//   forward:  a[k]  = sum_e (sum_s bits[e][k][s] X[k-1+s]) W_e   (+ deg_e bias_e)
//   reverse:  dM_e[k] = sum_s bits_t[e][k][s] da[k-1+s]          (stored, dt)
//             dX[k] = dX_in[k] + sum_e dM_e[k] W_e^T
// Aggregation D[h][r]: A operand = staged feature rows of X (transposed on
// the LDS write) or of da (feature-major already: plain copies), B operand =
// bit rows expanded in registers.  Transform D'[h_out][r]: A operand = rows
// of W_e^T (forward) or W_e (reverse), B operand = the aggregation
// accumulators themselves (accumulator-compatible k order; forward: split hi
// + lo in bf16 mode; reverse: the rounded dM that is stored).  Lanes then
// hold four consecutive features of one node: 16-byte fp32 stores of a / dX.
// WDIR: the weight fragments come straight from global memory, requested at
// the top of type e and consumed after its aggregation; the type loop has no
// barrier (waves drift freely and hide each other's latencies) and the bit
// rows of the next two types are in flight while a type is computed.
// Otherwise the weights are staged per type in LDS in 64-row chunks.
// TG type groups (WDIR only): the workgroup has TG * WAVES waves; wave w
// takes rows as wave w % WAVES and the types of group w / WAVES (a
// contiguous range), so TG waves share a SIMD and overlap one another's VALU,
// LDS and matrix work.  The groups' partial sums meet in LDS at the end (over
// the staged blocks): with TG = NTW = 2 group g completes row tile g (its own
// partial plus the other group's), otherwise group 0 completes both; either
// way a = (group 0 partial) + (group 1 partial).
// GRU, forward (WDIR): the node update of Eq. 1 runs on the completed
// aggregate in the same workgroup, so `a` goes to memory only for the
// reverse pass and the next state X' and the gates (r | z | n) are written
// here.  Wi^T and U^T are staged in LDS with the blocks; the GRU products
// take a (hi + lo in bf16 mode), h and r*h as operand fragments straight
// from registers (accumulator-compatible order).
// SN (supernodes next to the band, bf16 direct-weight forms): the first 32
// nodes are supernodes.  Per edge type the aggregation gets a fourth block,
// the supernode window (nodes 0..31 of X forward, of da reverse; staged once)
// against the slice bits of each row ([E][n_pad][sn_s/8]: forward the
// column slice, edges from a supernode into this row; reverse the
// transposed row slice, edges from this node into a supernode).  The rows of
// the supernodes themselves get their whole per-type aggregate from the
// record sn_rec = [P_e (sn_sr x H) | deg_e (sn_sr)], their sums over all nodes
// (forward R_e X, reverse C_e^T da) from a launch before the step: the wave holding rows 0..31
// copies P_e of its rows into LDS (global -> LDS, issued at the top of the
// type, waited for after the aggregation) and adds it to the aggregate (the
// record's first sn_sr rows, 16 or 32: the supernodes with edges).
// GRU, reverse (WDIR): the completed dX of these nodes is dL/dh' of the
// previous step's GRU, whose reverse (gru_bwd_wave) runs right here: it
// writes that step's da (feature-major), dh and G^, so one launch covers a
// whole reverse step.  Wi and U are staged in LDS (plain copies) with the
// blocks; dX itself is written only when `out` is not NULL.
// ---------------------------------------------------------------------------
#ifndef GGNN_BITS_TG0_PCT_REV
#define GGNN_BITS_TG0_PCT_REV 50
#endif
#ifndef GGNN_BITS_GW_TG0
#define GGNN_BITS_GW_TG0 0
#endif
#ifndef GGNN_BITS_DM_LDS
#define GGNN_BITS_DM_LDS 1
#endif
constexpr int kSnFused = 32;   // supernodes handled inside the fused step kernels
template <typename S, int H, int B, int WAVES, bool WDIR, int TG, bool REV, bool GRU, bool SN = false>
__global__ __launch_bounds__(TG * WAVES * kWave) void step_bits_kernel(
    const uint8_t* __restrict__ bits, const S* __restrict__ X, const S* __restrict__ W, const S* __restrict__ Wt,
    const float* __restrict__ bias,
    float* out, int n_pad, int E, const float* dX_in, S* __restrict__ dM, long ldm, const S* __restrict__ Wi,
    const S* __restrict__ U, const float* __restrict__ bg, S* __restrict__ h_out, S* __restrict__ saved,
    const S* __restrict__ rh_h, const S* __restrict__ rh_saved, S* __restrict__ rh_da, float* __restrict__ rh_dh,
    S* __restrict__ rh_ghat, const uint8_t* __restrict__ sn_bits, const float* __restrict__ sn_rec, int sn_s,
    int sn_sr) {
  using C = BitsCfg<S, H, B>;
  constexpr int NT = TG * WAVES * kWave;
  constexpr int V = C::V, KC = C::KC, VP = C::VP, RB = C::RB, NTW = C::NTW, WP = C::WP;
  constexpr int MT = H / 16, HK = H / 32;
  constexpr int WC = WDIR ? H : (H < 64 ? H : 64);   // weight rows per chunk
  constexpr int NP = (sizeof(S) == 2 && !REV) ? 2 : 1;
  constexpr int ROWB = B / 8;
  static_assert(!WDIR || C::WDIR, "direct weights need the staged blocks and H <= 64");
  static_assert(TG == 1 || WDIR, "type groups need the barrier-free loop");
  static_assert(TG == 1 || (TG - 1) * WAVES * kWave * NTW * MT * 16 <= (int)(C::NBUF * H * VP * sizeof(S)),
                "partial sums must fit in the staged-block space");
  static_assert(!GRU || WDIR, "the GRU epilogues are direct-weight forms");
  static_assert(!SN || (WDIR && sizeof(S) == 2 && C::RPW == kSnFused), "supernodes: bf16 direct-weight forms");
  constexpr int GWN = !GRU ? 8 : 2 * 3 * H * H;   // Wi and U in fragment order
  __shared__ __attribute__((aligned(16))) S vt[C::NBUF][H * VP];
  __shared__ __attribute__((aligned(16))) S wt[WDIR ? 8 : WC * WP];
  __shared__ __attribute__((aligned(16))) S gw[GWN];
  // SN: supernode window (fragment order, features permuted as the blocks)
  // and, per type group, the record rows of the wave holding nodes 0..31
  // (NTW x MT 1 KB copies, one 16-byte unit per lane each).
  __shared__ __attribute__((aligned(16))) S hubw[SN ? kSnFused * H : 8];
  // reverse, bf16 with the blocks staged: each wave's dM tile (RPW rows,
  // pitch DMP), for row-ordered stores
  constexpr bool DMS = REV && C::ALL && sizeof(S) == 2 && GGNN_BITS_DM_LDS;
  constexpr int DMP = H + 8;
  __shared__ __attribute__((aligned(16))) S dms[DMS ? TG * WAVES * C::RPW * DMP : 8];
  __shared__ __attribute__((aligned(1024))) float recb[SN ? TG * NTW * MT * 256 : 4];

  const int nb = n_pad / B;
  constexpr int NW = C::RPW * WAVES;
  const int tiles_per_row = B / NW;
  const int t = xcd_swizzle(blockIdx.x, gridDim.x);
  const int k = t / tiles_per_row;
  const int tid = threadIdx.x, wave = (tid / kWave) % WAVES, lane = tid % kWave;
  const int tg = tid / (WAVES * kWave);
  const int q = lane % 16, g = lane / 16;
  const int rw = (t % tiles_per_row) * NW + C::RPW * wave;   // first row of this wave
  const int s_lo = (k == 0) ? 1 : 0;
  const int s_hi = (k == nb - 1) ? 1 : 2;
  // this wave's types: group 0 takes the first TG0_PCT percent in the
  // reverse with two groups, else an even split
  const int e_mid = (REV && TG == 2 && GGNN_BITS_TG0_PCT_REV != 50) ? (E * GGNN_BITS_TG0_PCT_REV + 50) / 100 : E / 2;
  const int e_lo = TG == 2 ? (tg == 0 ? 0 : e_mid) : tg * E / TG;
  const int e_hi = TG == 2 ? (tg == 0 ? e_mid : E) : (tg + 1) * E / TG;

  // The bit rows of the first types are requested before the staging, so
  // their latency overlaps it; later types' rows are loaded while the current
  // one is computed (one type ahead, two with WDIR).
  RowBytes<RB> nx1[3][NTW], nx2[3][NTW];
  auto load_type = [&](int e, RowBytes<RB> (&dst)[3][NTW]) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      if (s < s_lo || s > s_hi) continue;
      const uint8_t* brow = bits + ((((size_t)e * nb + k) * 3 + s) * B + rw + q) * ROWB + g * (KC / 32);
#pragma unroll
      for (int n = 0; n < NTW; ++n) dst[s][n].load(brow + (size_t)16 * n * ROWB);
    }
  };
  if constexpr (C::ALL) {
    if (e_lo < e_hi) load_type(e_lo, nx1);
  }
  if constexpr (WDIR) {
    if (e_lo + 1 < e_hi) load_type(e_lo + 1, nx2);
  }

  // Staging of the three blocks in fragment order, vt[s][frag_off(f, c)] =
  // node (k-1+s)*B + c, feature f.  Forward: V x V tiles of node-major X,
  // transposed in registers (loads of whole 128-byte lines), one 16-byte
  // store per tile row.  Reverse: plain 16-byte copies of feature-major da.
  // With the GRU fused, Wi and U follow as further units (fragment order);
  // they are only read by the epilogue, so they are staged after the type
  // loop, while the waves of the other type group are still busy.  Each
  // thread issues the loads of up to PB units before its writes.
  constexpr int XT = !REV ? (KC / V) * (H / V) : H * (KC / V);   // units per block: tiles / 16-byte copies
  constexpr int GT = !REV ? (H / V) * (3 * H / V) : H * (3 * H / V);   // units per GRU weight
  const int nx = (s_hi - s_lo + 1) * XT;
  const int total = nx + (GRU ? 2 * GT : 0);
  auto stage_units = [&](int lo, int hi, int nthr, int thr) __attribute__((always_inline)) {
    if constexpr (C::ALL && !REV) {
      constexpr int PB = 2;
      for (int base = lo; base < hi; base += PB * nthr) {
        u32x4 r[PB][V];
#pragma unroll
        for (int u = 0; u < PB; ++u) {
          const int lin = base + u * nthr + thr;
          if (lin >= hi) {
          } else if (lin < nx) {
            const int slot = s_lo + lin / XT, rem = lin % XT;
            const int cq = rem % (KC / V), fq = rem / (KC / V);
            tile_load<S>(r[u], X + (size_t)((k - 1 + slot) * B + V * cq) * H + V * fq, H);
          } else {
            const int w = lin - nx, m = w / GT, rem = w % GT;
            const int hq = rem % (H / V), cq = rem / (H / V);
            tile_load<S>(r[u], (m ? U : Wi) + (size_t)(V * hq) * 3 * H + V * cq, 3 * H);
          }
        }
#pragma unroll
        for (int u = 0; u < PB; ++u) {
          const int lin = base + u * nthr + thr;
          if (lin >= hi) {
          } else if (lin < nx) {
            const int slot = s_lo + lin / XT, rem = lin % XT;
            const int cq = rem % (KC / V), fq = rem / (KC / V);
#pragma unroll
            for (int x = 0; x < V; ++x)
              *reinterpret_cast<u32x4*>(&vt[slot][frag_off<S, H, KC, C::KCONT>(perm_row(V * fq + x), V * cq)]) =
                  tile_row_T<S>(r[u], x);
          } else {
            const int w = lin - nx, m = w / GT, rem = w % GT;
            const int hq = rem % (H / V), cq = rem / (H / V);
            // row x of the transposed tile: gate column V*cq + x, input
            // features V*hq .. V*hq + V - 1 (runs of four)
#pragma unroll
            for (int x = 0; x < V; ++x) {
              const u32x4 o = tile_row_T<S>(r[u], x);
              const S* po = reinterpret_cast<const S*>(&o);
              const int col = V * cq + x;
#pragma unroll
              for (int i = 0; i < V; i += 4)
                put4<S>(gw, gru_fwd_idx<S, H>(m, col / 16, (V * hq + i) / 32), col % 16, V * hq + i, po + i);
            }
          }
        }
      }
    } else if constexpr (C::ALL) {
      constexpr int PB = 8;
      for (int base = lo; base < hi; base += PB * nthr) {
        u32x4 r[PB];
#pragma unroll
        for (int u = 0; u < PB; ++u) {
          const int lin = base + u * nthr + thr;
          if (lin >= hi) {
          } else if (lin < nx) {
            const int slot = s_lo + lin / XT, rem = lin % XT;
            const int h = rem / (KC / V), c = (rem % (KC / V)) * V;
            r[u] = *reinterpret_cast<const u32x4*>(X + (size_t)h * n_pad + (k - 1 + slot) * B + c);
          } else {
            const int w = lin - nx, m = w / GT, rem = w % GT;
            const int h = rem / (3 * H / V), c = (rem % (3 * H / V)) * V;
            r[u] = *reinterpret_cast<const u32x4*>((m ? U : Wi) + (size_t)h * 3 * H + c);
          }
        }
#pragma unroll
        for (int u = 0; u < PB; ++u) {
          const int lin = base + u * nthr + thr;
          if (lin >= hi) {
          } else if (lin < nx) {
            const int slot = s_lo + lin / XT, rem = lin % XT;
            const int h = rem / (KC / V), c = (rem % (KC / V)) * V;
            *reinterpret_cast<u32x4*>(&vt[slot][frag_off<S, H, KC, C::KCONT>(perm_row(h), c)]) = r[u];
          } else {
            const int w = lin - nx, m = w / GT, rem = w % GT;
            const int h = rem / (3 * H / V), c = (rem % (3 * H / V)) * V;
            // input feature h, gate columns c .. c + V - 1 (runs of four)
            const S* po = reinterpret_cast<const S*>(&r[u]);
#pragma unroll
            for (int i = 0; i < V; i += 4)
              put4<S>(gw, gru_rev_idx<S, H>(m, h / 16, (c + i) / H, ((c + i) % H) / 32), h % 16, (c + i) % H,
                      po + i);
          }
        }
      }
    }
  };
  // SN: the supernode window (nodes 0..31) in the layout of a staged block
  // chunk of 32 nodes; its loads are issued before the blocks' staging and
  // written after it.  Forward unit: two nodes x eight features of
  // node-major X; reverse unit: 16 bytes (V nodes) of one feature row of da.
  constexpr int HU = SN ? (!REV ? (kSnFused / 2) * (H / 8) : H * (kSnFused / V)) : 1;
  constexpr int HPT = (HU + NT - 1) / NT;
  u32x4 hx[SN ? HPT : 1][SN && !REV ? 2 : 1];
  if constexpr (SN) {
#pragma unroll
    for (int u = 0; u < HPT; ++u) {
      const int lin = u * NT + tid;
      if (lin < HU) {
        if constexpr (!REV) {
          const int cp = lin % (kSnFused / 2), f0 = (lin / (kSnFused / 2)) * 8;
          hx[u][0] = *reinterpret_cast<const u32x4*>(X + (size_t)(2 * cp) * H + f0);
          hx[u][!REV ? 1 : 0] = *reinterpret_cast<const u32x4*>(X + (size_t)(2 * cp + 1) * H + f0);
        } else {
          const int h = lin % H, c = (lin / H) * V;
          hx[u][0] = *reinterpret_cast<const u32x4*>(X + (size_t)h * n_pad + c);
        }
      }
    }
  }
  if constexpr (C::ALL) {
    stage_units(0, nx, NT, tid);
    if constexpr (SN) {
#pragma unroll
      for (int u = 0; u < HPT; ++u) {
        const int lin = u * NT + tid;
        if (lin < HU) {
          if constexpr (!REV) {
            const int cp = lin % (kSnFused / 2), f0 = (lin / (kSnFused / 2)) * 8;
            const u32x4 x0 = hx[u][0], x1 = hx[u][!REV ? 1 : 0];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              store_pair(&hubw[frag_off<S, H, kSnFused>(perm_row(f0 + 2 * i), 2 * cp)], x0[i] & 0xFFFFu,
                         x1[i] & 0xFFFFu);
              store_pair(&hubw[frag_off<S, H, kSnFused>(perm_row(f0 + 2 * i + 1), 2 * cp)], x0[i] >> 16,
                         x1[i] >> 16);
            }
          } else {
            const int h = lin % H, c = (lin / H) * V;
            *reinterpret_cast<u32x4*>(&hubw[frag_off<S, H, kSnFused>(perm_row(h), c)]) = hx[u][0];
          }
        }
      }
    }
    __syncthreads();
  }

  f32x4 acc[NTW][MT];
#pragma unroll
  for (int n = 0; n < NTW; ++n)
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[n][m] = f32x4{0.f, 0.f, 0.f, 0.f};

  // WDIR weight fragments: A row o = 16 mo + q, k values h in the
  // accumulator-compatible order 32 kk + 4 g + {0..3}, 32 kk + 16 + 4 g + {0..3}.
  // Forward: element (o, h) is W[e][h][o] (a column of W: 2-byte gathers);
  // reverse: it is W[e][o][h] (a row: two 8-byte loads).
  frag_t<S> wf[WDIR ? H / 16 : 1][WDIR ? HK : 1];
  auto load_wfrags = [&](int e) __attribute__((always_inline)) {
    if constexpr (WDIR) {
      const S* we = W + (size_t)e * H * H;
#pragma unroll
      for (int mo = 0; mo < H / 16; ++mo)
#pragma unroll
        for (int kk = 0; kk < HK; ++kk) {
          if constexpr (REV) {
            wf[mo][kk] = load8(we + (size_t)(16 * mo + q) * H + 32 * kk + 8 * g);   // features 32kk + 8g + 0..7
          } else if (Wt != nullptr) {
            // W_e^T row 16mo + q: features 32kk + 8g + 0..7
            wf[mo][kk] = load8(Wt + (size_t)e * H * H + (size_t)(16 * mo + q) * H + 32 * kk + 8 * g);
          } else {
            // column 16mo + q of W_e, rows 32kk + 8g + 0..7 (2-byte gathers)
            const S* p = we + (size_t)(32 * kk + 8 * g) * H + 16 * mo + q;
            if constexpr (sizeof(S) == 2) {
              u32x4 w;
#pragma unroll
              for (int d = 0; d < 4; ++d)
                w[d] = static_cast<uint32_t>(p[(size_t)(2 * d) * H]) |
                       (static_cast<uint32_t>(p[(size_t)(2 * d + 1) * H]) << 16);
              wf[mo][kk] = __builtin_bit_cast(bf16x8, w);
            } else {
#pragma unroll
              for (int x = 0; x < 8; ++x) wf[mo][kk][x] = p[(size_t)x * H];
            }
          }
        }
    }
  };

  // Per-type weight chunks in LDS (not WDIR): chunk rows o in [oc, oc + WC),
  // wt[o][h] = W[e][h][oc + o] (forward, transposed on the write) or
  // W[e][oc + o][h] (reverse, plain copies); H * WC / V 16-byte units,
  // prefetched into registers during the aggregation.
  constexpr int WU = WDIR ? 1 : (H * (WC / V) + NT - 1) / NT;
  u32x4 wreg[WU];
  auto load_w = [&](int e, int oc) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < WU; ++u) {
      const int lin = u * NT + tid;
      if ((H * (WC / V)) % NT == 0 || lin < H * (WC / V)) {
        if constexpr (REV) {
          const int o = lin / (H / V), h8 = (lin % (H / V)) * V;
          wreg[u] = *reinterpret_cast<const u32x4*>(W + (size_t)e * H * H + (size_t)(oc + o) * H + h8);
        } else {
          const int h = lin / (WC / V), o8 = (lin % (WC / V)) * V;
          wreg[u] = *reinterpret_cast<const u32x4*>(W + (size_t)e * H * H + (size_t)h * H + oc + o8);
        }
      }
    }
  };
  auto store_w = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < WU; ++u) {
      const int lin = u * NT + tid;
      if ((H * (WC / V)) % NT == 0 || lin < H * (WC / V)) {
        if constexpr (REV) {
          const int o = lin / (H / V), h8 = (lin % (H / V)) * V;
          *reinterpret_cast<u32x4*>(&wt[o * WP + h8]) = wreg[u];
        } else {
          const int h = lin / (WC / V), o8 = (lin % (WC / V)) * V;
          const S* pw = reinterpret_cast<const S*>(&wreg[u]);
#pragma unroll
          for (int x = 0; x < V; ++x) wt[(o8 + x) * WP + h] = pw[x];
        }
      }
    }
  };
  for (int e = e_lo; e < e_hi; ++e) {
    if constexpr (WDIR) {
      load_wfrags(e);      // consumed after the aggregation below
    } else {
      load_w(e, 0);        // in flight during the aggregation below
    }
    f32x4 pre[NTW][MT];
#pragma unroll
    for (int n = 0; n < NTW; ++n)
#pragma unroll
      for (int m = 0; m < MT; ++m) pre[n][m] = f32x4{0.f, 0.f, 0.f, 0.f};
    int deg[NTW];
#pragma unroll
    for (int n = 0; n < NTW; ++n) deg[n] = 0;
    RowBytes<RB> cur[3][NTW];
    if constexpr (C::ALL) {
#pragma unroll
      for (int s = 0; s < 3; ++s)
#pragma unroll
        for (int n = 0; n < NTW; ++n) {
          cur[s][n] = nx1[s][n];
          if constexpr (WDIR) nx1[s][n] = nx2[s][n];
        }
      if constexpr (WDIR) {
        if (e + 2 < e_hi) load_type(e + 2, nx2);
      } else {
        if (e + 1 < e_hi) load_type(e + 1, nx1);
      }
      if constexpr (C::KCONT) {
        // contiguous k order; a block with no edge into the wave's rows
        // stays all zero (and is skipped below)
        const uint32_t godd = static_cast<uint32_t>(g & 1);
#pragma unroll
        for (int s = 0; s < 3; ++s) {
          if (s < s_lo || s > s_hi) continue;
          uint32_t any = 0u;
#pragma unroll
          for (int n = 0; n < NTW; ++n)
#pragma unroll
            for (int i = 0; i < RowBytes<RB>::NW; ++i) any |= cur[s][n].w[i];
          if (__builtin_amdgcn_ballot_w64(any != 0u) == 0) continue;
#pragma unroll
          for (int n = 0; n < NTW; ++n) bytes_to_contiguous<RB>(cur[s][n].w, godd);
        }
      }
    }
    // SN: the slice bytes of this wave's rows (window columns 8g .. 8g + 7)
    // and, in the wave holding nodes 0..31, P_e of its rows (into LDS) and
    // their degrees; all in flight during the aggregation below.
    uint32_t hb[SN ? NTW : 1];
    float hdeg[SN ? NTW : 1];
    const bool hub_wave = SN && k * B + rw < kSnFused;   // wave-uniform
    if constexpr (SN) {
#pragma unroll
      for (int n = 0; n < NTW; ++n) {
        hb[n] = sn_bits[((size_t)e * n_pad + k * B + rw + 16 * n + q) * (size_t)(sn_s / 8) + g];
        hdeg[n] = 0.f;
      }
      if (hub_wave) {
        const uint32_t base = (uint32_t)(uintptr_t)recb + (uint32_t)(__builtin_amdgcn_readfirstlane(tg) * NTW * MT * 1024);
#pragma unroll
        for (int n = 0; n < NTW; ++n) {
          if (16 * n >= sn_sr) continue;
#pragma unroll
          for (int m = 0; m < MT; ++m)
            dma16(sn_rec + ((size_t)e * sn_sr + 16 * n + q) * H + 32 * (m / 2) + 8 * g + 4 * (m % 2),
                  base + (uint32_t)((n * MT + m) * 1024));
        }
        if (!REV && bias) {
#pragma unroll
          for (int n = 0; n < NTW; ++n)
            if (16 * n < sn_sr) hdeg[n] = sn_rec[(size_t)E * sn_sr * H + (size_t)e * sn_sr + 16 * n + q];
        }
      }
    }
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      if (s < s_lo || s > s_hi) continue;
      const uint8_t* brow = bits + ((((size_t)e * nb + k) * 3 + s) * B + rw + q) * ROWB;
      for (int c0 = 0; c0 < B; c0 += KC) {
        if constexpr (!C::ALL) {
          __syncthreads();
          if constexpr (REV) {
            stage_cols<S, H, KC, VP, NT, C::ROWS, true>(vt[0], X, n_pad, (k - 1 + s) * B + c0, tid);
          } else {
            stage_nodes_T<S, H, KC, VP, NT, C::ROWS>(vt[0], X, (k - 1 + s) * B + c0, tid);
          }
          __syncthreads();
        }
        const S* v = vt[C::ALL ? s : 0];
        RowBytes<RB> rb[NTW];
#pragma unroll
        for (int n = 0; n < NTW; ++n) {
          if constexpr (C::ALL) {
            rb[n] = cur[s][n];
          } else {
            rb[n].load(brow + (size_t)16 * n * ROWB + (c0 + g * (KC / 4)) / 8);
          }
          if (!REV && bias) deg[n] += rb[n].popc();
        }
#pragma unroll
        for (int kk = 0; kk < RB; ++kk) {
          if constexpr (C::KCONT) {
            // a k step with no edge into the wave's rows adds exact zeros
            uint32_t any_step = 0u;
#pragma unroll
            for (int n = 0; n < NTW; ++n) any_step |= rb[n].byte(kk);
            if (__builtin_amdgcn_ballot_w64(any_step != 0u) == 0) continue;
          }
          frag_t<S> bf[NTW];
#pragma unroll
          for (int n = 0; n < NTW; ++n) bf[n] = bits_frag<S>(rb[n].byte(kk));
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const frag_t<S> af = C::ROWS ? load8(&v[(16 * m + q) * VP + g * (KC / 4) + 8 * kk])
                                         : load_frag<S, H>(v, kk, m, lane);
#pragma unroll
            for (int n = 0; n < NTW; ++n) mma(pre[n][m], af, bf[n]);
          }
        }
      }
    }
    if constexpr (SN) {
      // the supernode block, and the record of the supernode rows
      uint32_t any = 0u;
#pragma unroll
      for (int n = 0; n < NTW; ++n) any |= hb[n];
      if (__builtin_amdgcn_ballot_w64(any != 0u) != 0) {
        frag_t<S> bf[NTW];
#pragma unroll
        for (int n = 0; n < NTW; ++n) {
          bf[n] = bits_frag<S>(hb[n]);
          if (!REV && bias) deg[n] += __popc(hb[n]);
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const frag_t<S> af = load_frag<S, H>(hubw, 0, m, lane);
#pragma unroll
          for (int n = 0; n < NTW; ++n) mma(pre[n][m], af, bf[n]);
        }
      }
      if (hub_wave) {
        wait_copies<0>();
        asm volatile("" ::: "memory");
        const float* rbuf = recb + tg * NTW * MT * 256;
#pragma unroll
        for (int n = 0; n < NTW; ++n) {
          if (16 * n >= sn_sr) continue;
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const f32x4 r = *reinterpret_cast<const f32x4*>(rbuf + ((n * MT + m) * 64 + lane) * 4);
#pragma unroll
            for (int j = 0; j < 4; ++j) pre[n][m][j] += r[j];
          }
        }
      }
    }
    // pre^T in accumulator layout: lane (node q), features 16m + 4g + j.
    frag_t<S> pf[NP][NTW][HK];
#pragma unroll
    for (int n = 0; n < NTW; ++n)
#pragma unroll
      for (int kk = 0; kk < HK; ++kk) {
        float v8[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v8[j] = pre[n][2 * kk][j];
          v8[4 + j] = pre[n][2 * kk + 1][j];
        }
        if constexpr (NP == 2) {
          split8(v8, pf[0][n][kk], pf[NP - 1][n][kk]);
        } else {
          pf[0][n][kk] = pack8<S>(v8);
        }
      }
    if constexpr (REV && DMS) {
      // dM_e rows of this wave's nodes through the wave's LDS tile: written
      // as the lanes hold them (node 16n + q, features 32kk + 8g .. + 7),
      // read back in row order, so that each store covers 1 KB of
      // consecutive rows (stored from the lanes, every store touched 16 rows
      // for 64 bytes each).  Wave-private, so no barrier.
      S* dt = dms + (tg * WAVES + wave) * (C::RPW * DMP);
#pragma unroll
      for (int n = 0; n < NTW; ++n)
#pragma unroll
        for (int kk = 0; kk < HK; ++kk)
          *reinterpret_cast<u32x4*>(dt + (16 * n + q) * DMP + 32 * kk + 8 * g) = __builtin_bit_cast(u32x4, pf[0][n][kk]);
      S* rows0 = dM + ((size_t)e * ldm + k * B + rw) * H;
#pragma unroll
      for (int i = 0; i < C::RPW * H / 8 / kWave; ++i) {
        const int u = i * kWave + lane;   // 16-byte unit u of the wave's rows: row u / (H / 8)
        const int r = u / (H / 8), c = (u % (H / 8)) * 8;
        *reinterpret_cast<u32x4*>(rows0 + (size_t)r * H + c) = *reinterpret_cast<const u32x4*>(dt + r * DMP + c);
      }
    } else if constexpr (REV) {
      // dM_e rows of this wave's nodes (node-major, rows of type e start at
      // row e * ldm): features 32kk + 8g .. 32kk + 8g + 7 (rev_row order).
#pragma unroll
      for (int n = 0; n < NTW; ++n) {
        S* row = dM + ((size_t)e * ldm + k * B + rw + 16 * n + q) * H + 4 * g;
#pragma unroll
        for (int kk = 0; kk < HK; ++kk) {
          if constexpr (sizeof(S) == 2) {
            *reinterpret_cast<u32x4*>(row + 32 * kk + 4 * g) = __builtin_bit_cast(u32x4, pf[0][n][kk]);
          } else {
            const f32x8 w = pf[0][n][kk];
            *reinterpret_cast<f32x4*>(row + 32 * kk + 4 * g) = f32x4{w[0], w[1], w[2], w[3]};
            *reinterpret_cast<f32x4*>(row + 32 * kk + 4 * g + 4) = f32x4{w[4], w[5], w[6], w[7]};
          }
        }
      }
    }
    if constexpr (WDIR) {
#pragma unroll
      for (int mo = 0; mo < H / 16; ++mo)
#pragma unroll
        for (int kk = 0; kk < HK; ++kk)
#pragma unroll
          for (int n = 0; n < NTW; ++n)
#pragma unroll
            for (int part = 0; part < NP; ++part) mma(acc[n][mo], wf[mo][kk], pf[part][n][kk]);
    } else {
      for (int oc = 0; oc < H; oc += WC) {
        __syncthreads();
        store_w();
        __syncthreads();
        if (oc + WC < H) load_w(e, oc + WC);   // next chunk, in flight during this one
#pragma unroll
        for (int mo = 0; mo < WC / 16; ++mo)
#pragma unroll
          for (int kk = 0; kk < HK; ++kk) {
            const frag_t<S> af = load8(&wt[(16 * mo + q) * WP + 32 * kk + 8 * g]);
#pragma unroll
            for (int n = 0; n < NTW; ++n)
#pragma unroll
              for (int part = 0; part < NP; ++part) mma(acc[n][oc / 16 + mo], af, pf[part][n][kk]);
          }
      }
    }
    if (!REV && bias) {
#pragma unroll
      for (int n = 0; n < NTW; ++n) {
        int d = deg[n];
        d += __shfl_xor(d, 16);
        d += __shfl_xor(d, 32);
        float fd = static_cast<float>(d);
        if constexpr (SN) fd += hdeg[n];
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[n][m][j] += fd * bias[e * H + 16 * m + 4 * g + j];
      }
    }
  }
  // Row tiles this wave completes: all of them, or with two groups and two
  // tiles per wave, tile tg.
  constexpr bool SPLIT = (TG == 2 && NTW == 2);
  // GRU weights for the epilogue (read after the barriers below).
  if constexpr (C::ALL && GRU) {
    if (GGNN_BITS_GW_TG0 && TG == 2) {
      if (tg == 0) stage_units(nx, total, WAVES * kWave, tid);   // the group that finishes first
    } else {
      stage_units(nx, total, NT, tid);
    }
  }
  // Epilogue operands of this wave's tile requested now, in flight across
  // the barriers: h (forward) or the gates of the previous step (reverse).
  // h as raw 16-byte units in bf16 (features 32kk + 8g.., split at use:
  // split_tiles16), as fragments in fp32.
  constexpr bool HRAW = sizeof(S) == 2;
  frag_t<S> hf_pre[(GRU && !REV && SPLIT && !HRAW) ? H / 32 : 1];
  u32x4 hraw_pre[(GRU && !REV && SPLIT && HRAW) ? H / 32 : 1];
  GruBwdIn<S, H> gin_pre;
  if constexpr (GRU && SPLIT) {
    const int node = k * B + rw + 16 * tg + q;
    if constexpr (!REV) {
#pragma unroll
      for (int kk = 0; kk < H / 32; ++kk) {
        if constexpr (HRAW)
          hraw_pre[kk] = *reinterpret_cast<const u32x4*>(X + (size_t)node * H + 32 * kk + 8 * g);
        else
          hf_pre[kk] = rowfrag<S>(X + (size_t)node * H, kk, g);
      }
    } else {
      gin_pre.load(rh_saved, rh_h, node, g);
    }
  }
  if constexpr (TG > 1) {
    f32x4* red = reinterpret_cast<f32x4*>(&vt[0][0]);
    __syncthreads();   // every wave is done reading the staged blocks
    if constexpr (SPLIT) {
      // Each group hands the other group's tile over through LDS (static
      // register indices: the tile is picked by a uniform branch).
#pragma unroll
      for (int n = 0; n < NTW; ++n) {
        if (n == tg) continue;
#pragma unroll
        for (int m = 0; m < MT; ++m) red[(((tg * WAVES + wave) * MT) + m) * kWave + lane] = acc[n][m];
      }
      __syncthreads();
#pragma unroll
      for (int n = 0; n < NTW; ++n) {
        if (n != tg) continue;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const f32x4 r = red[((((1 - tg) * WAVES + wave) * MT) + m) * kWave + lane];
          // a = (group 0 partial) + (group 1 partial), in that order
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[n][m][j] = n == 0 ? acc[n][m][j] + r[j] : r[j] + acc[n][m][j];
        }
      }
    } else {
      // Groups 1.. leave their sums in LDS; group 0 adds them in group order.
      if (tg > 0) {
#pragma unroll
        for (int n = 0; n < NTW; ++n)
#pragma unroll
          for (int m = 0; m < MT; ++m) red[((((tg - 1) * WAVES + wave) * NTW + n) * MT + m) * kWave + lane] = acc[n][m];
      }
      __syncthreads();
      if (tg > 0) return;
#pragma unroll
      for (int gi = 1; gi < TG; ++gi)
#pragma unroll
        for (int n = 0; n < NTW; ++n)
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const f32x4 r = red[((((gi - 1) * WAVES + wave) * NTW + n) * MT + m) * kWave + lane];
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[n][m][j] += r[j];
          }
    }
  }
#pragma unroll
  for (int n = 0; n < NTW; ++n) {
    if (SPLIT && n != tg) continue;
    const size_t row = (size_t)(k * B + rw + 16 * n + q) * H + 4 * g;
    f32x4 gg[MT];   // reverse: dX of this tile
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      f32x4 v = acc[n][m];
      if (REV && dX_in) {
        const f32x4 b = *reinterpret_cast<const f32x4*>(dX_in + row + 16 * m);
        v = f32x4{b[0] + v[0], b[1] + v[1], b[2] + v[2], b[3] + v[3]};
      }
      gg[m] = v;
      if (!REV || out) store4(out + row + 16 * m, v[0], v[1], v[2], v[3]);
    }
    if constexpr (GRU && REV) {
      auto wl = [&](int which, int row, int gate, int kk) __attribute__((always_inline)) {
        return load_fragi<S>(gw, gru_rev_idx<S, H>(which, row / 16, gate, kk), lane);
      };
      if constexpr (!SPLIT) gin_pre.load(rh_saved, rh_h, k * B + rw + 16 * n + q, g);
      gru_bwd_wave<S, H>(gg, k * B + rw + 16 * n, q, g, gin_pre, wl, rh_da, n_pad, rh_dh, rh_ghat);
    }
    if constexpr (GRU && !REV) {
      // GRU of Eq. 1 (Cho et al. 2014 form) for this tile's 16 nodes, as in
      // the stand-alone GRU kernel: D[feature][node] with A = Wi^T / U^T
      // fragments (LDS) and B = a (hi + lo), h, r*h fragments.
      constexpr int KS = H / 32;
      const int node = k * B + rw + 16 * n + q;
      frag_t<S> af[NP][KS], hf[KS], rh[KS];
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        float v8[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v8[j] = acc[n][2 * kk][j];
          v8[4 + j] = acc[n][2 * kk + 1][j];
        }
        if constexpr (NP == 2) {
          split8(v8, af[0][kk], af[NP - 1][kk]);
        } else {
          af[0][kk] = pack8<S>(v8);
        }
        if constexpr (HRAW) {
          const u32x4 raw =
              SPLIT ? hraw_pre[kk] : *reinterpret_cast<const u32x4*>(X + (size_t)node * H + 32 * kk + 8 * g);
          u32x2 t[2];
          split_tiles16(raw, t);
          hf[kk] = __builtin_bit_cast(frag_t<S>, u32x4{t[0][0], t[0][1], t[1][0], t[1][1]});
        } else if constexpr (SPLIT) {
          hf[kk] = hf_pre[kk];
        } else {
          hf[kk] = rowfrag<S>(X + (size_t)node * H, kk, g);
        }
      }
      // Weight fragments of gate columns 16*t16 .. 16*t16 + 15 (fragment order).
      auto gfrag = [&](int mat, int t16, int kk) __attribute__((always_inline)) {
        return load_fragi<S>(gw, gru_fwd_idx<S, H>(mat, t16, kk), lane);
      };
      constexpr int NC = H / 16;   // 16-feature tiles of one gate
      // r for all features (r*h is an operand of the candidate product); the
      // k loops are outermost, so the NC accumulators are independent chains.
      f32x4 ar[NC];
#pragma unroll
      for (int c = 0; c < NC; ++c) ar[c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const frag_t<S> w0 = gfrag(0, c, kk);
#pragma unroll
          for (int part = 0; part < NP; ++part) mma(ar[c], w0, af[part][kk]);
          mma(ar[c], gfrag(1, c, kk), hf[kk]);
        }
#pragma unroll
      for (int c2 = 0; c2 < KS; ++c2) {
        float rhv[8], rv[8];
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const int f = 32 * c2 + 16 * p + 4 * g;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            rv[4 * p + j] = sigmoidf_(ar[2 * c2 + p][j] + bg[f + j]);
            rhv[4 * p + j] = rv[4 * p + j] * static_cast<float>(hf[c2][4 * p + j]);
          }
          if constexpr (!HRAW)
            store4(saved + (size_t)node * 3 * H + f, rv[4 * p], rv[4 * p + 1], rv[4 * p + 2], rv[4 * p + 3]);
        }
        if constexpr (HRAW) {   // r of the two tiles as one 16-byte store per lane
          const u32x4 pr = __builtin_bit_cast(u32x4, pack8<S>(rv));
          store_tiles16(saved + (size_t)node * 3 * H + 32 * c2, u32x2{pr[0], pr[1]}, u32x2{pr[2], pr[3]}, g);
        }
        rh[c2] = pack8<S>(rhv);
      }
      // z, n and the new state (2 NC independent chains).
      f32x4 az[NC], an[NC];
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        az[c] = f32x4{0.f, 0.f, 0.f, 0.f};
        an[c] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const frag_t<S> wz = gfrag(0, NC + c, kk), wn = gfrag(0, 2 * NC + c, kk);
#pragma unroll
          for (int part = 0; part < NP; ++part) {
            mma(az[c], wz, af[part][kk]);
            mma(an[c], wn, af[part][kk]);
          }
          mma(az[c], gfrag(1, NC + c, kk), hf[kk]);
          mma(an[c], gfrag(1, 2 * NC + c, kk), rh[kk]);
        }
      float zk[8], nk[8], ok[8];   // tiles c - 1, c (c odd) for the paired stores
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int f = 16 * c + 4 * g;
        float z[4], nn[4], o[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          z[j] = sigmoidf_(az[c][j] + bg[H + f + j]);
          nn[j] = tanhf_(an[c][j] + bg[2 * H + f + j]);
          const float hv = static_cast<float>(hf[c / 2][4 * (c % 2) + j]);
          o[j] = z[j] * hv + (1.f - z[j]) * nn[j];
          zk[4 * (c % 2) + j] = z[j];
          nk[4 * (c % 2) + j] = nn[j];
          ok[4 * (c % 2) + j] = o[j];
        }
        if constexpr (HRAW) {
          if (c % 2 == 1) {   // h', z, n of tiles c - 1, c as 16-byte stores
            const u32x4 po = __builtin_bit_cast(u32x4, pack8<S>(ok)), pz = __builtin_bit_cast(u32x4, pack8<S>(zk)),
                        pn = __builtin_bit_cast(u32x4, pack8<S>(nk));
            store_tiles16(h_out + (size_t)node * H + 32 * (c / 2), u32x2{po[0], po[1]}, u32x2{po[2], po[3]}, g);
            store_tiles16(saved + (size_t)node * 3 * H + H + 32 * (c / 2), u32x2{pz[0], pz[1]}, u32x2{pz[2], pz[3]},
                          g);
            store_tiles16(saved + (size_t)node * 3 * H + 2 * H + 32 * (c / 2), u32x2{pn[0], pn[1]},
                          u32x2{pn[2], pn[3]}, g);
          }
        } else {
          store4(h_out + (size_t)node * H + f, o[0], o[1], o[2], o[3]);
          store4(saved + (size_t)node * 3 * H + H + f, z[0], z[1], z[2], z[3]);
          store4(saved + (size_t)node * 3 * H + 2 * H + f, nn[0], nn[1], nn[2], nn[3]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Reverse: dM[e][h][j*B + c] = sum_s sum_r bits_t[e][j][s][c][r] da[h][(j-1+s)*B + r],
// dM rows of length ldm >= n_pad.
// Workgroup: RPW*WAVES columns c of block j; wave w: RPW of them.  D[c][h]:
// A operand = transposed bit rows c expanded in registers, B operand = staged
// da rows (feature-major, plain copies).  Lanes hold four consecutive nodes
// of one feature: 8-byte (bf16) stores into feature-major dM.
// ---------------------------------------------------------------------------
template <typename S, int H, int B, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void bits_bwd_kernel(const uint8_t* __restrict__ bits_t,
                                                                  const S* __restrict__ da, S* __restrict__ dM,
                                                                  int n_pad, int E, int groups, long ldm) {
  using C = BitsCfg<S, H, B>;
  constexpr int NT = WAVES * kWave;
  constexpr int V = C::V, KC = C::KC, VP = C::VP, RB = C::RB, NTW = C::NTW;
  constexpr int NTL = H / 16;
  constexpr int ROWB = B / 8;
  __shared__ __attribute__((aligned(16))) S vt[C::NBUF][H * VP];

  const int nb = n_pad / B;
  constexpr int NW = C::RPW * WAVES;
  const int tiles_per_blk = B / NW;
  // Logical id = (tile, type group), the group fastest: the groups of one
  // tile share the staged da blocks through one XCD's L2.
  const int t0 = xcd_swizzle(blockIdx.x, gridDim.x);
  const int grp = t0 % groups, t = t0 / groups;
  const int e_lo = grp * E / groups, e_hi = (grp + 1) * E / groups;
  const int j = t / tiles_per_blk;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = lane % 16, g = lane / 16;
  const int cw = (t % tiles_per_blk) * NW + C::RPW * wave;
  const int s_lo = (j == 0) ? 1 : 0;
  const int s_hi = (j == nb - 1) ? 1 : 2;

  if constexpr (C::ALL) {
    // The three da blocks, plain 16-byte copies; each thread issues up to
    // four loads before its LDS writes.
    constexpr int UPB = H * (KC / V);            // units per block
    constexpr int PB = 4;
    const int total = (s_hi - s_lo + 1) * UPB;
    for (int base = 0; base < total; base += PB * NT) {
      u32x4 r[PB];
#pragma unroll
      for (int u = 0; u < PB; ++u) {
        const int lin = base + u * NT + tid;
        if (lin < total) {
          const int slot = s_lo + lin / UPB, rem = lin % UPB;
          const int h = rem / (KC / V), c = (rem % (KC / V)) * V;
          r[u] = *reinterpret_cast<const u32x4*>(da + (size_t)h * n_pad + (j - 1 + slot) * B + c);
        }
      }
#pragma unroll
      for (int u = 0; u < PB; ++u) {
        const int lin = base + u * NT + tid;
        if (lin < total) {
          const int slot = s_lo + lin / UPB, rem = lin % UPB;
          const int h = rem / (KC / V), c = (rem % (KC / V)) * V;
          *reinterpret_cast<u32x4*>(&vt[slot][frag_off<S, H, KC>(h, c)]) = r[u];
        }
      }
    }
    __syncthreads();
  }
  RowBytes<RB> nxt[3][NTW];
  auto load_type = [&](int e, RowBytes<RB> (&dst)[3][NTW]) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      if (s < s_lo || s > s_hi) continue;
      const uint8_t* brow = bits_t + ((((size_t)e * nb + j) * 3 + s) * B + cw + q) * ROWB + g * (KC / 32);
#pragma unroll
      for (int m = 0; m < NTW; ++m) dst[s][m].load(brow + (size_t)16 * m * ROWB);
    }
  };
  if constexpr (C::ALL) load_type(e_lo, nxt);
  for (int e = e_lo; e < e_hi; ++e) {
    f32x4 acc[NTW][NTL];
#pragma unroll
    for (int m = 0; m < NTW; ++m)
#pragma unroll
      for (int n = 0; n < NTL; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    RowBytes<RB> cur[3][NTW];
    if constexpr (C::ALL) {
#pragma unroll
      for (int s = 0; s < 3; ++s)
#pragma unroll
        for (int m = 0; m < NTW; ++m) cur[s][m] = nxt[s][m];
      if (e + 1 < e_hi) load_type(e + 1, nxt);
    }
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      if (s < s_lo || s > s_hi) continue;
      const uint8_t* brow = bits_t + ((((size_t)e * nb + j) * 3 + s) * B + cw + q) * ROWB;
      for (int c0 = 0; c0 < B; c0 += KC) {
        if constexpr (!C::ALL) {
          __syncthreads();
          stage_cols<S, H, KC, VP, NT, C::ROWS, false>(vt[0], da, n_pad, (j - 1 + s) * B + c0, tid);
          __syncthreads();
        }
        const S* v = vt[C::ALL ? s : 0];
        RowBytes<RB> rb[NTW];
#pragma unroll
        for (int m = 0; m < NTW; ++m) {
          if constexpr (C::ALL) {
            rb[m] = cur[s][m];
          } else {
            rb[m].load(brow + (size_t)16 * m * ROWB + (c0 + g * (KC / 4)) / 8);
          }
        }
#pragma unroll
        for (int kk = 0; kk < RB; ++kk) {
          frag_t<S> af[NTW];
#pragma unroll
          for (int m = 0; m < NTW; ++m) af[m] = bits_frag<S>(rb[m].byte(kk));
#pragma unroll
          for (int n = 0; n < NTL; ++n) {
            const frag_t<S> bf = C::ROWS ? load8(&v[(16 * n + q) * VP + g * (KC / 4) + 8 * kk])
                                         : load_frag<S, H>(v, kk, n, lane);
#pragma unroll
            for (int m = 0; m < NTW; ++m) mma(acc[m][n], af[m], bf);
          }
        }
      }
    }
    S* out = dM + (size_t)e * H * ldm + (size_t)j * B + cw + 4 * g;
#pragma unroll
    for (int m = 0; m < NTW; ++m)
#pragma unroll
      for (int n = 0; n < NTL; ++n)
        store4(out + (size_t)(16 * n + q) * ldm + 16 * m, acc[m][n][0], acc[m][n][1], acc[m][n][2], acc[m][n][3]);
  }
}

// W_e^T from W_e for every edge type: Wt[e][o][h] = W[e][h][o], 8 x 8 tiles
// transposed in registers (16-byte loads and stores).
template <typename S>
__global__ void transpose_weights_kernel(const S* __restrict__ W, S* __restrict__ Wt, int H, int E) {
  constexpr int V = 16 / sizeof(S);
  const int tiles = (H / V) * (H / V);
  const long lin = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (lin >= (long)E * tiles) return;
  const int e = (int)(lin / tiles), rem = (int)(lin % tiles);
  const int hq = rem / (H / V), oq = rem % (H / V);
  u32x4 r[V];
  tile_load<S>(r, W + (size_t)e * H * H + (size_t)(V * hq) * H + V * oq, H);
#pragma unroll
  for (int x = 0; x < V; ++x)
    *reinterpret_cast<u32x4*>(Wt + (size_t)e * H * H + (size_t)(V * oq + x) * H + V * hq) = tile_row_T<S>(r, x);
}

}  // namespace dev

// Workgroup size: the largest (up to four waves, never more rows than a block
// holds) that still gives at least this many workgroups.
#ifndef GGNN_BITS_FWD_MIN_BLOCKS
#define GGNN_BITS_FWD_MIN_BLOCKS 64
#endif
#ifndef GGNN_BITS_BWD_MIN_BLOCKS
#define GGNN_BITS_BWD_MIN_BLOCKS 64
#endif
#ifndef GGNN_BITS_TG2_MAX_BLOCKS
#define GGNN_BITS_TG2_MAX_BLOCKS 512
#endif
#ifndef GGNN_BITS_BWD_WAVES
#define GGNN_BITS_BWD_WAVES 4096
#endif

namespace {
// One launch of a bit-band kernel.  mode 0: fused forward step; 1: fused
// reverse step (dM node-major, dX); 2: reverse product only (dM feature-major).
struct BitsArgs {
  int mode;
  const void* bits;
  const void* V;        // X (forward) or da (reverse)
  const void* W;
  const float* bias;
  void* out;            // a, dX_out or dM
  const float* dX_in;
  void* dM;             // mode 1
  long ldm;
  int n_pad, E;
  const void* Wt = nullptr;   // mode 0: W_e^T [E][H][H] (optional; used by the direct-weight forms)
  const void* Wi = nullptr;   // mode 0 with the GRU epilogue (when non-NULL and supported)
  const void* U = nullptr;
  const float* bg = nullptr;
  void* h_out = nullptr;
  void* saved = nullptr;
  bool* fused_gru = nullptr;  // set to whether the GRU ran in the step
  // mode 1 with the previous step's GRU reverse (when rh_da != NULL and supported)
  const void* rh_h = nullptr;
  const void* rh_saved = nullptr;
  void* rh_da = nullptr;
  float* rh_dh = nullptr;
  void* rh_ghat = nullptr;
  const SnStep* sn = nullptr;   // fused supernode share (bf16 direct-weight forms with the GRU or the t = 0 reverse)
};

// Launch shape of a bit-band kernel (mode as in BitsArgs).
struct BitsPlan {
  int waves, groups, blocks;
  bool tg2;
};
template <typename S, int H, int B>
BitsPlan bits_plan(int mode, int n_pad, int E) {
  using C = dev::BitsCfg<S, H, B>;
  const int nb = n_pad / B;
  const bool fused = mode != 2;
  int waves = B / C::RPW < 4 ? B / C::RPW : 4;
  // Streamed blocks at H = 256, forward: eight waves (128 rows) share each
  // staged chunk, halving the staging per row (the reverse step's
  // eight-wave form would spill registers).
  if constexpr (!C::ALL && H >= 256) {
    if (mode == 0) waves = B / C::RPW < 8 ? B / C::RPW : 8;
  }
  const long min_blocks = fused ? GGNN_BITS_FWD_MIN_BLOCKS : GGNN_BITS_BWD_MIN_BLOCKS;
  while (waves > C::MINW && (long)nb * (B / (C::RPW * waves)) < min_blocks) waves /= 2;
  const int tiles = nb * (B / (C::RPW * waves));
  // The plain reverse product writes one output per edge type, so types can
  // be split over workgroups freely: enough groups for about
  // GGNN_BITS_BWD_WAVES waves.
  int groups = 1;
  if (!fused) {
    const long want = (GGNN_BITS_BWD_WAVES + (long)tiles * waves - 1) / ((long)tiles * waves);
    groups = (int)(want < 1 ? 1 : (want > E ? E : want));
  }
  const int blocks = tiles * groups;
  // Fused steps: two type groups per workgroup (two waves per SIMD) when the
  // grid alone does not give every SIMD several waves.
  return BitsPlan{waves, groups, blocks, C::WDIR && blocks <= GGNN_BITS_TG2_MAX_BLOCKS};
}

template <typename S, int H, int B>
hipError_t bits_launch(const BitsArgs& A, hipStream_t st) {
  using C = dev::BitsCfg<S, H, B>;
  const BitsPlan plan = bits_plan<S, H, B>(A.mode, A.n_pad, A.E);
  const int waves = plan.waves, groups = plan.groups, blocks = plan.blocks;
  const bool tg2 = plan.tg2;
  const uint8_t* bp = static_cast<const uint8_t*>(A.bits);
  const S* vp = static_cast<const S*>(A.V);
  const S* wp = static_cast<const S*>(A.W);
  float* op = static_cast<float*>(A.out);
  S* dmp = static_cast<S*>(A.dM);
  // The GRU epilogue rides along only in the two-group form (a small grid,
  // where the separate GRU launch would cost most).
  const bool gru = A.mode == 0 && A.Wi != nullptr && C::WDIR && tg2;
  const bool rgru = A.mode == 1 && A.rh_da != nullptr && C::WDIR && tg2;
  if (A.fused_gru) *A.fused_gru = gru || rgru;
  if (rgru) op = nullptr;   // dX goes straight into the GRU reverse
  // Supernodes ride along only in the two-group direct-weight forms: the
  // forward with its GRU, the reverse with or without it.
  const bool sn = A.sn != nullptr;
  if (sn && !(sizeof(S) == 2 && C::WDIR && C::RPW == dev::kSnFused && tg2 && (A.mode == 1 || gru)))
    return hipErrorNotSupported;
  const uint8_t* snb = sn ? static_cast<const uint8_t*>(A.sn->bits) : nullptr;
  const float* snrec = sn ? A.sn->rec : nullptr;
  const int sns = sn ? A.sn->s : 0, snr = sn ? A.sn->sr : 0;
#define GGNN_STEP_SN(WV, TGN, REVB, GRUB, SNB)                                                                \
  hipLaunchKernelGGL((dev::step_bits_kernel<S, H, B, WV, C::WDIR, TGN, REVB, GRUB, SNB>), dim3(blocks),       \
                     dim3(TGN * WV * 64), 0, st, bp, vp, wp, static_cast<const S*>(A.Wt), A.bias, op, A.n_pad,  \
                     A.E, A.dX_in, dmp, A.ldm,                                                                  \
                     static_cast<const S*>(A.Wi), static_cast<const S*>(A.U), A.bg, static_cast<S*>(A.h_out),  \
                     static_cast<S*>(A.saved), static_cast<const S*>(A.rh_h), static_cast<const S*>(A.rh_saved), \
                     static_cast<S*>(A.rh_da), A.rh_dh, static_cast<S*>(A.rh_ghat), snb, snrec, sns, snr)
#define GGNN_STEP(WV, TGN, REVB, GRUB)                                                                        \
  do {                                                                                                        \
    if constexpr (sizeof(S) == 2 && C::WDIR && C::RPW == dev::kSnFused && TGN == 2 && (REVB || GRUB)) {       \
      if (sn) {                                                                                               \
        GGNN_STEP_SN(WV, TGN, REVB, GRUB, true);                                                              \
        break;                                                                                                \
      }                                                                                                       \
    }                                                                                                         \
    GGNN_STEP_SN(WV, TGN, REVB, GRUB, false);                                                                 \
  } while (0)
#define GGNN_BITS_CASE(WV)                                                                                   \
  case WV:                                                                                                   \
    if constexpr (B / C::RPW >= WV && WV >= C::MINW && (WV <= 4 || (!C::ALL && H >= 256))) {         \
      if (A.mode == 0 && gru)                                                                                \
        GGNN_STEP(WV, (C::WDIR ? 2 : 1), false, C::WDIR);                                                    \
      else if (A.mode == 0 && tg2)                                                                           \
        GGNN_STEP(WV, (C::WDIR ? 2 : 1), false, false);                                                      \
      else if (A.mode == 0)                                                                                  \
        GGNN_STEP(WV, 1, false, false);                                                                      \
      else {                                                                                                 \
        if constexpr (WV <= 4) { /* eight-wave forms: forward only */                                       \
          if (A.mode == 1 && rgru)                                                                           \
            GGNN_STEP(WV, (C::WDIR ? 2 : 1), true, C::WDIR);                                                 \
          else if (A.mode == 1 && tg2)                                                                       \
            GGNN_STEP(WV, (C::WDIR ? 2 : 1), true, false);                                                   \
          else if (A.mode == 1)                                                                              \
            GGNN_STEP(WV, 1, true, false);                                                                   \
          else                                                                                               \
            hipLaunchKernelGGL((dev::bits_bwd_kernel<S, H, B, WV>), dim3(blocks), dim3(WV * 64), 0, st, bp,  \
                               vp, static_cast<S*>(A.out), A.n_pad, A.E, groups, A.ldm);                     \
        }                                                                                                    \
      }                                                                                                      \
    }                                                                                                        \
    break;
  switch (waves) {
    GGNN_BITS_CASE(8)
    GGNN_BITS_CASE(4)
    GGNN_BITS_CASE(2)
    GGNN_BITS_CASE(1)
  }
#undef GGNN_BITS_CASE
#undef GGNN_STEP
#undef GGNN_STEP_SN
  return hipGetLastError();
}

template <typename S, int H>
hipError_t bits_h(int B, const BitsArgs& A, hipStream_t st) {
  switch (B) {
    case 32: return bits_launch<S, H, 32>(A, st);
    case 64: return bits_launch<S, H, 64>(A, st);
    case 128: return bits_launch<S, H, 128>(A, st);
    case 256: return bits_launch<S, H, 256>(A, st);
    case 512: return bits_launch<S, H, 512>(A, st);
  }
  return hipErrorInvalidValue;
}

template <typename S>
hipError_t bits_t(int H, int B, const BitsArgs& A, hipStream_t st) {
  switch (H) {
    case 32: return bits_h<S, 32>(B, A, st);
    case 64: return bits_h<S, 64>(B, A, st);
    case 128: return bits_h<S, 128>(B, A, st);
    case 256: return bits_h<S, 256>(B, A, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace

namespace GGNN_IMPL_NS {
hipError_t launch_step_fwd_bits(int n_pad, int B, int H, int E, const void* bits, const void* X, const void* W,
                                const float* bias, float* a, hipStream_t st) {
  return bits_t<dev::dt_t>(H, B, BitsArgs{0, bits, X, W, bias, a, nullptr, nullptr, 0, n_pad, E}, st);
}

hipError_t launch_step_fwd_bits_gru(int n_pad, int B, int H, int E, const void* bits, const void* X, const void* W,
                                    const void* Wt, const float* bias, float* a, const void* Wi, const void* U,
                                    const float* bg, void* h_out, void* saved, bool* fused, hipStream_t st) {
  BitsArgs A{0, bits, X, W, bias, a, nullptr, nullptr, 0, n_pad, E};
  A.Wt = Wt;
  A.Wi = Wi;
  A.U = U;
  A.bg = bg;
  A.h_out = h_out;
  A.saved = saved;
  A.fused_gru = fused;
  return bits_t<dev::dt_t>(H, B, A, st);
}

hipError_t launch_transpose_weights(int H, int E, const void* W, void* Wt, hipStream_t st) {
  using S = dev::dt_t;
  constexpr int V = 16 / sizeof(S);
  const long n = (long)E * (H / V) * (H / V);
  hipLaunchKernelGGL((dev::transpose_weights_kernel<S>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                     static_cast<const S*>(W), static_cast<S*>(Wt), H, E);
  return hipGetLastError();
}

hipError_t launch_step_bwd_bits(int n_pad, int B, int H, int E, const void* bits_t_, const void* da, const void* W,
                                const float* dX_in, float* dX_out, void* dM, long ldm, hipStream_t st) {
  return bits_t<dev::dt_t>(H, B, BitsArgs{1, bits_t_, da, W, nullptr, dX_out, dX_in, dM, ldm, n_pad, E}, st);
}

hipError_t launch_step_bwd_bits_gru(int n_pad, int B, int H, int E, const void* bits_t_, const void* da,
                                    const void* W, const float* dX_in, float* dX_out, void* dM, long ldm,
                                    const void* Wi, const void* U, const void* h_prev, const void* saved_prev,
                                    void* da_prev, float* dh_prev, void* ghat_prev, bool* fused, hipStream_t st) {
  BitsArgs A{1, bits_t_, da, W, nullptr, dX_out, dX_in, dM, ldm, n_pad, E};
  A.Wi = Wi;
  A.U = U;
  A.rh_h = h_prev;
  A.rh_saved = saved_prev;
  A.rh_da = da_prev;
  A.rh_dh = dh_prev;
  A.rh_ghat = ghat_prev;
  A.fused_gru = fused;
  return bits_t<dev::dt_t>(H, B, A, st);
}

hipError_t launch_banded_bwd_bits(int n_pad, int B, int H, int E, const void* bits_t_, const void* da, void* dM,
                                  long ldm, hipStream_t st) {
  return bits_t<dev::dt_t>(H, B, BitsArgs{2, bits_t_, da, nullptr, nullptr, dM, nullptr, nullptr, ldm, n_pad, E},
                           st);
}

#if GGNN_DT_BF16
namespace {
template <int H, int B>
bool sn_fusable_hb(int n_pad, int E) {
  using C = dev::BitsCfg<dev::bf16s, H, B>;
  if constexpr (!C::WDIR || C::RPW != dev::kSnFused) {
    return false;
  } else {
    return bits_plan<dev::bf16s, H, B>(0, n_pad, E).tg2 && bits_plan<dev::bf16s, H, B>(1, n_pad, E).tg2;
  }
}
template <int H>
bool sn_fusable_h(int B, int n_pad, int E) {
  switch (B) {
    case 32: return sn_fusable_hb<H, 32>(n_pad, E);
    case 64: return sn_fusable_hb<H, 64>(n_pad, E);
    case 128: return sn_fusable_hb<H, 128>(n_pad, E);
    case 256: return sn_fusable_hb<H, 256>(n_pad, E);
    case 512: return sn_fusable_hb<H, 512>(n_pad, E);
  }
  return false;
}
}  // namespace

bool step_sn_fusable(int n_pad, int B, int H, int E) {
  switch (H) {
    case 32: return sn_fusable_h<32>(B, n_pad, E);
    case 64: return sn_fusable_h<64>(B, n_pad, E);
  }
  return false;
}

hipError_t launch_step_fwd_bits_gru_sn(int n_pad, int B, int H, int E, const void* bits, const void* X, const void* W,
                                       const void* Wt, const float* bias, float* a, const void* Wi, const void* U,
                                       const float* bg, void* h_out, void* saved, const SnStep& sn, hipStream_t st) {
  BitsArgs A{0, bits, X, W, bias, a, nullptr, nullptr, 0, n_pad, E};
  A.Wt = Wt;
  A.Wi = Wi;
  A.U = U;
  A.bg = bg;
  A.h_out = h_out;
  A.saved = saved;
  A.sn = &sn;
  return bits_t<dev::bf16s>(H, B, A, st);
}

hipError_t launch_step_bwd_bits_sn(int n_pad, int B, int H, int E, const void* bits_t_, const void* da,
                                   const void* W, const float* dX_in, float* dX_out, void* dM, long ldm,
                                   const void* Wi, const void* U, const void* h_prev, const void* saved_prev,
                                   void* da_prev, float* dh_prev, void* ghat_prev, const SnStep& sn, hipStream_t st) {
  BitsArgs A{1, bits_t_, da, W, nullptr, dX_out, dX_in, dM, ldm, n_pad, E};
  A.Wi = Wi;
  A.U = U;
  A.rh_h = h_prev;
  A.rh_saved = saved_prev;
  A.rh_da = da_prev;
  A.rh_dh = dh_prev;
  A.rh_ghat = ghat_prev;
  A.sn = &sn;
  return bits_t<dev::bf16s>(H, B, A, st);
}
#endif
}  // namespace GGNN_IMPL_NS

}  // namespace ggnn
