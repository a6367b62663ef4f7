// Weight gradient of the message transform at H = 256 (bf16), the largest
// single contraction of the reverse pass: over all T * n_pad rows k,
//   P[split][e][h_in][h_out] = sum_k X[k][h_in] dM[e][k][h_out],
//   Pb[split][e][h_out]      = sum_k dM[e][k][h_out]
// (partials per row split, summed later in a fixed order), with dM stored
// node-major by the reverse step kernels (row k of type e at (e ldk + k) H).
//
// It streams 47 GB at the 1M-node workload: what bounds it is how many bytes
// each compute unit keeps in flight.  Loads that pass through registers are
// limited by the registers left next to the accumulators (one chunk at a
// time); here the rows go from global memory straight to LDS
// (global_load_lds_dwordx4: each lane's 16 bytes land at the wave's LDS base
// + 16 lane), three chunks ahead of the one being multiplied, in a ring of
// four LDS slots.  The loads are issued from inline assembly, so that the
// compiler does not wait for all of them before every LDS read; the kernel
// waits for exactly the chunk it needs (s_waitcnt vmcnt counts these loads in
// issue order) and then meets the other waves at a barrier.
//
// Workgroup: 8 waves, one row split, one edge type, all 256 input features
// (dM, the large operand, read once).  Wave (wi, wo) of a 2 x 4 grid owns
// input tiles 8 wi .. 8 wi + 7 and output tiles 4 wo .. 4 wo + 3.  A chunk
// is 32 rows of X and of dM_e, node-major, unpadded; the 16-element groups of
// chunk row r are XOR-permuted by sw(r) = (r & 3) | ((r >> 3) & 1) << 2 (the
// permutation is applied to each lane's source address, the LDS writes being
// contiguous), so that the rows of one transposing read fall on disjoint
// banks.  Splits are multiples of 128 rows and K = T n_pad a multiple of 32,
// so every chunk is whole.
#include "device_common.h"
#include "kernels.h"
#include "lds_dma.h"

namespace ggnn {
namespace dev {
namespace wgw {

constexpr int H = 256, KC = 32, WI = 2, WO = 4, NWV = WI * WO, NT = 64 * NWV;
constexpr int TI = 16 / WI, TO = 16 / WO;   // input / output tiles per wave
constexpr int SLOT = 2 * KC * H;            // elements of one slot: X rows, then dM rows
constexpr int NSLOT = 4;
constexpr int IPW = KC * H * 2 / 1024 / NWV;   // 1 KB loads per wave per operand and chunk (2)

__device__ __forceinline__ int sw(int r) { return (r & 3) | (((r >> 3) & 1) << 2); }

// Fragment of a swizzled k-major [KC][256] tile: lane (q, g) receives
// elements (k0 + 8g + j, n0 + q), j = 0..7 (n0 a multiple of 16); two
// transposing reads, four rows apart (rows r and r + 4 share the swizzle).
__device__ __forceinline__ bf16x8 frag(const bf16s* base, int k0, int n0, int lane) {
  const int p = lane % 16, g = lane / 16;
  const int row = k0 + 8 * g + p / 4;
  const bf16s* a0 = base + row * H + ((n0 ^ (sw(row) << 4)) + 4 * (p % 4));
  const tr_v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_tr_v4i16*)(const_cast<bf16s*>(a0)));
  const tr_v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_tr_v4i16*)(const_cast<bf16s*>(a0) + 4 * H));
  typedef short v8i16 __attribute__((ext_vector_type(8)));
  const v8i16 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

__global__ __launch_bounds__(NT) void transform_wgrad_nm256_kernel(const bf16s* __restrict__ X,
                                                                   const bf16s* __restrict__ dM, long ldk,
                                                                   float* __restrict__ P, float* __restrict__ Pb,
                                                                   long K, int E, int rows_per_split) {
  __shared__ __attribute__((aligned(1024))) bf16s ring[NSLOT * SLOT];

  const int tid = threadIdx.x, lane = tid % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int q = lane % 16, g = lane / 16;
  const int wi = wave % WI, wo = wave / WI;
  const int bid = xcd_swizzle(blockIdx.x, gridDim.x);
  const int e = bid % E;
  const int split = bid / E;
  const long nlo = (long)split * rows_per_split;
  const long nhi = min(K, nlo + rows_per_split);
  const int nchunks = nlo < nhi ? (int)((nhi - nlo) / KC) : 0;
  const bf16s* dMe = dM + (size_t)e * ldk * H;
  const uint32_t ring_lds = (uint32_t)(uintptr_t)ring;

  // This lane's part of a chunk: copy j of the wave covers chunk rows
  // r = 2 (IPW wave + j) + lane / 32, 16-byte unit lane % 32 of the row, whose
  // source is the unit of column (8 (lane % 32)) ^ (16 sw(r)).
  int src_off[IPW];   // element offset within the chunk's first row
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int r = 2 * (IPW * wave + j) + lane / 32;
    src_off[j] = r * H + ((8 * (lane % 32)) ^ (sw(r) << 4));
  }
  auto issue = [&](int chunk, int slot) __attribute__((always_inline)) {
    const size_t row0 = (size_t)(nlo + (long)chunk * KC) * H;
    const uint32_t base = ring_lds + (uint32_t)(slot * SLOT) * 2u;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const uint32_t at = base + (uint32_t)(2 * (IPW * wave + j)) * H * 2u;
      dma16(X + row0 + src_off[j], at);
      dma16(dMe + row0 + src_off[j], at + (uint32_t)KC * H * 2u);
    }
  };

  f32x4 acc[TI][TO];
  float bsum[TO];
#pragma unroll
  for (int o = 0; o < TO; ++o) {
    bsum[o] = 0.f;
#pragma unroll
    for (int i = 0; i < TI; ++i) acc[i][o] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  auto compute = [&](int slot) __attribute__((always_inline)) {
    const bf16s* sx = ring + slot * SLOT;
    const bf16s* sd = sx + KC * H;
#pragma unroll
    for (int k0 = 0; k0 < KC; k0 += 32) {
      bf16x8 fb[TO];
#pragma unroll
      for (int o = 0; o < TO; ++o) {
        fb[o] = frag(sd, k0, 16 * (wo * TO + o), lane);
        if (wi == 0) {
#pragma unroll
          for (int x = 0; x < 8; ++x) bsum[o] += static_cast<float>(fb[o][x]);
        }
      }
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        const bf16x8 fa = frag(sx, k0, 16 * (wi * TI + i), lane);
#pragma unroll
        for (int o = 0; o < TO; ++o) mma(acc[i][o], fa, fb[o]);
      }
    }
  };
  // Chunk c in slot c % 4; before multiplying it, wait for this wave's copies
  // of it (the chunks after it that were issued may stay in flight), meet the
  // other waves, and issue chunk c + 3 into the slot chunk c - 1 used (every
  // wave is past its products).
  constexpr int PER = 2 * IPW;   // copies per wave and chunk
  auto stage = [&](int c, int slot) __attribute__((always_inline)) {
    const int later = nchunks - 1 - c;   // chunks after c already issued (at most 2)
    if (later >= 2) wait_copies<2 * PER>();
    else if (later == 1) wait_copies<PER>();
    else wait_copies<0>();
    __syncthreads();
    if (c + 3 < nchunks) issue(c + 3, (slot + 3) % NSLOT);
    compute(slot);
  };
#pragma unroll
  for (int c = 0; c < 3; ++c)
    if (c < nchunks) issue(c, c);
  for (int c = 0; c < nchunks; c += NSLOT) {
    stage(c, 0);
    if (c + 1 >= nchunks) break;
    stage(c + 1, 1);
    if (c + 2 >= nchunks) break;
    stage(c + 2, 2);
    if (c + 3 >= nchunks) break;
    stage(c + 3, 3);
  }

  // D[h_in = 16 (wi TI + i) + 4g + j][h_out = 16 (wo TO + o) + q]
  float* out = P + ((size_t)split * E + e) * H * H;
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int o = 0; o < TO; ++o)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        out[(size_t)(16 * (wi * TI + i) + 4 * g + j) * H + 16 * (wo * TO + o) + q] = acc[i][o][j];
  if (Pb != nullptr && wi == 0) {
#pragma unroll
    for (int o = 0; o < TO; ++o) {
      float v = bsum[o];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g == 0) Pb[((size_t)split * E + e) * H + 16 * (wo * TO + o) + q] = v;
    }
  }
}

}  // namespace wgw

// ---------------------------------------------------------------------------
// Weight gradients of the GRU at H = 256 (bf16) over all T * n_pad rows k
// (a, h, saved and G^ stacked over t):
//   P[split][0][i][c] = sum_k a[k][i] G^[k][c]          (dWi)
//   P[split][1][i][c] = sum_k x_c[k][i] G^[k][c]        (dU)
//   Pb[split][c]      = sum_k G^[k][c]                  (db)
// with x_c = h for the first 2H gate columns and r*h for the last H (r the
// first H values of the saved gates); a enters rounded to bf16 and r*h is
// formed in fp32 and rounded to bf16, as at the other widths.
//
// The contraction streams 3.6 KB per row (a in fp32, h, r, G^) over 8.4 M
// rows at the 1M-node workload.  Loads staged through registers leave one
// chunk in flight per workgroup, which then waits on memory at every chunk;
// here each workgroup owns one row split and one of the six 256 x 256 output
// tiles (matrix m in {dWi, dU} x gate block gb), reads G^'s 256-column block
// and one input operand (a, h, or h and r), and copies the rows from global
// memory straight to LDS (global_load_lds_dwordx4) two 32-row chunks ahead of
// the one being multiplied, in a ring of three 48 KB slots.  The six tiles of
// a split are neighbouring workgroups (one XCD, shared L2).  (Pairing both
// matrices of one input half and gate block in a workgroup instead, so that
// the workgroups sharing a G^ block do equal work, fetched more: over a
// split's thousands of chunks independent workgroups drift apart whatever
// their balance, and the L2 serves few of the shared rows either way.)
//
// Slot layouts (32 rows each): dWi: a as fp32 [32][256] (32 KB) then the G^
// block [32][256] bf16; dU on the r and z blocks: h, G^ block; dU on the n
// block: h, r (then r * h), G^ block.  bf16 tiles are XOR-permuted by sw(r) as above; in
// the fp32 tile, the 4-column units of row r are XOR-permuted by
// 16 ((r >> 3) & 3), so that the four 8-row groups of one strided fragment
// read fall on disjoint banks.  Waves form a 2 x 4 grid as above.
// ---------------------------------------------------------------------------
namespace gwg {

// XCD of logical workgroup lb (the inverse of xcd_swizzle's grouping).
__device__ __forceinline__ int xcd_of(int lb, int nblocks) {
  const int per = nblocks / 8, rem = nblocks % 8;
  return lb < rem * (per + 1) ? lb / (per + 1) : rem + (lb - rem * (per + 1)) / per;
}

// Pacing of the workgroups of one row split (up to 8; wave 0 of each,
// before the stage's barrier).  The output tiles of a split read shared rows
// of their operands but do unequal work per chunk; left alone they drift
// apart by many chunks over a split and each fetches the shared rows from
// memory itself (49 GB per launch at the 1M-node workload, against 29.5 GB
// of operands).  Each publishes the chunk it has reached in counters[tile]
// (a vector store); every PACE_EVERY chunks it reads the split's 8 counters
// (one scalar load that bypasses the scalar cache, so that these waits do
// not mix with the copies' vmcnt) and, while a sibling on its XCD (bit t of
// sibs) is more than PACE_SLACK chunks behind, sleeps and reads again
// (32.6 GB fetched, 11.5 -> 10.2 ms; the poll interval and slack made no
// difference between 1 and 8 chunks).  Only the timing depends on this:
// every workgroup reads its own operands and writes its own partials.
// After PACE_TRIES reads without the laggard catching up, pacing stops for
// the rest of the launch (a sibling that is not resident, or counters left
// by an earlier launch, cost one bounded wait).
#ifndef GGNN_PACE_EVERY
#define GGNN_PACE_EVERY 4
#endif
#ifndef GGNN_PACE_SLACK
#define GGNN_PACE_SLACK 3
#endif
constexpr int PACE_EVERY = GGNN_PACE_EVERY, PACE_SLACK = GGNN_PACE_SLACK, PACE_TRIES = 64;
typedef int i32x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ bool pace_split(int* counters, int tile, uint32_t sibs, int c, int lane, bool on) {
  if (lane == 0) __hip_atomic_store(counters + tile, c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (!on || c % PACE_EVERY != 0 || c < PACE_SLACK) return on;
  for (int tries = 0; tries < PACE_TRIES; ++tries) {
    i32x8 v;
    asm volatile("s_load_dwordx8 %0, %1, 0x0 glc\n\ts_waitcnt lgkmcnt(0)" : "=s"(v) : "s"(counters) : "memory");
    int lag = 0x7fffffff;
#pragma unroll
    for (int t = 0; t < 8; ++t)
      if ((sibs >> t) & 1u) lag = min(lag, v[t]);
    if (lag >= c - PACE_SLACK) return true;
    __builtin_amdgcn_s_sleep(4);
  }
  return false;
}

// Siblings of tile `tile` among the ntile workgroups of split `split`
// (logical ids split * ntile + t) that run on the same XCD as logical
// workgroup bid.
__device__ __forceinline__ uint32_t pace_siblings(int bid, int split, int tile, int ntile, int nblocks) {
  uint32_t sibs = 0u;
  const int mine = xcd_of(bid, nblocks);
  for (int t = 0; t < ntile; ++t)
    if (t != tile && xcd_of(split * ntile + t, nblocks) == mine) sibs |= 1u << t;
  return sibs;
}


constexpr int H = 256, G3 = 3 * H, KC = 32, WI = 2, WO = 4, NWV = WI * WO, NT = 64 * NWV;
constexpr int TI = 16 / WI, TO = 16 / WO;
constexpr int TILE16 = KC * H * 2;          // bytes of a bf16 [32][256] tile
constexpr int SLOT = 3 * TILE16;            // bytes of one slot (48 KB)
constexpr int NSLOT = 3;
constexpr int NTILE = 6;                    // output tiles per split

// Fragment of the fp32 a tile, rounded to bf16: lane (q, g) receives
// a(8g + j, n0 + q), j = 0..7.
__device__ __forceinline__ bf16x8 frag_f32(const float* base, int n0, int lane) {
  const int q = lane % 16, g = lane / 16;
  float v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int row = 8 * g + j;
    v[j] = base[row * H + ((n0 ^ (((row >> 3) & 3) << 4)) + q)];
  }
  return pack8<bf16s>(v);
}

// KIND 0: dWi (operand a), 1: dU on the r or z block (h), 2: dU on the n
// block (r * h).
template <int KIND>
__device__ __forceinline__ void gru_wgrad256_body(const float* __restrict__ a, const bf16s* __restrict__ h,
                                                  const bf16s* __restrict__ saved, const bf16s* __restrict__ ghat,
                                                  float* __restrict__ P, float* __restrict__ Pb, long K,
                                                  int rows_per_split, int split, int m, int gb, int wave, int lane,
                                                  unsigned char* ring, int* __restrict__ prog, int tile,
                                                  uint32_t sibs) {
  const int q = lane % 16, g = lane / 16;
  const int wi = wave % WI, wo = wave / WI;
  const long nlo = (long)split * rows_per_split;
  const long nhi = min(K, nlo + rows_per_split);
  const int nchunks = nlo < nhi ? (int)((nhi - nlo) / KC) : 0;
  const uint32_t ring_lds = (uint32_t)(uintptr_t)ring;
  // byte offsets of the operand tiles within a slot
  constexpr int OFF_G = KIND == 1 ? TILE16 : 2 * TILE16;
  constexpr int OFF_R = TILE16;   // KIND 2 only
  constexpr int PER = KIND == 1 ? 4 : 6;   // copies per wave and chunk

  // This lane's element offsets relative to the chunk's first row.  bf16
  // tiles: copy j (0, 1) of the wave covers chunk rows r = 2 (2 wave + j) +
  // lane / 32, 8-element unit lane % 32 of the row.  fp32 a: copy j (0..3)
  // covers row 4 wave + j, 4-element unit lane.
  int off_h[2], off_g[2], off_a[4];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r = 2 * (2 * wave + j) + lane / 32;
    const int u = (8 * (lane % 32)) ^ (wgw::sw(r) << 4);
    off_h[j] = r * H + u;
    off_g[j] = r * G3 + gb * H + u;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = 4 * wave + j;
    off_a[j] = r * H + ((4 * lane) ^ (((r >> 3) & 3) << 4));
  }
  auto issue = [&](int chunk, int slot) __attribute__((always_inline)) {
    const size_t row0 = (size_t)(nlo + (long)chunk * KC);
    const uint32_t base = ring_lds + (uint32_t)(slot * SLOT);
    if constexpr (KIND == 0) {
      const float* ac = a + row0 * H;
#pragma unroll
      for (int j = 0; j < 4; ++j) dma16(ac + off_a[j], base + (uint32_t)((4 * wave + j) * H * 4));
    } else {
      const bf16s* hc = h + row0 * H;
      const bf16s* rc = saved + row0 * G3;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const uint32_t at = base + (uint32_t)(2 * (2 * wave + j) * H * 2);
        dma16(hc + off_h[j], at);
        if constexpr (KIND == 2) dma16(rc + (off_g[j] - gb * H), at + OFF_R);
      }
    }
    const bf16s* gc = ghat + row0 * G3;
#pragma unroll
    for (int j = 0; j < 2; ++j) dma16(gc + off_g[j], base + (uint32_t)(OFF_G + 2 * (2 * wave + j) * H * 2));
  };

  f32x4 acc[TI][TO];
  float bsum[TO];
#pragma unroll
  for (int o = 0; o < TO; ++o) {
    bsum[o] = 0.f;
#pragma unroll
    for (int i = 0; i < TI; ++i) acc[i][o] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const bool do_bias = KIND == 0 && wi == 0;
  auto compute = [&](int slot) __attribute__((always_inline)) {
    const unsigned char* sb = ring + slot * SLOT;
    const bf16s* sg = reinterpret_cast<const bf16s*>(sb + OFF_G);
    bf16x8 fb[TO];
#pragma unroll
    for (int o = 0; o < TO; ++o) {
      fb[o] = wgw::frag(sg, 0, 16 * (wo * TO + o), lane);
      if (do_bias) {
#pragma unroll
        for (int x = 0; x < 8; ++x) bsum[o] += static_cast<float>(fb[o][x]);
      }
    }
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      const int n0 = 16 * (wi * TI + i);
      bf16x8 fa;
      if constexpr (KIND == 0) {
        fa = frag_f32(reinterpret_cast<const float*>(sb), n0, lane);
      } else {   // h, or r * h (formed over the r tile below)
        fa = wgw::frag(reinterpret_cast<const bf16s*>(sb + (KIND == 2 ? OFF_R : 0)), 0, n0, lane);
      }
#pragma unroll
      for (int o = 0; o < TO; ++o) mma(acc[i][o], fa, fb[o]);
    }
  };
  // Chunk c in slot c % 3: wait for this wave's copies of it (chunk c + 1's
  // may stay in flight), meet the other waves, issue chunk c + 2 into the
  // slot chunk c - 1 used (every wave is past its products), multiply.  The
  // slot is a run-time value: with the loop unrolled over the three slots the
  // compiler keeps every slot's fragment addresses in registers and spills.
#pragma unroll
  for (int c = 0; c < 2; ++c)
    if (c < nchunks) issue(c, c);
  int slot = 0;
  bool pace = sibs != 0u;
#pragma clang loop unroll(disable)
  for (int c = 0; c < nchunks; ++c) {
    if (c + 1 < nchunks) wait_copies<PER>();
    else wait_copies<0>();
    if constexpr (KIND == 2) {
      // r * h of the chunk, formed once (in fp32, rounded to bf16) and
      // written over the r tile (h and r share one layout): each lane forms
      // the 16-byte units its own copies brought in (the same LDS offsets in
      // both tiles), so the wait for its own copies is enough and the
      // products are shared by the barrier below.  (Formed per fragment
      // instead, every element was formed by four waves and the vector ALU
      // work bound these tiles; formed after the barrier by any thread, a
      // second barrier per chunk followed.)
      asm volatile("" ::: "memory");
      unsigned char* sb = ring + slot * SLOT;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int off = 2 * (2 * wave + j) * H * 2 + 16 * lane;
        const u32x4 hv = *reinterpret_cast<const u32x4*>(sb + off);
        u32x4 rv = *reinterpret_cast<const u32x4*>(sb + OFF_R + off);
#pragma unroll
        for (int x = 0; x < 4; ++x) rv[x] = pk2(lo_f(hv[x]) * lo_f(rv[x]), hi_f(hv[x]) * hi_f(rv[x]));
        *reinterpret_cast<u32x4*>(sb + OFF_R + off) = rv;
      }
    }
    if (wave == 0) pace = pace_split(prog + split * 8, tile, sibs, c, lane, pace);
    __syncthreads();
    if (c + 2 < nchunks) issue(c + 2, slot == 0 ? 2 : slot - 1);
    compute(slot);
    slot = slot == 2 ? 0 : slot + 1;
  }

  // D[i = 16 (wi TI + i) + 4g + j][c = gb H + 16 (wo TO + o) + q]
  float* out = P + ((size_t)split * 2 + m) * H * G3 + gb * H;
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int o = 0; o < TO; ++o)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        out[(size_t)(16 * (wi * TI + i) + 4 * g + j) * G3 + 16 * (wo * TO + o) + q] = acc[i][o][j];
  if (do_bias) {
#pragma unroll
    for (int o = 0; o < TO; ++o) {
      float v = bsum[o];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g == 0) Pb[(size_t)split * G3 + gb * H + 16 * (wo * TO + o) + q] = v;
    }
  }
}

__global__ __launch_bounds__(NT) void gru_wgrad256_kernel(const float* __restrict__ a, const bf16s* __restrict__ h,
                                                          const bf16s* __restrict__ saved,
                                                          const bf16s* __restrict__ ghat, float* __restrict__ P,
                                                          float* __restrict__ Pb, long K, int rows_per_split,
                                                          int* __restrict__ prog) {
  __shared__ __attribute__((aligned(1024))) unsigned char ring[NSLOT * SLOT];
  const int tid = threadIdx.x, lane = tid % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int bid = xcd_swizzle(blockIdx.x, gridDim.x);
  const int tile = bid % NTILE, split = bid / NTILE;
  const int m = tile / 3, gb = tile % 3;
  // siblings: the other tiles of this split that run on this workgroup's XCD
  const uint32_t sibs = prog != nullptr ? pace_siblings(bid, split, tile, NTILE, gridDim.x) : 0u;
  if (m == 0)
    gru_wgrad256_body<0>(a, h, saved, ghat, P, Pb, K, rows_per_split, split, m, gb, wave, lane, ring, prog, tile, sibs);
  else if (gb < 2)
    gru_wgrad256_body<1>(a, h, saved, ghat, P, Pb, K, rows_per_split, split, m, gb, wave, lane, ring, prog, tile, sibs);
  else
    gru_wgrad256_body<2>(a, h, saved, ghat, P, Pb, K, rows_per_split, split, m, gb, wave, lane, ring, prog, tile, sibs);
}

}  // namespace gwg
}  // namespace dev

hipError_t launch_transform_wgrad_nm256(int nsplit, int rows_per_split, long K, int E, const void* X, const void* dM,
                                        long ldk, float* P, float* Pb, hipStream_t st) {
  if (rows_per_split % dev::wgw::KC != 0 || K % dev::wgw::KC != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(dev::wgw::transform_wgrad_nm256_kernel, dim3(nsplit * E), dim3(dev::wgw::NT), 0, st,
                     static_cast<const dev::bf16s*>(X), static_cast<const dev::bf16s*>(dM), ldk, P, Pb, K, E,
                     rows_per_split);
  return hipGetLastError();
}

hipError_t launch_gru_wgrad256(int nsplit, int rows_per_split, long K, const float* a, const void* h,
                               const void* saved, const void* ghat, float* P, float* Pb, int* prog, hipStream_t st) {
  if (rows_per_split % dev::gwg::KC != 0 || K % dev::gwg::KC != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(dev::gwg::gru_wgrad256_kernel, dim3(nsplit * dev::gwg::NTILE), dim3(dev::gwg::NT), 0, st, a,
                     static_cast<const dev::bf16s*>(h), static_cast<const dev::bf16s*>(saved),
                     static_cast<const dev::bf16s*>(ghat), P, Pb, K, rows_per_split, prog);
  return hipGetLastError();
}

}  // namespace ggnn
