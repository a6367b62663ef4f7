// Device helpers shared by the gfx950 kernels: storage types, bf16 rounding,
// matrix-core fragments and the 16x16 MFMA tile step.
//
// Tile convention (one wave = 64 lanes; l = lane id, g = l / 16, q = l % 16):
//   D[16][16] += A[16][32] * B[32][16] over one 32-wide k step.
//   A fragment: lane holds row m = q of A, eight k values of group g.
//   B fragment: lane holds column n = q of B, the same eight k values.
//   D (accumulator, 4 floats): lane holds D[4g + j][q], j = 0..3.
// Which eight of the 32 k indices group g holds is a free choice (the sum
// over k does not care) as long as A and B agree; kernels pick an order that
// makes their memory reads contiguous.  bf16 uses one
// v_mfma_f32_16x16x32_bf16; fp32 uses eight v_mfma_f32_16x16x4_f32, the i-th
// taking element i of the same fragments, so one kernel source serves both.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

// Each kernel source is compiled twice: GGNN_DT_BF16=1 builds its bf16
// kernels (matrix-core results kept in VGPRs), GGNN_DT_BF16=0 its fp32 ones.
// The launchers of one build live in namespace ggnn::GGNN_IMPL_NS.
#ifndef GGNN_DT_BF16
#error "compile with -DGGNN_DT_BF16=1 (bf16 kernels) or -DGGNN_DT_BF16=0 (fp32 kernels)"
#endif
#if GGNN_DT_BF16
#define GGNN_IMPL_NS impl_bf16
#else
#define GGNN_IMPL_NS impl_f32
#endif

namespace ggnn {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t bf16s;  // bf16 storage word
#if GGNN_DT_BF16
typedef bf16s dt_t;      // storage type of the bf16 object (GGNN_DT_BF16)
#else
typedef float dt_t;
#endif
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16s v) { return __uint_as_float(static_cast<uint32_t>(v) << 16); }

// Round to nearest bf16, ties to even: gfx950 converts two floats per
// instruction (v_cvt_pk_bf16_f32), element 0 in the low half.
__device__ __forceinline__ uint32_t pk2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ bf16s f2bf(float f) { return __builtin_bit_cast(bf16s, static_cast<__bf16>(f)); }
// The two bf16 halves of a packed word as floats.
__device__ __forceinline__ float lo_f(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Storage element -> float and back.
template <typename S> __device__ __forceinline__ float to_f(S v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<bf16s>(bf16s v) { return bf2f(v); }
template <typename S> __device__ __forceinline__ S from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16s from_f<bf16s>(float v) { return f2bf(v); }

// Fragment type of a storage type.
template <typename S> struct Frag;
template <> struct Frag<float> { using type = f32x8; };
template <> struct Frag<bf16s> { using type = bf16x8; };
template <typename S> using frag_t = typename Frag<S>::type;

__device__ __forceinline__ void mma(f32x4& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x4& acc, const f32x8& a, const f32x8& b) {
#pragma unroll
  for (int i = 0; i < 8; ++i) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[i], acc, 0, 0, 0);
}

// ---- fragment builders -------------------------------------------------

// Eight contiguous elements (16 B for bf16, 32 B for fp32; p 16-B aligned).
__device__ __forceinline__ bf16x8 load8(const bf16s* p) {
  u32x4 v = *reinterpret_cast<const u32x4*>(p);
  return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ f32x8 load8(const float* p) {
  f32x4 a = *reinterpret_cast<const f32x4*>(p);
  f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
  f32x8 r;
  r[0] = a.x; r[1] = a.y; r[2] = a.z; r[3] = a.w;
  r[4] = b.x; r[5] = b.y; r[6] = b.z; r[7] = b.w;
  return r;
}

// Two runs of four contiguous elements (8-B / 16-B aligned).
__device__ __forceinline__ bf16x8 load4x2(const bf16s* p0, const bf16s* p1) {
  u32x2 a = *reinterpret_cast<const u32x2*>(p0);
  u32x2 b = *reinterpret_cast<const u32x2*>(p1);
  u32x4 v = u32x4{a.x, a.y, b.x, b.y};
  return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ f32x8 load4x2(const float* p0, const float* p1) {
  f32x4 a = *reinterpret_cast<const f32x4*>(p0);
  f32x4 b = *reinterpret_cast<const f32x4*>(p1);
  f32x8 r;
  r[0] = a.x; r[1] = a.y; r[2] = a.z; r[3] = a.w;
  r[4] = b.x; r[5] = b.y; r[6] = b.z; r[7] = b.w;
  return r;
}

// Eight elements at a stride (transposed read, typically from LDS).
__device__ __forceinline__ bf16x8 load8_strided(const bf16s* p, int stride) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = static_cast<uint32_t>(p[(2 * i) * stride]) | (static_cast<uint32_t>(p[(2 * i + 1) * stride]) << 16);
  u32x4 v = u32x4{w[0], w[1], w[2], w[3]};
  return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ f32x8 load8_strided(const float* p, int stride) {
  f32x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = p[i * stride];
  return r;
}

// Build a fragment from eight floats, rounding to the storage type.
template <typename S> __device__ __forceinline__ frag_t<S> pack8(const float* v);
template <> __device__ __forceinline__ bf16x8 pack8<bf16s>(const float* v) {
  u32x4 u = u32x4{pk2(v[0], v[1]), pk2(v[2], v[3]), pk2(v[4], v[5]), pk2(v[6], v[7])};
  return __builtin_bit_cast(bf16x8, u);
}
template <> __device__ __forceinline__ f32x8 pack8<float>(const float* v) {
  f32x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = v[i];
  return r;
}

// Store four consecutive elements from floats (8 B for bf16, 16 B for fp32).
__device__ __forceinline__ void store4(bf16s* p, float a, float b, float c, float d) {
  *reinterpret_cast<u32x2*>(p) = u32x2{pk2(a, b), pk2(c, d)};
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<f32x4*>(p) = f32x4{a, b, c, d};
}

// Load four consecutive elements as floats.
__device__ __forceinline__ f32x4 load4f(const bf16s* p) {
  u32x2 v = *reinterpret_cast<const u32x2*>(p);
  return f32x4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u), __uint_as_float(v.y << 16),
                     __uint_as_float(v.y & 0xFFFF0000u)};
}
__device__ __forceinline__ f32x4 load4f(const float* p) { return *reinterpret_cast<const f32x4*>(p); }

// Store four floats as storage elements.  For bf16 the value is split into
// hi = bf16(x) and lo = bf16(x - hi) (hi + lo equals x to about 16 bits);
// for fp32 only `hi` is written (hi and lo then point to the same place).
__device__ __forceinline__ void split_store4(bf16s* hi, bf16s* lo, f32x4 v) {
  const uint32_t h0 = pk2(v[0], v[1]), h1 = pk2(v[2], v[3]);
  *reinterpret_cast<u32x2*>(hi) = u32x2{h0, h1};
  *reinterpret_cast<u32x2*>(lo) =
      u32x2{pk2(v[0] - lo_f(h0), v[1] - hi_f(h0)), pk2(v[2] - lo_f(h1), v[3] - hi_f(h1))};
}
__device__ __forceinline__ void split_store4(float* hi, float*, f32x4 v) { *reinterpret_cast<f32x4*>(hi) = v; }

// Split eight floats into bf16 hi and lo fragments (see split_store4).
__device__ __forceinline__ void split8(const float* v, bf16x8& hi, bf16x8& lo) {
  u32x4 h, l;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = pk2(v[2 * i], v[2 * i + 1]);
    l[i] = pk2(v[2 * i] - lo_f(h[i]), v[2 * i + 1] - hi_f(h[i]));
  }
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}

// A V x V tile (V = 16 / sizeof(S): 8 x 8 bf16 or 4 x 4 fp32) moved from
// global memory to LDS transposed: V row loads of 16 bytes, a transpose in
// registers (v_perm_b32 on 16-bit halves for bf16), V 16-byte LDS stores.
//   tile_load:    r[i] = src[i * ss .. i * ss + V)
//   tile_store_T: dst[x * P + i] = r[i][x]          (dst, P 16-byte aligned)
template <typename S>
__device__ __forceinline__ void tile_load(u32x4 (&r)[16 / sizeof(S)], const S* src, long ss) {
#pragma unroll
  for (int i = 0; i < (int)(16 / sizeof(S)); ++i) r[i] = *reinterpret_cast<const u32x4*>(src + i * ss);
}
//   tile_row_T:   row x of the transposed tile, (r[0][x], ..., r[V-1][x])
template <typename S>
__device__ __forceinline__ u32x4 tile_row_T(const u32x4 (&r)[16 / sizeof(S)], int x) {
  if constexpr (sizeof(S) == 2) {
    const uint32_t sel = (x & 1) ? 0x07060302u : 0x05040100u;   // high or low halves of r[2j], r[2j+1]
    u32x4 o;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) o[jj] = __builtin_amdgcn_perm(r[2 * jj + 1][x / 2], r[2 * jj][x / 2], sel);
    return o;
  } else {
    return u32x4{r[0][x], r[1][x], r[2][x], r[3][x]};
  }
}
template <typename S, int P>
__device__ __forceinline__ void tile_store_T(S* dst, const u32x4 (&r)[16 / sizeof(S)]) {
#pragma unroll
  for (int x = 0; x < (int)(16 / sizeof(S)); ++x) *reinterpret_cast<u32x4*>(dst + x * P) = tile_row_T<S>(r, x);
}

// Fragment order in LDS: operand fragments stored so that, for each
// fragment, the 64 lanes' copies are contiguous (per 16-byte vector), so a
// wave's fragment read covers consecutive bytes.  The LDS serves 16 lanes'
// 16-byte reads per pass from 64 four-byte banks: such a read never
// conflicts, where rows read at a padded pitch took two passes.
// fo: element e (0..7) of lane `lane`'s copy of fragment `idx`.
template <typename S>
__device__ __forceinline__ int fo(int idx, int lane, int e) {
  constexpr int V = 16 / (int)sizeof(S), NV = 8 / V;
  return ((idx * NV + e / V) * 64 + lane) * V + e % V;
}
template <typename S>
__device__ __forceinline__ frag_t<S> load_fragi(const S* v, int idx, int lane) {
  if constexpr (sizeof(S) == 2) {
    return load8(v + fo<S>(idx, lane, 0));
  } else {
    return load4x2(v + fo<S>(idx, lane, 0), v + fo<S>(idx, lane, 4));
  }
}
// GRU weights Wi, U ([H][3H]) staged in LDS in fragment order, each
// fragment holding eight input features in accumulator-compatible order
// (32kk + 4g + {0..3}, 32kk + 16 + 4g + {0..3}) of one gate column:
//   gru_fwd_frag: A operand of D[gate col][node], rows = gate columns
//                 col..col+15 (mat 0 = Wi, 1 = U);
//   gru_rev_frag: operand rows = input features row..row+15, k = gate
//                 columns gate*H + 32kk + ... (the reverse products).
template <typename S, int H>
__device__ __forceinline__ int gru_fwd_idx(int mat, int col16, int kk) {
  return (mat * (3 * H / 16) + col16) * (H / 32) + kk;
}
template <typename S, int H>
__device__ __forceinline__ int gru_rev_idx(int mat, int row16, int gate, int kk) {
  return ((mat * (H / 16) + row16) * 3 + gate) * (H / 32) + kk;
}
// Place four consecutive elements `w` (8 bytes bf16, 16 bytes fp32) of the
// k run starting at k0 (4-aligned, within a 32-step) of fragment `idx`, row
// r16 (0..15) of its operand tile.
template <typename S>
__device__ __forceinline__ void put4(S* base, int idx, int r16, int k0, const S* w) {
  const int kk32 = k0 % 32, half = kk32 / 16, g = (kk32 % 16) / 4;
  S* d = base + fo<S>(idx, r16 + 16 * g, 4 * half);
  if constexpr (sizeof(S) == 2) {
    *reinterpret_cast<u32x2*>(d) = *reinterpret_cast<const u32x2*>(w);
  } else {
    *reinterpret_cast<u32x4*>(d) = *reinterpret_cast<const u32x4*>(w);
  }
}


// Fragment of an operand stored k-major in LDS (element (k, n) at
// base[k * P + n]): lane (q, g) receives elements (k0 + 8g + j, n0 + q),
// j = 0..7.  For bf16 this is two transposing reads (ds_read_b64_tr_b16: in
// each group of 16 lanes, lane i receives element i % 4 of the 8-byte runs
// addressed by lanes i / 4, 4 + i / 4, 8 + i / 4 and 12 + i / 4); lane p of a
// group addresses row k0 + 8g + p / 4 (+ 4 for the second read) at column
// n0 + 4 (p % 4).  n0 and P are multiples of 4; the rows of one 16-lane
// group fall on disjoint banks when P * 2 bytes is 160 mod 256.
typedef short tr_v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) tr_v4i16 lds_tr_v4i16;
__device__ __forceinline__ bf16x8 tr_frag(const bf16s* base, int P, int k0, int n0, int lane) {
  const int p = lane % 16, g = lane / 16;
  bf16s* a0 = const_cast<bf16s*>(base) + (k0 + 8 * g + p / 4) * P + n0 + 4 * (p % 4);
  const tr_v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_tr_v4i16*)(a0));
  const tr_v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_tr_v4i16*)(a0 + 4 * P));
  typedef short v8i16 __attribute__((ext_vector_type(8)));
  const v8i16 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ f32x8 tr_frag(const float* base, int P, int k0, int n0, int lane) {
  const int q = lane % 16, g = lane / 16;
  f32x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = base[(k0 + 8 * g + j) * P + n0 + q];
  return r;
}

// 16-byte vector copy unit (8 bf16 or 4 fp32 elements).
template <typename S> struct Vec16 { static constexpr int elems = 16 / sizeof(S); };

// Gate nonlinearities: hardware exp2 and reciprocal (v_exp_f32, v_rcp_f32,
// each within about 1 ulp) instead of an IEEE division sequence.
__device__ __forceinline__ float sigmoidf_(float x) { return __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }
__device__ __forceinline__ float tanhf_(float x) {
  // tanh(x) = 1 - 2 / (exp(2x) + 1), saturating cleanly for large |x|
  return 1.0f - 2.0f * __builtin_amdgcn_rcpf(__expf(2.0f * x) + 1.0f);
}

// A lane's NB bit-row bytes (NB = 4 or 8) from the split order to the
// contiguous one.  Split: lane group g (lanes 16g .. 16g + 15) holds row
// bytes NB g .. NB g + NB - 1, as a 32-bit load per 4 bytes delivers them;
// contiguous: byte kk of lane group g is row byte 4 kk + g, so that one
// matrix-core k step covers 32 consecutive block columns.  A 4 x 4
// transpose between the lane groups of a wave: one permlane32 and one
// permlane16 swap and byte permutes.  `odd` is g & 1.
template <int NB>
__device__ __forceinline__ void bytes_to_contiguous(uint32_t* w, uint32_t odd) {
  static_assert(NB == 4 || NB == 8, "contiguous order for 4- or 8-byte rows");
  if constexpr (NB == 8) {
    // lane g' holds k steps 2g' (w[0]) and 2g'+1 (w[1]), byte d = group d.
    // Pair the two steps per destination group: L for groups 0, 1, U for 2, 3.
    uint32_t L = __builtin_amdgcn_perm(w[1], w[0], 0x05010400u);
    uint32_t U = __builtin_amdgcn_perm(w[1], w[0], 0x07030602u);
    // lanes 0-31 keep L and take L of lanes 32-63; lanes 32-63 keep U.
    auto r32 = __builtin_amdgcn_permlane32_swap(L, U, false, false);
    L = r32[0];
    U = r32[1];
    uint32_t X0 = __builtin_amdgcn_perm(U, L, 0x05040100u);   // pairs for the even group of the half
    uint32_t X1 = __builtin_amdgcn_perm(U, L, 0x07060302u);   // pairs for the odd group
    auto r16 = __builtin_amdgcn_permlane16_swap(X0, X1, false, false);
    X0 = r16[0];   // pairs of source lane groups 0 and 2
    X1 = r16[1];   // pairs of source lane groups 1 and 3
    w[0] = __builtin_amdgcn_perm(X1, X0, 0x05040100u);      // steps 0..3
    w[1] = __builtin_amdgcn_perm(X1, X0, 0x07060302u);      // steps 4..7
    (void)odd;
  } else {
    // lane g' holds k step g' (byte d = group d).
    const uint32_t D = w[0];
    const uint32_t Yr = __builtin_amdgcn_perm(D, D, 0x01000302u);   // halves rotated
    auto r32 = __builtin_amdgcn_permlane32_swap(D, Yr, false, false);
    const uint32_t Z = __builtin_amdgcn_perm(r32[1], r32[0], 0x05040100u);
    auto r16 = __builtin_amdgcn_permlane16_swap(Z, Z, false, false);
    w[0] = __builtin_amdgcn_perm(r16[1], r16[0], odd ? 0x07030501u : 0x06020400u);
  }
}

// Logical workgroup index spread so that consecutive logical tiles land on the
// same XCD (workgroups are dispatched round-robin over the 8 XCDs, each with
// its own L2): neighbouring tiles then share operand data in one L2.
__device__ __forceinline__ int xcd_swizzle(int bid, int nblocks) {
  constexpr int kXcd = 8;
  int per = nblocks / kXcd;        // full rounds
  int rem = nblocks % kXcd;
  int xcd = bid % kXcd;
  int idx = bid / kXcd;
  // XCDs [0, rem) own per + 1 tiles, the rest own per.
  int base = xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per;
  return base + idx;
}

}  // namespace dev
}  // namespace ggnn
