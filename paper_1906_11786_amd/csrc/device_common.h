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

namespace ggnn {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t bf16s;  // bf16 storage word

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16s v) { return __uint_as_float(static_cast<uint32_t>(v) << 16); }

// Round to nearest bf16, ties to even (finite inputs).
__device__ __forceinline__ bf16s f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<bf16s>(u >> 16);
}

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
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = static_cast<uint32_t>(f2bf(v[2 * i])) | (static_cast<uint32_t>(f2bf(v[2 * i + 1])) << 16);
  u32x4 u = u32x4{w[0], w[1], w[2], w[3]};
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
  u32x2 v = u32x2{static_cast<uint32_t>(f2bf(a)) | (static_cast<uint32_t>(f2bf(b)) << 16),
                       static_cast<uint32_t>(f2bf(c)) | (static_cast<uint32_t>(f2bf(d)) << 16)};
  *reinterpret_cast<u32x2*>(p) = v;
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
  bf16s h[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = f2bf(v[i]);
    l[i] = f2bf(v[i] - bf2f(h[i]));
  }
  *reinterpret_cast<u32x2*>(hi) = u32x2{static_cast<uint32_t>(h[0]) | (static_cast<uint32_t>(h[1]) << 16),
                                        static_cast<uint32_t>(h[2]) | (static_cast<uint32_t>(h[3]) << 16)};
  *reinterpret_cast<u32x2*>(lo) = u32x2{static_cast<uint32_t>(l[0]) | (static_cast<uint32_t>(l[1]) << 16),
                                        static_cast<uint32_t>(l[2]) | (static_cast<uint32_t>(l[3]) << 16)};
}
__device__ __forceinline__ void split_store4(float* hi, float*, f32x4 v) { *reinterpret_cast<f32x4*>(hi) = v; }

// Split eight floats into bf16 hi and lo fragments (see split_store4).
__device__ __forceinline__ void split8(const float* v, bf16x8& hi, bf16x8& lo) {
  float h[8], l[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    h[i] = bf2f(f2bf(v[i]));
    l[i] = v[i] - h[i];
  }
  hi = pack8<bf16s>(h);
  lo = pack8<bf16s>(l);
}

// 16-byte vector copy unit (8 bf16 or 4 fp32 elements).
template <typename S> struct Vec16 { static constexpr int elems = 16 / sizeof(S); };

__device__ __forceinline__ float sigmoidf_(float x) { return 1.0f / (1.0f + __expf(-x)); }
__device__ __forceinline__ float tanhf_(float x) {
  // tanh(x) = 1 - 2 / (exp(2x) + 1), saturating cleanly for large |x|
  float e = __expf(2.0f * x);
  return 1.0f - 2.0f / (e + 1.0f);
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
