// Shared device/host helpers for the gfx950 ResNet-18 training-step library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace rn18 {

// bf16 is stored as its raw 16-bit pattern; MFMA operands reinterpret 16-byte
// chunks as vectors of __bf16.
typedef uint16_t bf16_t;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

enum Prec { PREC_F32 = 0, PREC_BF16 = 1 };

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float floatx2_t __attribute__((ext_vector_type(2)));

// Round-to-nearest-even float -> bf16 (gfx950 v_cvt_pk_bf16_f32; a NaN stays
// a NaN).
__device__ inline bf16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ inline uint32_t f2bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2_t{lo, hi}, bf16x2_t));
}
__device__ __host__ inline float bf2f(bf16_t b) {
  return __builtin_bit_cast(float, ((uint32_t)b) << 16);
}

// Element-type traits: a 16-byte chunk holds VW elements.
template <typename T> struct TT;
template <> struct TT<float> {
  static constexpr int VW = 4;
  __device__ static inline float to_f(float v) { return v; }
  __device__ static inline float from_f(float v) { return v; }
};
template <> struct TT<bf16_t> {
  static constexpr int VW = 8;
  __device__ static inline float to_f(bf16_t v) { return bf2f(v); }
  __device__ static inline bf16_t from_f(float v) { return f2bf(v); }
};

// Unpack / pack a 16-byte chunk (uint4) to / from VW floats.
template <typename T> __device__ inline void unpack(const uint4& q, float* f);
template <> __device__ inline void unpack<float>(const uint4& q, float* f) {
  f[0] = __builtin_bit_cast(float, q.x); f[1] = __builtin_bit_cast(float, q.y);
  f[2] = __builtin_bit_cast(float, q.z); f[3] = __builtin_bit_cast(float, q.w);
}
template <> __device__ inline void unpack<bf16_t>(const uint4& q, float* f) {
  uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __builtin_bit_cast(float, w[i] << 16);
    f[2 * i + 1] = __builtin_bit_cast(float, w[i] & 0xffff0000u);
  }
}
template <typename T> __device__ inline uint4 pack(const float* f);
template <> __device__ inline uint4 pack<float>(const float* f) {
  uint4 q;
  q.x = __builtin_bit_cast(uint32_t, f[0]); q.y = __builtin_bit_cast(uint32_t, f[1]);
  q.z = __builtin_bit_cast(uint32_t, f[2]); q.w = __builtin_bit_cast(uint32_t, f[3]);
  return q;
}
template <> __device__ inline uint4 pack<bf16_t>(const float* f) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = f2bf2(f[2 * i], f[2 * i + 1]);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// Division by a runtime constant d >= 1 for numerators below 2^31, as a
// multiply-high, an add and a shift (round-up multiplier of Granlund and
// Montgomery): l = ceil(log2 d), m = floor(2^32 (2^l - d) / d) + 1,
// n / d = (umulhi(n, m) + n) >> l.
struct FastDiv {
  uint32_t d, m, l;
  FastDiv() : d(1), m(1), l(0) {}
  explicit FastDiv(uint32_t dd) : d(dd ? dd : 1) {
    l = 0;
    while ((1ull << l) < d) ++l;
    m = (uint32_t)((((1ull << 32) * ((1ull << l) - d)) / d) + 1);
  }
  __device__ inline uint32_t div(uint32_t n) const { return (__umulhi(n, m) + n) >> l; }
};

// Sticky device error bits.
enum DevErr { DEVERR_LABEL = 1, DEVERR_NONFINITE = 2 };

inline int ceil_div(long a, long b) { return (int)((a + b - 1) / b); }

}  // namespace rn18
