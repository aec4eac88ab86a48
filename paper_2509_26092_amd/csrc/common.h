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

// IEEE binary16 storage (the fp16 precision with loss scaling).
typedef _Float16 f16_t;
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

enum Prec { PREC_F32 = 0, PREC_BF16 = 1, PREC_F16 = 2 };

// Elements of the compute type per 16-byte chunk.
inline int prec_vw(int prec) { return prec == PREC_F32 ? 4 : 8; }
inline int prec_bytes(int prec) { return prec == PREC_F32 ? 4 : 2; }

template <typename T> constexpr int prec_of();
template <> constexpr int prec_of<float>() { return PREC_F32; }
template <> constexpr int prec_of<uint16_t>() { return PREC_BF16; }
template <> constexpr int prec_of<f16_t>() { return PREC_F16; }

// Call f with a value of the storage type of `prec` (float, bf16_t or
// f16_t): the host-side dispatch of every templated kernel launch.
template <typename F>
inline int with_prec(int prec, F&& f) {
  switch (prec) {
    case PREC_F32: return f(float{});
    case PREC_BF16: return f(uint16_t{});
    case PREC_F16: return f(f16_t{});
    default: return -1;
  }
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float floatx2_t __attribute__((ext_vector_type(2)));

// Blocks are dealt round-robin to the 8 XCDs (block b to XCD b % 8), each
// with its own L2: this maps block b to a logical block index so that each
// XCD takes a contiguous range of them and neighbouring work shares its L2.
__device__ inline int xcd_remap(int b, int nb) {
  int per = nb >> 3, rem = nb & 7;
  int x = b & 7, r = b >> 3;
  return x * per + (x < rem ? x : rem) + r;
}

// Round-to-nearest-even float -> bf16 (gfx950 v_cvt_pk_bf16_f32; a NaN stays
// a NaN).
__device__ inline bf16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ inline uint32_t f2bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2_t{lo, hi}, bf16x2_t));
}
__device__ __host__ inline float bf2f(bf16_t b) {
  return __builtin_bit_cast(float, ((uint32_t)b) << 16);
}
// Round-to-nearest-even float -> fp16 (v_cvt_f16_f32 in the default rounding
// mode; beyond the largest finite value the result is infinite, so an
// overflow is visible to the finiteness check of loss scaling).
__device__ inline uint32_t f2h2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2_t{lo, hi}, f16x2_t));
}
__device__ inline float h2f(uint16_t b) { return (float)__builtin_bit_cast(_Float16, b); }

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
template <> struct TT<f16_t> {
  static constexpr int VW = 8;
  __device__ static inline float to_f(f16_t v) { return (float)v; }
  __device__ static inline f16_t from_f(float v) { return (f16_t)v; }
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
template <> __device__ inline void unpack<f16_t>(const uint4& q, float* f) {
  uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = h2f((uint16_t)(w[i] & 0xffffu));
    f[2 * i + 1] = h2f((uint16_t)(w[i] >> 16));
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
template <> __device__ inline uint4 pack<f16_t>(const float* f) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = f2h2(f[2 * i], f[2 * i + 1]);
  return make_uint4(w[0], w[1], w[2], w[3]);
}
// Two floats as the 32-bit word of two storage elements (low element first).
template <typename T> __device__ inline uint32_t pack2(float lo, float hi);
template <> __device__ inline uint32_t pack2<bf16_t>(float lo, float hi) { return f2bf2(lo, hi); }
template <> __device__ inline uint32_t pack2<f16_t>(float lo, float hi) { return f2h2(lo, hi); }
// One 16-bit storage element to float.
template <typename T> __device__ inline float s16_to_f(uint16_t b);
template <> __device__ inline float s16_to_f<bf16_t>(uint16_t b) { return bf2f(b); }
template <> __device__ inline float s16_to_f<f16_t>(uint16_t b) { return h2f(b); }

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
