// Device helpers shared by the batch-norm, pooling and convolution kernels:
// the BN affine and the stored ReLU output that the backward passes recompute
// masks from, and the stem's 3x3 stride-2 pad-1 max-pool arithmetic.
#ifndef RN18_POOL_H
#define RN18_POOL_H

#include <math.h>

#include "common.h"

namespace rn18 {

// Batch-norm affine of one value: y * scale + shift as a single fused
// multiply-add, so that every kernel that recomputes an activation (or its
// ReLU mask) from y gets the bits the forward pass stored.
__device__ inline float bn_affine(float y, float scale, float shift) { return __builtin_fmaf(y, scale, shift); }

// relu(bn(y)) as the forward pass stores it (rounded to the storage type):
// the backward pass recomputes ReLU masks from y with this, so each mask
// decision equals the one the stored activation encodes.
template <typename T>
__device__ inline float relu_stored(float y, float sc, float sf) {
  const float t = bn_affine(y, sc, sf);
  return TT<T>::to_f(TT<T>::from_f(t > 0.f ? t : 0.f));
}

// The VW argmax bytes of one 16-byte chunk as one word load / store.
template <int VW> struct ArgVec;
template <> struct ArgVec<8> {
  __device__ static inline void load(const uint8_t* p, uint8_t (&a)[8]) {
    const uint2 v = *(const uint2*)p;
#pragma unroll
    for (int e = 0; e < 4; ++e) { a[e] = (uint8_t)(v.x >> (8 * e)); a[4 + e] = (uint8_t)(v.y >> (8 * e)); }
  }
  __device__ static inline void store(uint8_t* p, const uint8_t (&a)[8]) {
    uint2 v = make_uint2(0u, 0u);
#pragma unroll
    for (int e = 0; e < 4; ++e) { v.x |= (uint32_t)a[e] << (8 * e); v.y |= (uint32_t)a[4 + e] << (8 * e); }
    *(uint2*)p = v;
  }
};
template <> struct ArgVec<4> {
  __device__ static inline void load(const uint8_t* p, uint8_t (&a)[4]) {
    const uint32_t v = *(const uint32_t*)p;
#pragma unroll
    for (int e = 0; e < 4; ++e) a[e] = (uint8_t)(v >> (8 * e));
  }
  __device__ static inline void store(uint8_t* p, const uint8_t (&a)[4]) {
    uint32_t v = 0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) v |= (uint32_t)a[e] << (8 * e);
    *(uint32_t*)p = v;
  }
};

// Output gradients and argmax bytes of the two pool windows (i, j) and
// (i, j + 1), channel chunk cc. The loads are branch-free (clamped to a valid
// window) so that both are in flight together; windows past the output edge
// get argmax 0xff, which matches no tap.
template <typename T>
__device__ inline void pool_window_pair(const T* __restrict__ dy, const uint8_t* __restrict__ arg, int n, int i,
                                        int j, int cc, int cpr, int Ho, int Wo, float (*g)[TT<T>::VW],
                                        uint8_t (*a)[TT<T>::VW]) {
  constexpr int VW = TT<T>::VW;
#pragma unroll
  for (int dj = 0; dj < 2; ++dj) {
    const bool in = i < Ho && j + dj < Wo;
    const int oq = ((n * Ho + min(i, Ho - 1)) * Wo + min(j + dj, Wo - 1)) * cpr + cc;
    unpack<T>(((const uint4*)dy)[oq], g[dj]);
    ArgVec<VW>::load(arg + (long)oq * VW, a[dj]);
#pragma unroll
    for (int e = 0; e < VW; ++e) a[dj][e] = in ? a[dj][e] : (uint8_t)0xff;
  }
}

// Gradient of the pool input at the 2x2 quad of pixels (2qi + py, 2qj + px),
// py, px in {0, 1}: the sum over the windows whose (first) maximum is the
// pixel of their output gradients, in tap order (kh, kw). g[di][dj], a[di][dj]
// are the four windows (qi + di, qj + dj) that can pick a pixel of the quad.
// acc[2*py + px][] receives VW fp32 sums, not yet rounded.
template <int VW>
__device__ inline void pool_quad_combine(const float (*g)[2][VW], const uint8_t (*a)[2][VW], float (*acc)[VW]) {
  // pixel row offset py takes window rows (tap row kh, window di) in kh order:
  // py = 0: (1, 0); py = 1: (0, 1), (2, 0). Columns likewise.
#pragma unroll
  for (int py = 0; py < 2; ++py)
#pragma unroll
    for (int px = 0; px < 2; ++px) {
      float* o = acc[2 * py + px];
#pragma unroll
      for (int e = 0; e < VW; ++e) o[e] = 0.f;
#pragma unroll
      for (int rh = 0; rh < 2; ++rh) {
        if (py == 0 && rh == 1) continue;
        const int kh = py == 0 ? 1 : (rh == 0 ? 0 : 2), di = py == 0 ? 0 : (rh == 0 ? 1 : 0);
#pragma unroll
        for (int rw = 0; rw < 2; ++rw) {
          if (px == 0 && rw == 1) continue;
          const int kw = px == 0 ? 1 : (rw == 0 ? 0 : 2), dj = px == 0 ? 0 : (rw == 0 ? 1 : 0);
          const uint8_t tap = (uint8_t)(kh * 3 + kw);
#pragma unroll
          for (int e = 0; e < VW; ++e)
            if (a[di][dj][e] == tap) o[e] += g[di][dj][e];
        }
      }
    }
}

// The same for one quad, loading its four windows.
template <typename T>
__device__ inline void pool_grad_quad(const T* __restrict__ dy, const uint8_t* __restrict__ arg, int n, int qi,
                                      int qj, int cc, int cpr, int Ho, int Wo, float (*acc)[TT<T>::VW]) {
  constexpr int VW = TT<T>::VW;
  float g[2][2][VW];
  uint8_t a[2][2][VW];
  pool_window_pair<T>(dy, arg, n, qi, qj, cc, cpr, Ho, Wo, g[0], a[0]);
  pool_window_pair<T>(dy, arg, n, qi + 1, qj, cc, cpr, Ho, Wo, g[1], a[1]);
  pool_quad_combine<VW>(g, a, acc);
}

// Max over the 3x3 window of output (n, i, j), channel chunk cc, of the
// values v = act(x) (act maps a loaded fp32 chunk in place); -inf padding,
// first maximum in (kh, kw) order wins.
template <typename T, typename Act>
__device__ inline void pool_max_window(const T* __restrict__ x, int n, int i, int j, int cc, int H, int W, int C,
                                       const Act& act, float* best, uint8_t* bi) {
  constexpr int VW = TT<T>::VW;
#pragma unroll
  for (int e = 0; e < VW; ++e) { best[e] = -INFINITY; bi[e] = 0; }
  // branch-free: taps outside the input load a clamped pixel and count as -inf
  float v[3][3][VW];
#pragma unroll
  for (int kh = 0; kh < 3; ++kh)
#pragma unroll
    for (int kw = 0; kw < 3; ++kw) {
      const int h = 2 * i - 1 + kh, w = 2 * j - 1 + kw;
      const int hc = min(max(h, 0), H - 1), wc = min(max(w, 0), W - 1);
      unpack<T>(((const uint4*)x)[((n * H + hc) * W + wc) * (C / VW) + cc], v[kh][kw]);
    }
#pragma unroll
  for (int kh = 0; kh < 3; ++kh)
#pragma unroll
    for (int kw = 0; kw < 3; ++kw) {
      const int h = 2 * i - 1 + kh, w = 2 * j - 1 + kw;
      const bool in = (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W;
      act(v[kh][kw]);
#pragma unroll
      for (int e = 0; e < VW; ++e)
        if (in && v[kh][kw][e] > best[e]) { best[e] = v[kh][kw][e]; bi[e] = (uint8_t)(kh * 3 + kw); }
    }
}

}  // namespace rn18
#endif
