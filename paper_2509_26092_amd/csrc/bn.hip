// Batch normalisation (training mode) over an NHWC tensor viewed as [M][C]:
// statistics per channel over all M = N*H*W rows.
//
// Statistics are two-level and deterministic. Forward: the conv epilogue
// writes per-tile partial sums of (v - shift) and (v - shift)^2 with a sample
// of the channel as the shift (well conditioned when |mean| >> std), and a
// finalize kernel merges the tiles in fp64. Backward: each block reduces a
// contiguous range of rows to per-channel partial sums in fp32 (16-byte row
// chunks read coalesced, then a fixed-order LDS reduction), combined in fp64.
//
// The elementwise passes (apply + ReLU + residual, backward apply) are 16-byte
// HBM streams with the per-channel coefficients staged in LDS.
#include <hip/hip_ext.h>

#include "kernels.h"
#include "pool.h"

namespace rn18 {

namespace {

constexpr int kMaxC = 512;

// Blocks of a grid-sweeping reduction over M rows, rows_per_iter rows per
// block step: every thread takes at least min_rows rows and at most cap
// blocks run, but while each thread would still take 8 rows there are at
// least floor_blocks. Measured on the BN backward reductions at bf16: up to
// two blocks per CU with 16 rows per thread beat more blocks with fewer rows
// (50176 x 256: 784 blocks 20.4 us, 392 blocks 15.7 us), and a grid smaller
// than the CU count is slower again.
int pick_blocks(long M, int rows_per_iter, int min_rows, int cap, int floor_blocks) {
  long b = M / ((long)rows_per_iter * min_rows);
  if (b > cap) b = cap;
  const long lo8 = M / ((long)rows_per_iter * 8), lo = lo8 < floor_blocks ? lo8 : floor_blocks;
  if (b < lo) b = lo;
  if (b < 1) b = 1;
  return (int)b;
}

__device__ inline double block_sum_d(double v, double* sh) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) sh[tid] += sh[tid + s];
    __syncthreads();
  }
  double r = sh[0];
  __syncthreads();
  return r;
}

// Batch statistics from the per-tile partials (rows n, shift x0, sum of
// v - x0, sum of (v - x0)^2) of the forward conv epilogue. Every tile's sums
// are re-referenced to one sample of the channel, K = tile 0's shift, in
// fp64 (d = x0 - K: S1 += s1 + n d, S2 += s2 + 2 d s1 + n d^2), so the
// tiles simply add. Stage 1: grid (channel groups of 64, tile chunks), 4
// thread groups per block over a chunk's tiles, fixed-order combine; stage 2:
// per channel, 4 thread groups over the chunks, fixed-order combine, then
// mean = K + S1/M, biased variance
// S2/M - (S1/M)^2 for normalising, unbiased (M/(M-1)) for the running one.
// With a single chunk (at most 64 tiles) stage 1 finishes the statistics
// itself and stage 2 is not launched.
struct BnStatsOut {
  const float* gamma;
  const float* beta;
  float eps, mom;
  float* rm;
  float* rv;
  float* mean;
  float* rstd;
  float* scale;
  float* shift;
};

__device__ inline void bn_stats_finish(int c, double N, double S1, double S2, double K, const BnStatsOut& o) {
  const double m1 = S1 / N;
  double var = S2 / N - m1 * m1;
  if (var < 0.0) var = 0.0;
  const double mean = K + m1;
  const double rstd = 1.0 / sqrt(var + (double)o.eps);
  const double sc = (double)o.gamma[c] * rstd;
  o.mean[c] = (float)mean;
  o.rstd[c] = (float)rstd;
  o.scale[c] = (float)sc;
  o.shift[c] = (float)((double)o.beta[c] - mean * sc);
  if (o.rm) {
    o.rm[c] = (float)((1.0 - o.mom) * (double)o.rm[c] + o.mom * mean);
    o.rv[c] = (float)((1.0 - o.mom) * (double)o.rv[c] + o.mom * (N > 1.0 ? var * (N / (N - 1.0)) : 0.0));
  }
}

__global__ __launch_bounds__(256) void bn_stats_tiles_reduce_kernel(const float* __restrict__ st, int ntiles, int C,
                                                                    int per_chunk, double* __restrict__ red,
                                                                    BnStatsOut o) {
  __shared__ double sh[3][4][64];
  const int cl = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + cl;
  const int z0 = blockIdx.y * per_chunk, z1 = min(ntiles, z0 + per_chunk);
  double N = 0.0, S1 = 0.0, S2 = 0.0;
  if (c < C) {
    const double K = (double)((const float4*)st)[c].y;
#pragma unroll 8
    for (int z = z0 + q; z < z1; z += 4) {
      const float4 p = ((const float4*)st)[(long)z * C + c];
      const double n = p.x, d = (double)p.y - K, s1 = p.z;
      N += n;
      S1 += s1 + n * d;
      S2 += (double)p.w + 2.0 * d * s1 + n * d * d;
    }
  }
  sh[0][q][cl] = N; sh[1][q][cl] = S1; sh[2][q][cl] = S2;
  __syncthreads();
  if (q == 0 && c < C) {
    double v[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) v[k] = ((sh[k][0][cl] + sh[k][1][cl]) + sh[k][2][cl]) + sh[k][3][cl];
    if (gridDim.y == 1) {
      bn_stats_finish(c, v[0], v[1], v[2], (double)((const float4*)st)[c].y, o);
    } else {
      double* out = red + ((long)blockIdx.y * C + c) * 3;
#pragma unroll
      for (int k = 0; k < 3; ++k) out[k] = v[k];
    }
  }
}

__global__ __launch_bounds__(256) void bn_stats_tiles_final_kernel(const float* __restrict__ st,
                                                                   const double* __restrict__ red, int nchunks, int C,
                                                                   BnStatsOut o) {
  __shared__ double sh[3][4][64];
  const int cl = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + cl;
  double N = 0.0, S1 = 0.0, S2 = 0.0;
  if (c < C) {
#pragma unroll 4
    for (int r = q; r < nchunks; r += 4) {
      const double* p = red + ((long)r * C + c) * 3;
      N += p[0];
      S1 += p[1];
      S2 += p[2];
    }
  }
  sh[0][q][cl] = N; sh[1][q][cl] = S1; sh[2][q][cl] = S2;
  __syncthreads();
  if (q != 0 || c >= C) return;
  N = ((sh[0][0][cl] + sh[0][1][cl]) + sh[0][2][cl]) + sh[0][3][cl];
  S1 = ((sh[1][0][cl] + sh[1][1][cl]) + sh[1][2][cl]) + sh[1][3][cl];
  S2 = ((sh[2][0][cl] + sh[2][1][cl]) + sh[2][2][cl]) + sh[2][3][cl];
  bn_stats_finish(c, N, S1, S2, (double)((const float4*)st)[c].y, o);
}


template <typename T>
__global__ __launch_bounds__(256) void bn_apply_kernel(const T* __restrict__ y, const float* __restrict__ scale,
                                                       const float* __restrict__ shift, int relu, int res_mode,
                                                       const T* __restrict__ r, const float* __restrict__ scale2,
                                                       const float* __restrict__ shift2, T* __restrict__ z,
                                                       long nchunks, int C, uint8_t* __restrict__ mbits) {
  constexpr int VW = TT<T>::VW;
  __shared__ float sc[kMaxC], sf[kMaxC], sc2[kMaxC], sf2[kMaxC];
  for (int c = threadIdx.x; c < C; c += 256) {
    sc[c] = scale[c];
    sf[c] = shift[c];
    if (res_mode == 2) { sc2[c] = scale2[c]; sf2[c] = shift2[c]; }
  }
  __syncthreads();
  const int cpr = C / VW;
  for (long q = blockIdx.x * 256l + threadIdx.x; q < nchunks; q += (long)gridDim.x * 256) {
    const int c0 = (int)(q % cpr) * VW;
    float v[VW];
    unpack<T>(((const uint4*)y)[q], v);
#pragma unroll
    for (int e = 0; e < VW; ++e) v[e] = bn_affine(v[e], sc[c0 + e], sf[c0 + e]);
    if (res_mode == 1) {
      float w[VW];
      unpack<T>(((const uint4*)r)[q], w);
#pragma unroll
      for (int e = 0; e < VW; ++e) v[e] += w[e];
    } else if (res_mode == 2) {
      float w[VW];
      unpack<T>(((const uint4*)r)[q], w);
#pragma unroll
      for (int e = 0; e < VW; ++e) v[e] += w[e] * sc2[c0 + e] + sf2[c0 + e];
    }
    if (relu) {
#pragma unroll
      for (int e = 0; e < VW; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
    }
    const uint4 pk = pack<T>(v);
    ((uint4*)z)[q] = pk;
    if (mbits) {
      // bit e: element e of the chunk as stored is > 0 (its ReLU mask)
      float vr[VW];
      unpack<T>(pk, vr);
      uint32_t b = 0;
#pragma unroll
      for (int e = 0; e < VW; ++e) b |= (vr[e] > 0.f ? 1u : 0u) << e;
      mbits[q] = (uint8_t)b;
    }
  }
}

__global__ void bn_eval_coef_kernel(const float* gamma, const float* beta, const float* rm, const float* rv,
                                    float eps, int C, float* scale, float* shift) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= C) return;
  const double rstd = 1.0 / sqrt((double)rv[c] + (double)eps);
  const double s = (double)gamma[c] * rstd;
  scale[c] = (float)s;
  shift[c] = (float)((double)beta[c] - (double)rm[c] * s);
}

template <typename T>
__global__ __launch_bounds__(256) void bn_bwd_partial_kernel(const T* __restrict__ dz, const uint8_t* __restrict__ mb,
                                                             const T* __restrict__ y, const float* __restrict__ mean,
                                                             const float* __restrict__ rstd,
                                                             const float* __restrict__ mscale,
                                                             const float* __restrict__ mshift, long M, int C,
                                                             float* __restrict__ part) {
  constexpr int VW = TT<T>::VW;
  __shared__ float red[2][256 * VW];
  const int tpc = C / VW, rpi = 256 / tpc;
  const int tid = threadIdx.x, cg = tid % tpc, rr = tid / tpc;
  // the grid sweeps the rows together: at each step block b takes rows
  // (step * G + b) * rpi .. + rpi - 1, so the whole grid reads one contiguous
  // stretch of each tensor at a time
  const long gstride = (long)gridDim.x * rpi;
  float mu[VW], rs[VW], s1[VW], s2[VW], msc[VW], msf[VW];
#pragma unroll
  for (int e = 0; e < VW; ++e) {
    mu[e] = mean[cg * VW + e];
    rs[e] = rstd[cg * VW + e];
    msc[e] = mscale ? mscale[cg * VW + e] : 0.f;
    msf[e] = mscale ? mshift[cg * VW + e] : 0.f;
    s1[e] = s2[e] = 0.f;
  }
  // four rows per step, all loads issued before any is used (rows past the
  // end load the thread's first row of the step and add nothing)
  constexpr int U = 4;
  for (long r0 = (long)blockIdx.x * rpi + rr; r0 < M; r0 += U * gstride) {
    uint4 qg[U], qy[U];
    uint32_t qm[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const long r = r0 + u * gstride < M ? r0 + u * gstride : r0;
      const long o = r * C + cg * VW;
      qg[u] = *(const uint4*)(dz + o);
      qy[u] = *(const uint4*)(y + o);
      if (mb) qm[u] = mb[r * tpc + cg];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool live_row = r0 + u * gstride < M;
      float g[VW], yy[VW];
      unpack<T>(qg[u], g);
      unpack<T>(qy[u], yy);
      if (mb) {
#pragma unroll
        for (int e = 0; e < VW; ++e) g[e] = (qm[u] >> e) & 1u ? g[e] : 0.f;
      } else if (mscale) {
        // the ReLU mask of relu(bn(y)), from the stored value's arithmetic
#pragma unroll
        for (int e = 0; e < VW; ++e) g[e] = relu_stored<T>(yy[e], msc[e], msf[e]) > 0.f ? g[e] : 0.f;
      }
#pragma unroll
      for (int e = 0; e < VW; ++e) {
        const float gv = live_row ? g[e] : 0.f;
        s1[e] += gv;
        s2[e] += gv * ((yy[e] - mu[e]) * rs[e]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < VW; ++e) {
    red[0][rr * C + cg * VW + e] = s1[e];
    red[1][rr * C + cg * VW + e] = s2[e];
  }
  __syncthreads();
  for (int c = tid; c < C; c += 256) {
    float a = 0.f, b = 0.f;
    for (int q = 0; q < rpi; ++q) {
      a += red[0][q * C + c];
      b += red[1][q * C + c];
    }
    part[((long)blockIdx.x * C + c) * 2 + 0] = a;
    part[((long)blockIdx.x * C + c) * 2 + 1] = b;
  }
}

__global__ __launch_bounds__(256) void bn_bwd_final_kernel(const float* __restrict__ part, int nblk, long M, int C,
                                                           const float* gamma, const float* rstd, float* dgamma,
                                                           float* dbeta, float* coef) {
  __shared__ double sh[256];
  const int c = blockIdx.x;
  double a = 0.0, b = 0.0;
  for (int q = threadIdx.x; q < nblk; q += 256) {
    a += part[((long)q * C + c) * 2 + 0];
    b += part[((long)q * C + c) * 2 + 1];
  }
  a = block_sum_d(a, sh);
  b = block_sum_d(b, sh);
  if (threadIdx.x == 0) {
    dbeta[c] = (float)a;
    dgamma[c] = (float)b;
    const double rs = (double)rstd[c];
    const double k1 = (double)gamma[c] * rs;
    coef[3 * c + 0] = (float)k1;
    coef[3 * c + 1] = (float)(-k1 * rs * b / (double)M);
    coef[3 * c + 2] = (float)(-k1 * a / (double)M);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void bn_bwd_apply_kernel(const T* __restrict__ dz, const uint8_t* __restrict__ mb,
                                                           const T* __restrict__ y, const float* __restrict__ mean,
                                                           const float* __restrict__ coef,
                                                           const float* __restrict__ mscale,
                                                           const float* __restrict__ mshift, T* __restrict__ dy,
                                                           long nchunks, int C) {
  constexpr int VW = TT<T>::VW;
  __shared__ float k1[kMaxC], k2[kMaxC], k3[kMaxC], mu[kMaxC], msc[kMaxC], msf[kMaxC];
  for (int c = threadIdx.x; c < C; c += 256) {
    k1[c] = coef[3 * c];
    k2[c] = coef[3 * c + 1];
    k3[c] = coef[3 * c + 2];
    mu[c] = mean[c];
    if (mscale) { msc[c] = mscale[c]; msf[c] = mshift[c]; }
  }
  __syncthreads();
  const int cpr = C / VW;
  for (long q = blockIdx.x * 256l + threadIdx.x; q < nchunks; q += (long)gridDim.x * 256) {
    const int c0 = (int)(q % cpr) * VW;
    float g[VW], yy[VW], o[VW];
    unpack<T>(((const uint4*)dz)[q], g);
    unpack<T>(((const uint4*)y)[q], yy);
    if (mb) {
      const uint32_t m = mb[q];
#pragma unroll
      for (int e = 0; e < VW; ++e) g[e] = (m >> e) & 1u ? g[e] : 0.f;
    } else if (mscale) {
#pragma unroll
      for (int e = 0; e < VW; ++e) g[e] = relu_stored<T>(yy[e], msc[c0 + e], msf[c0 + e]) > 0.f ? g[e] : 0.f;
    }
#pragma unroll
    for (int e = 0; e < VW; ++e) o[e] = k1[c0 + e] * g[e] + k2[c0 + e] * (yy[e] - mu[c0 + e]) + k3[c0 + e];
    ((uint4*)dy)[q] = pack<T>(o);
  }
}

// ---------------------------------------------------------------- stem + max pool
// The stem's BN-apply + ReLU feeds only the 3x3 stride-2 max pool, so the
// forward pass goes from the conv output y straight to the pooled tensor and
// its argmax; the ReLU output itself is never stored. The backward pass reads
// the pooled gradient and the argmax and gathers the gradient of each stem
// pixel on the fly (rounded to the storage type, as a stored tensor would be),
// with the ReLU mask recomputed from y by the same arithmetic.

template <typename T>
__global__ __launch_bounds__(256) void bn_apply_pool_kernel(const T* __restrict__ y, const float* __restrict__ scale,
                                                            const float* __restrict__ shift, T* __restrict__ pool,
                                                            uint8_t* __restrict__ arg, int N, int H, int W, int C,
                                                            int Ho, int Wo) {
  constexpr int VW = TT<T>::VW;
  __shared__ float sc[kMaxC], sf[kMaxC];
  for (int c = threadIdx.x; c < C; c += 256) { sc[c] = scale[c]; sf[c] = shift[c]; }
  __syncthreads();
  const int cpr = C / VW;
  const int total = N * Ho * Wo * cpr;
  for (int q = blockIdx.x * 256 + threadIdx.x; q < total; q += gridDim.x * 256) {
    const int pix = q / cpr, cc = q - pix * cpr;
    const int t2 = pix / Wo, j = pix - t2 * Wo;
    const int n = t2 / Ho, i = t2 - n * Ho;
    const int c0 = cc * VW;
    auto act = [&](float* v) {
#pragma unroll
      for (int e = 0; e < VW; ++e) v[e] = relu_stored<T>(v[e], sc[c0 + e], sf[c0 + e]);
    };
    float best[VW];
    uint8_t bi[VW];
    pool_max_window<T>(y, n, i, j, cc, H, W, C, act, best, bi);
    ((uint4*)pool)[q] = pack<T>(best);
    ArgVec<VW>::store(arg + (long)q * VW, bi);
  }
}

// Masked stem gradients of the pixels of quad (n, qi, qj), chunk cg: g[p][]
// (0 for pixels past the edge) and y[p][], p = 2*py + px.
template <typename T>
__device__ inline void stem_grad_quad(const T* __restrict__ dpool, const uint8_t* __restrict__ arg,
                                      const T* __restrict__ y, const float* sc, const float* sf, int n, int qi, int qj,
                                      int cg, int cpr, int H, int W, int Ho, int Wo, float (*g)[TT<T>::VW],
                                      float (*yy)[TT<T>::VW]) {
  constexpr int VW = TT<T>::VW;
  pool_grad_quad<T>(dpool, arg, n, qi, qj, cg, cpr, Ho, Wo, g);
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int h = 2 * qi + (p >> 1), w = 2 * qj + (p & 1);
    unpack<T>(((const uint4*)y)[((n * H + min(h, H - 1)) * W + min(w, W - 1)) * cpr + cg], yy[p]);
  }
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int h = 2 * qi + (p >> 1), w = 2 * qj + (p & 1);
    const bool in = h < H && w < W;
#pragma unroll
    for (int e = 0; e < VW; ++e) {
      const float gr = TT<T>::to_f(TT<T>::from_f(g[p][e]));
      const bool live = in && relu_stored<T>(yy[p][e], sc[cg * VW + e], sf[cg * VW + e]) > 0.f;
      g[p][e] = live ? gr : 0.f;
      yy[p][e] = in ? yy[p][e] : 0.f;
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void bn_bwd_partial_pool_kernel(const T* __restrict__ dpool,
                                                                  const uint8_t* __restrict__ arg,
                                                                  const T* __restrict__ y,
                                                                  const float* __restrict__ scale,
                                                                  const float* __restrict__ shift,
                                                                  const float* __restrict__ mean,
                                                                  const float* __restrict__ rstd, int N, int H, int W,
                                                                  int C, int Ho, int Wo, float* __restrict__ part) {
  constexpr int VW = TT<T>::VW;
  __shared__ float red[2][256 * VW];
  __shared__ float sc[kMaxC], sf[kMaxC];
  for (int c = threadIdx.x; c < C; c += 256) { sc[c] = scale[c]; sf[c] = shift[c]; }
  __syncthreads();
  const int Hq = (H + 1) / 2, Wq = (W + 1) / 2;
  const int Mq = N * Hq * Wq;
  const int tpc = C / VW, rpi = 256 / tpc;
  const int tid = threadIdx.x, cg = tid % tpc, rr = tid / tpc;
  const int per_blk = (Mq + gridDim.x - 1) / gridDim.x;
  const int q_begin = blockIdx.x * per_blk;
  const int q_end = min(Mq, q_begin + per_blk);
  float mu[VW], rs[VW], s1[VW], s2[VW];
#pragma unroll
  for (int e = 0; e < VW; ++e) {
    mu[e] = mean[cg * VW + e];
    rs[e] = rstd[cg * VW + e];
    s1[e] = s2[e] = 0.f;
  }
  for (int q = q_begin + rr; q < q_end; q += rpi) {
    const int t2 = q / Wq, qj = q - t2 * Wq;
    const int n = t2 / Hq, qi = t2 - n * Hq;
    float g[4][VW], yy[4][VW];
    stem_grad_quad<T>(dpool, arg, y, sc, sf, n, qi, qj, cg, tpc, H, W, Ho, Wo, g, yy);
#pragma unroll
    for (int p = 0; p < 4; ++p)
#pragma unroll
      for (int e = 0; e < VW; ++e) {
        s1[e] += g[p][e];
        s2[e] += g[p][e] * ((yy[p][e] - mu[e]) * rs[e]);
      }
  }
#pragma unroll
  for (int e = 0; e < VW; ++e) {
    red[0][rr * C + cg * VW + e] = s1[e];
    red[1][rr * C + cg * VW + e] = s2[e];
  }
  __syncthreads();
  for (int c = tid; c < C; c += 256) {
    float a = 0.f, b = 0.f;
    for (int q = 0; q < rpi; ++q) {
      a += red[0][q * C + c];
      b += red[1][q * C + c];
    }
    part[((long)blockIdx.x * C + c) * 2 + 0] = a;
    part[((long)blockIdx.x * C + c) * 2 + 1] = b;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void bn_bwd_apply_pool_kernel(const T* __restrict__ dpool,
                                                                const uint8_t* __restrict__ arg,
                                                                const T* __restrict__ y,
                                                                const float* __restrict__ scale,
                                                                const float* __restrict__ shift,
                                                                const float* __restrict__ mean,
                                                                const float* __restrict__ coef, T* __restrict__ dy,
                                                                int N, int H, int W, int C, int Ho, int Wo) {
  constexpr int VW = TT<T>::VW;
  __shared__ float k1[kMaxC], k2[kMaxC], k3[kMaxC], mu[kMaxC], sc[kMaxC], sf[kMaxC];
  for (int c = threadIdx.x; c < C; c += 256) {
    k1[c] = coef[3 * c];
    k2[c] = coef[3 * c + 1];
    k3[c] = coef[3 * c + 2];
    mu[c] = mean[c];
    sc[c] = scale[c];
    sf[c] = shift[c];
  }
  __syncthreads();
  const int cpr = C / VW;
  const int Hq = (H + 1) / 2, Wq = (W + 1) / 2;
  const int nq = N * Hq * Wq * cpr;
  for (int q = blockIdx.x * 256 + threadIdx.x; q < nq; q += gridDim.x * 256) {
    const int quad = q / cpr, cg = q - quad * cpr;
    const int t2 = quad / Wq, qj = quad - t2 * Wq;
    const int n = t2 / Hq, qi = t2 - n * Hq;
    const int c0 = cg * VW;
    float g[4][VW], yy[4][VW];
    stem_grad_quad<T>(dpool, arg, y, sc, sf, n, qi, qj, cg, cpr, H, W, Ho, Wo, g, yy);
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int h = 2 * qi + (p >> 1), w = 2 * qj + (p & 1);
      if (h >= H || w >= W) continue;
      float o[VW];
#pragma unroll
      for (int e = 0; e < VW; ++e) o[e] = k1[c0 + e] * g[p][e] + k2[c0 + e] * (yy[p][e] - mu[c0 + e]) + k3[c0 + e];
      ((uint4*)dy)[((n * H + h) * W + w) * cpr + cg] = pack<T>(o);
    }
  }
}

int stream_blocks(long nchunks) {
  long b = (nchunks + 255) / 256;
  if (b > 8192) b = 8192;
  if (b < 1) b = 1;
  return (int)b;
}

inline int ok() { return hipGetLastError() == hipSuccess ? 0 : -4; }

}  // namespace

int bn_apply_launch(int prec, const void* y, const float* scale, const float* shift, int relu, int res_mode,
                    const void* r, const float* scale2, const float* shift2, void* z, long M, int C, hipStream_t s,
                    uint8_t* mbits) {
  const long nchunks = M * C / prec_vw(prec);
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(bn_apply_kernel<T>, dim3(stream_blocks(nchunks)), dim3(256), 0, s, (const T*)y, scale, shift,
                       relu, res_mode, (const T*)r, scale2, shift2, (T*)z, nchunks, C, mbits);
    return ok();
  });
}

int bn_eval_coef_launch(const float* gamma, const float* beta, const float* rm, const float* rv, float eps, int C,
                        float* scale, float* shift, hipStream_t s) {
  hipLaunchKernelGGL(bn_eval_coef_kernel, dim3((C + 255) / 256), dim3(256), 0, s, gamma, beta, rm, rv, eps, C, scale,
                     shift);
  return ok();
}

int bn_bwd_partial_blocks(int prec, long M, int C) {
  return pick_blocks(M, 256 / (C / prec_vw(prec)), 16, 512, 256);
}

int bn_bwd_partial_pool_blocks(int prec, int N, int H, int W, int C) {
  const int rpi = 256 / (C / prec_vw(prec));
  return pick_blocks((long)N * ((H + 1) / 2) * ((W + 1) / 2), rpi, 8, 1024, 0);
}

int bn_bwd_partial_launch(int prec, const void* dz, const uint8_t* mb, const void* y, const float* mean,
                          const float* rstd, long M, int C, float* part, int* nblk, hipStream_t s,
                          const float* mscale, const float* mshift) {
  const int nb = bn_bwd_partial_blocks(prec, M, C);
  *nblk = nb;
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(bn_bwd_partial_kernel<T>, dim3(nb), dim3(256), 0, s, (const T*)dz, mb, (const T*)y, mean, rstd,
                       mscale, mshift, M, C, part);
    return ok();
  });
}

int bn_bwd_final_launch(const float* part, int nblk, long M, int C, const float* gamma, const float* rstd,
                        float* dgamma, float* dbeta, float* coef, hipStream_t s) {
  hipLaunchKernelGGL(bn_bwd_final_kernel, dim3(C), dim3(256), 0, s, part, nblk, M, C, gamma, rstd, dgamma, dbeta,
                     coef);
  return ok();
}

int bn_bwd_apply_launch(int prec, const void* dz, const uint8_t* mb, const void* y, const float* mean, const float* coef,
                        void* dy, long M, int C, hipStream_t s, const float* mscale, const float* mshift,
                        hipEvent_t done) {
  const long nchunks = M * C / prec_vw(prec);
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    if (done) {
      // the event completes with this kernel: no separate marker on the queue
      hipExtLaunchKernelGGL(bn_bwd_apply_kernel<T>, dim3(stream_blocks(nchunks)), dim3(256), 0, s, nullptr, done, 0,
                            (const T*)dz, mb, (const T*)y, mean, coef, mscale, mshift, (T*)dy, nchunks, C);
    } else {
      hipLaunchKernelGGL(bn_bwd_apply_kernel<T>, dim3(stream_blocks(nchunks)), dim3(256), 0, s, (const T*)dz, mb,
                         (const T*)y, mean, coef, mscale, mshift, (T*)dy, nchunks, C);
    }
    return ok();
  });
}

int bn_apply_pool_launch(int prec, const void* y, const float* scale, const float* shift, void* pool, uint8_t* arg,
                         int N, int H, int W, int C, int Ho, int Wo, hipStream_t s) {
  const int vw = prec_vw(prec);
  if (C > kMaxC || (long)N * H * W * (C / vw) >= (1l << 31)) return -1;  // 32-bit chunk indices
  const long total = (long)N * Ho * Wo * (C / vw);
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(bn_apply_pool_kernel<T>, dim3(stream_blocks(total)), dim3(256), 0, s, (const T*)y, scale, shift,
                       (T*)pool, arg, N, H, W, C, Ho, Wo);
    return ok();
  });
}

int bn_bwd_partial_pool_launch(int prec, const void* dpool, const uint8_t* arg, const void* y, const float* scale,
                               const float* shift, const float* mean, const float* rstd, int N, int H, int W, int C,
                               int Ho, int Wo, float* part, int* nblk, hipStream_t s) {
  const int vw = prec_vw(prec);
  if (C > kMaxC || (long)N * H * W * (C / vw) >= (1l << 31)) return -1;  // 32-bit chunk indices
  const int nb = bn_bwd_partial_pool_blocks(prec, N, H, W, C);
  *nblk = nb;
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(bn_bwd_partial_pool_kernel<T>, dim3(nb), dim3(256), 0, s, (const T*)dpool, arg, (const T*)y,
                       scale, shift, mean, rstd, N, H, W, C, Ho, Wo, part);
    return ok();
  });
}

int bn_bwd_apply_pool_launch(int prec, const void* dpool, const uint8_t* arg, const void* y, const float* scale,
                             const float* shift, const float* mean, const float* coef, void* dy, int N, int H, int W,
                             int C, int Ho, int Wo, hipStream_t s) {
  const int vw = prec_vw(prec);
  if (C > kMaxC || (long)N * H * W * (C / vw) >= (1l << 31)) return -1;  // 32-bit chunk indices
  const long nchunks = (long)N * ((H + 1) / 2) * ((W + 1) / 2) * (C / vw);
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(bn_bwd_apply_pool_kernel<T>, dim3(stream_blocks(nchunks)), dim3(256), 0, s, (const T*)dpool,
                       arg, (const T*)y, scale, shift, mean, coef, (T*)dy, N, H, W, C, Ho, Wo);
    return ok();
  });
}

int bn_stats_tiles_chunks(int ntiles) {
  int r = (ntiles + 63) / 64;
  return r < 1 ? 1 : r > 64 ? 64 : r;
}

int bn_stats_tiles_final_launch(const float* tile_stats, int ntiles, int C, double* scratch, const float* gamma,
                                const float* beta, float eps, float momentum, float* run_mean, float* run_var,
                                float* mean, float* rstd, float* scale, float* shift, hipStream_t s) {
  const int chunks = bn_stats_tiles_chunks(ntiles);
  const int per_chunk = (ntiles + chunks - 1) / chunks;
  const BnStatsOut o{gamma, beta, eps, momentum, run_mean, run_var, mean, rstd, scale, shift};
  hipLaunchKernelGGL(bn_stats_tiles_reduce_kernel, dim3((C + 63) / 64, chunks), dim3(256), 0, s, tile_stats, ntiles,
                     C, per_chunk, scratch, o);
  if (chunks > 1)
    hipLaunchKernelGGL(bn_stats_tiles_final_kernel, dim3((C + 63) / 64), dim3(256), 0, s, tile_stats, scratch, chunks,
                       C, o);
  return ok();
}

}  // namespace rn18
