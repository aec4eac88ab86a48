// Batch normalisation (training mode) over an NHWC tensor viewed as [M][C]:
// statistics per channel over all M = N*H*W rows.
//
// Statistics are two-level and deterministic: each block reduces a contiguous
// range of rows to per-channel partial sums in fp32 (16-byte row chunks read
// coalesced, then a fixed-order LDS reduction), and a finalize kernel combines
// the block partials in fp64. The forward sums are taken of (y - y[0][c]):
// shifting by a sample of the channel keeps Sum(v^2) - (Sum v)^2/M well
// conditioned when |mean| >> std.
//
// The elementwise passes (apply + ReLU + residual, backward apply) are 16-byte
// HBM streams with the per-channel coefficients staged in LDS.
#include "kernels.h"

namespace rn18 {

namespace {

constexpr int kMaxC = 512;

int pick_blocks(long M, int rows_per_iter) {
  long b = M / ((long)rows_per_iter * 8);  // >= 8 rows per thread
  if (b > 1024) b = 1024;
  if (b < 1) b = 1;
  return (int)b;
}

template <typename T>
__global__ __launch_bounds__(256) void bn_stats_partial_kernel(const T* __restrict__ y, long M, int C,
                                                               float* __restrict__ part) {
  constexpr int VW = TT<T>::VW;
  __shared__ float red[2][256 * VW];
  const int tpc = C / VW, rpi = 256 / tpc;
  const int tid = threadIdx.x, cg = tid % tpc, rr = tid / tpc;
  const long rows_per_blk = (M + gridDim.x - 1) / gridDim.x;
  const long r_begin = blockIdx.x * rows_per_blk;
  const long r_end = min(M, r_begin + rows_per_blk);
  float piv[VW], s1[VW], s2[VW];
  unpack<T>(*(const uint4*)(y + cg * VW), piv);
#pragma unroll
  for (int e = 0; e < VW; ++e) s1[e] = s2[e] = 0.f;
  for (long r = r_begin + rr; r < r_end; r += rpi) {
    float v[VW];
    unpack<T>(*(const uint4*)(y + r * C + cg * VW), v);
#pragma unroll
    for (int e = 0; e < VW; ++e) {
      const float d = v[e] - piv[e];
      s1[e] += d;
      s2[e] += d * d;
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

template <typename T>
__global__ __launch_bounds__(256) void bn_stats_final_kernel(const T* __restrict__ y, const float* __restrict__ part,
                                                             int nblk, long M, int C, const float* gamma,
                                                             const float* beta, float eps, float mom, float* rm,
                                                             float* rv, float* mean_o, float* rstd_o,
                                                             float* scale_o, float* shift_o) {
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
    const double piv = (double)TT<T>::to_f(y[c]);
    const double md = a / (double)M;
    double var = b / (double)M - md * md;
    if (var < 0.0) var = 0.0;
    const double mean = piv + md;
    const double rstd = 1.0 / sqrt(var + (double)eps);
    const double sc = (double)gamma[c] * rstd;
    mean_o[c] = (float)mean;
    rstd_o[c] = (float)rstd;
    scale_o[c] = (float)sc;
    shift_o[c] = (float)((double)beta[c] - mean * sc);
    if (rm) {
      rm[c] = (float)((1.0 - mom) * (double)rm[c] + mom * mean);
      rv[c] = (float)((1.0 - mom) * (double)rv[c] + mom * var * ((double)M / (double)(M - 1)));
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void bn_apply_kernel(const T* __restrict__ y, const float* __restrict__ scale,
                                                       const float* __restrict__ shift, int relu, int res_mode,
                                                       const T* __restrict__ r, const float* __restrict__ scale2,
                                                       const float* __restrict__ shift2, T* __restrict__ z,
                                                       long nchunks, int C) {
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
    for (int e = 0; e < VW; ++e) v[e] = v[e] * sc[c0 + e] + sf[c0 + e];
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
    ((uint4*)z)[q] = pack<T>(v);
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
__global__ __launch_bounds__(256) void bn_bwd_partial_kernel(const T* __restrict__ dz, const T* __restrict__ mz,
                                                             const T* __restrict__ y, const float* __restrict__ mean,
                                                             const float* __restrict__ rstd, long M, int C,
                                                             float* __restrict__ part) {
  constexpr int VW = TT<T>::VW;
  __shared__ float red[2][256 * VW];
  const int tpc = C / VW, rpi = 256 / tpc;
  const int tid = threadIdx.x, cg = tid % tpc, rr = tid / tpc;
  const long rows_per_blk = (M + gridDim.x - 1) / gridDim.x;
  const long r_begin = blockIdx.x * rows_per_blk;
  const long r_end = min(M, r_begin + rows_per_blk);
  float mu[VW], rs[VW], s1[VW], s2[VW];
#pragma unroll
  for (int e = 0; e < VW; ++e) {
    mu[e] = mean[cg * VW + e];
    rs[e] = rstd[cg * VW + e];
    s1[e] = s2[e] = 0.f;
  }
  for (long r = r_begin + rr; r < r_end; r += rpi) {
    const long o = r * C + cg * VW;
    float g[VW], yy[VW];
    unpack<T>(*(const uint4*)(dz + o), g);
    unpack<T>(*(const uint4*)(y + o), yy);
    if (mz) {
      float m[VW];
      unpack<T>(*(const uint4*)(mz + o), m);
#pragma unroll
      for (int e = 0; e < VW; ++e) g[e] = m[e] > 0.f ? g[e] : 0.f;
    }
#pragma unroll
    for (int e = 0; e < VW; ++e) {
      s1[e] += g[e];
      s2[e] += g[e] * ((yy[e] - mu[e]) * rs[e]);
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
__global__ __launch_bounds__(256) void bn_bwd_apply_kernel(const T* __restrict__ dz, const T* __restrict__ mz,
                                                           const T* __restrict__ y, const float* __restrict__ mean,
                                                           const float* __restrict__ coef, T* __restrict__ dy,
                                                           long nchunks, int C) {
  constexpr int VW = TT<T>::VW;
  __shared__ float k1[kMaxC], k2[kMaxC], k3[kMaxC], mu[kMaxC];
  for (int c = threadIdx.x; c < C; c += 256) {
    k1[c] = coef[3 * c];
    k2[c] = coef[3 * c + 1];
    k3[c] = coef[3 * c + 2];
    mu[c] = mean[c];
  }
  __syncthreads();
  const int cpr = C / VW;
  for (long q = blockIdx.x * 256l + threadIdx.x; q < nchunks; q += (long)gridDim.x * 256) {
    const int c0 = (int)(q % cpr) * VW;
    float g[VW], yy[VW], o[VW];
    unpack<T>(((const uint4*)dz)[q], g);
    unpack<T>(((const uint4*)y)[q], yy);
    if (mz) {
      float m[VW];
      unpack<T>(((const uint4*)mz)[q], m);
#pragma unroll
      for (int e = 0; e < VW; ++e) g[e] = m[e] > 0.f ? g[e] : 0.f;
    }
#pragma unroll
    for (int e = 0; e < VW; ++e) o[e] = k1[c0 + e] * g[e] + k2[c0 + e] * (yy[e] - mu[c0 + e]) + k3[c0 + e];
    ((uint4*)dy)[q] = pack<T>(o);
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

int bn_stats_partial_launch(int prec, const void* y, long M, int C, float* part, int* nblk, hipStream_t s) {
  const int vw = prec == PREC_BF16 ? 8 : 4;
  const int rpi = 256 / (C / vw);
  const int nb = pick_blocks(M, rpi);
  *nblk = nb;
  if (prec == PREC_BF16)
    hipLaunchKernelGGL(bn_stats_partial_kernel<bf16_t>, dim3(nb), dim3(256), 0, s, (const bf16_t*)y, M, C, part);
  else
    hipLaunchKernelGGL(bn_stats_partial_kernel<float>, dim3(nb), dim3(256), 0, s, (const float*)y, M, C, part);
  return ok();
}

int bn_stats_final_launch(int prec, const void* y, const float* part, int nblk, long M, int C, const float* gamma,
                          const float* beta, float eps, float momentum, float* run_mean, float* run_var,
                          float* mean, float* rstd, float* scale, float* shift, hipStream_t s) {
  if (prec == PREC_BF16)
    hipLaunchKernelGGL(bn_stats_final_kernel<bf16_t>, dim3(C), dim3(256), 0, s, (const bf16_t*)y, part, nblk, M, C,
                       gamma, beta, eps, momentum, run_mean, run_var, mean, rstd, scale, shift);
  else
    hipLaunchKernelGGL(bn_stats_final_kernel<float>, dim3(C), dim3(256), 0, s, (const float*)y, part, nblk, M, C,
                       gamma, beta, eps, momentum, run_mean, run_var, mean, rstd, scale, shift);
  return ok();
}

int bn_apply_launch(int prec, const void* y, const float* scale, const float* shift, int relu, int res_mode,
                    const void* r, const float* scale2, const float* shift2, void* z, long M, int C, hipStream_t s) {
  const int vw = prec == PREC_BF16 ? 8 : 4;
  const long nchunks = M * C / vw;
  if (prec == PREC_BF16)
    hipLaunchKernelGGL(bn_apply_kernel<bf16_t>, dim3(stream_blocks(nchunks)), dim3(256), 0, s, (const bf16_t*)y,
                       scale, shift, relu, res_mode, (const bf16_t*)r, scale2, shift2, (bf16_t*)z, nchunks, C);
  else
    hipLaunchKernelGGL(bn_apply_kernel<float>, dim3(stream_blocks(nchunks)), dim3(256), 0, s, (const float*)y, scale,
                       shift, relu, res_mode, (const float*)r, scale2, shift2, (float*)z, nchunks, C);
  return ok();
}

int bn_eval_coef_launch(const float* gamma, const float* beta, const float* rm, const float* rv, float eps, int C,
                        float* scale, float* shift, hipStream_t s) {
  hipLaunchKernelGGL(bn_eval_coef_kernel, dim3((C + 255) / 256), dim3(256), 0, s, gamma, beta, rm, rv, eps, C, scale,
                     shift);
  return ok();
}

int bn_bwd_partial_launch(int prec, const void* dz, const void* mz, const void* y, const float* mean,
                          const float* rstd, long M, int C, float* part, int* nblk, hipStream_t s) {
  const int vw = prec == PREC_BF16 ? 8 : 4;
  const int rpi = 256 / (C / vw);
  const int nb = pick_blocks(M, rpi);
  *nblk = nb;
  if (prec == PREC_BF16)
    hipLaunchKernelGGL(bn_bwd_partial_kernel<bf16_t>, dim3(nb), dim3(256), 0, s, (const bf16_t*)dz,
                       (const bf16_t*)mz, (const bf16_t*)y, mean, rstd, M, C, part);
  else
    hipLaunchKernelGGL(bn_bwd_partial_kernel<float>, dim3(nb), dim3(256), 0, s, (const float*)dz, (const float*)mz,
                       (const float*)y, mean, rstd, M, C, part);
  return ok();
}

int bn_bwd_final_launch(const float* part, int nblk, long M, int C, const float* gamma, const float* rstd,
                        float* dgamma, float* dbeta, float* coef, hipStream_t s) {
  hipLaunchKernelGGL(bn_bwd_final_kernel, dim3(C), dim3(256), 0, s, part, nblk, M, C, gamma, rstd, dgamma, dbeta,
                     coef);
  return ok();
}

int bn_bwd_apply_launch(int prec, const void* dz, const void* mz, const void* y, const float* mean, const float* coef,
                        void* dy, long M, int C, hipStream_t s) {
  const int vw = prec == PREC_BF16 ? 8 : 4;
  const long nchunks = M * C / vw;
  if (prec == PREC_BF16)
    hipLaunchKernelGGL(bn_bwd_apply_kernel<bf16_t>, dim3(stream_blocks(nchunks)), dim3(256), 0, s,
                       (const bf16_t*)dz, (const bf16_t*)mz, (const bf16_t*)y, mean, coef, (bf16_t*)dy, nchunks, C);
  else
    hipLaunchKernelGGL(bn_bwd_apply_kernel<float>, dim3(stream_blocks(nchunks)), dim3(256), 0, s, (const float*)dz,
                       (const float*)mz, (const float*)y, mean, coef, (float*)dy, nchunks, C);
  return ok();
}

}  // namespace rn18
