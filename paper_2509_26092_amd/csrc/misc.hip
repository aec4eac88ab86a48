// Streams and small kernels of the training step: input ingest (NCHW fp32 ->
// NHWC with channels padded to the 16-byte vector), weight repack (OIHW fp32
// master -> forward and data-gradient layouts in the compute type), max pool
// with first-maximum argmax and its gather-form backward, global average pool,
// an LDS-tiled fp32 GEMM for the classifier, softmax cross-entropy with a
// deterministic loss reduction, SGD-momentum, and the parameter-server merge.
#include <math.h>

#include "kernels.h"
#include "pool.h"

namespace rn18 {

namespace {

inline int ok() { return hipGetLastError() == hipSuccess ? 0 : -4; }

int grid_for(long work, int per_block = 256, int cap = 16384) {
  long b = (work + per_block - 1) / per_block;
  if (b > cap) b = cap;
  if (b < 1) b = 1;
  return (int)b;
}

// ------------------------------------------------------------------ ingest
// A non-finite image value sets the sticky DEVERR_NONFINITE flag (a NaN
// could otherwise vanish in a ReLU and leave a finite loss).
template <typename T>
__global__ void ingest_kernel(const float* __restrict__ img, T* __restrict__ x, long npix, int HW, int Cp,
                              unsigned* err) {
  for (long p = blockIdx.x * 256l + threadIdx.x; p < npix; p += (long)gridDim.x * 256) {
    const long n = p / HW, hw = p - n * HW;
    const float* src = img + n * 3 * HW + hw;
    float v[8] = {src[0], src[HW], src[2 * HW], 0.f, 0.f, 0.f, 0.f, 0.f};
    if (!(__builtin_isfinite(v[0]) && __builtin_isfinite(v[1]) && __builtin_isfinite(v[2])))
      atomicOr(err, (unsigned)DEVERR_NONFINITE);
    ((uint4*)x)[p] = pack<T>(v);  // Cp elements = exactly 16 bytes
  }
}

template <typename T>
__global__ void ingest_s2d_kernel(const float* __restrict__ img, T* __restrict__ x, long npix, int H, int W,
                                  unsigned* err) {
  constexpr int VW = TT<T>::VW;
  const int Hs = H / 2, Ws = W / 2;
  const long HW = (long)H * W;
  for (long p = blockIdx.x * 256l + threadIdx.x; p < npix; p += (long)gridDim.x * 256) {
    const long n = p / ((long)Hs * Ws);
    const int r = (int)(p - n * Hs * Ws);
    const int i = r / Ws, j = r - i * Ws;
    const float* src = img + n * 3 * HW + (long)(2 * i) * W + 2 * j;
    float v[16];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int c = 0; c < 3; ++c) v[q * 3 + c] = src[c * HW + (q >> 1) * W + (q & 1)];
    bool fin = true;
#pragma unroll
    for (int c = 0; c < 12; ++c) fin = fin && __builtin_isfinite(v[c]);
    if (!fin) atomicOr(err, (unsigned)DEVERR_NONFINITE);
#pragma unroll
    for (int c = 12; c < 16; ++c) v[c] = 0.f;
#pragma unroll
    for (int q = 0; q < 16 / VW; ++q) ((uint4*)x)[p * (16 / VW) + q] = pack<T>(v + q * VW);
  }
}

// ------------------------------------------------------------------ repack
template <typename T>
__global__ void repack_kernel(const float* __restrict__ st, T* __restrict__ wf, T* __restrict__ wd,
                              const RepackEntry* __restrict__ tab, int nent, long total) {
  __shared__ RepackEntry t[24];
  for (int i = threadIdx.x; i < nent; i += blockDim.x) t[i] = tab[i];
  __syncthreads();
  for (long e = blockIdx.x * 256l + threadIdx.x; e < total; e += (long)gridDim.x * 256) {
    int k = 0;
    while (k + 1 < nent && e >= t[k + 1].nprefix) ++k;
    const RepackEntry& r = t[k];
    const long l = e - r.nprefix;
    const int per_co = r.KHW * r.Cin_p;
    const int co = (int)(l / per_co);
    const int rem = (int)(l - (long)co * per_co);
    const int tap = rem / r.Cin_p, ci = rem - tap * r.Cin_p;
    float v = 0.f;
    if (r.mode == 1) {
      // 4x4 tap (a, b), channel (2*dy + dx)*3 + c  <-  7x7 tap (2a+dy-1, 2b+dx-1) of channel c
      if (ci < 12) {
        const int q = ci / 3, c = ci - 3 * q;
        const int kh = 2 * (tap >> 2) + (q >> 1) - 1, kw = 2 * (tap & 3) + (q & 1) - 1;
        if (kh >= 0 && kw >= 0) v = st[r.src + (((long)co * 3 + c) * 7 + kh) * 7 + kw];
      }
    } else if (ci < r.Cin) {
      v = st[r.src + ((long)co * r.Cin + ci) * r.KHW + tap];
    }
    const T tv = TT<T>::from_f(v);
    wf[r.dst_f + l] = tv;
    if (r.dst_d >= 0) wd[r.dst_d + ((long)ci * r.KHW + tap) * r.Cout + co] = tv;
  }
}

// Weight shadows of the 3x3 and 1x1 convs through LDS, one block per tile of
// 32 output x 32 input channels with all its taps: the fp32 weights
// [Cout][Cin][KHW] are read in contiguous rows, and both layouts are written
// in runs of consecutive channels. Entry fields: n = tiles of the conv,
// nprefix = tiles before it.
constexpr int kRepackT = 32, kRepackMaxKHW = 9;
template <typename T>
__global__ __launch_bounds__(256) void repack_tiled_kernel(const float* __restrict__ st, T* __restrict__ wf,
                                                           T* __restrict__ wd, const RepackEntry* __restrict__ tab,
                                                           int nent) {
  __shared__ RepackEntry t[24];
  __shared__ float s[kRepackT * (kRepackT * kRepackMaxKHW + 1)];
  for (int i = threadIdx.x; i < nent; i += blockDim.x) t[i] = tab[i];
  __syncthreads();
  int k = 0;
  while (k + 1 < nent && (long)blockIdx.x >= t[k + 1].nprefix) ++k;
  const RepackEntry& r = t[k];
  const int KHW = r.KHW, Cin = r.Cin, Cin_p = r.Cin_p, Cout = r.Cout;
  const int ntci = (Cin_p + kRepackT - 1) / kRepackT;
  const int l = (int)(blockIdx.x - r.nprefix);
  const int co0 = (l / ntci) * kRepackT, ci0 = (l % ntci) * kRepackT;
  const int nco = min(kRepackT, Cout - co0), nci = min(kRepackT, Cin_p - ci0);
  const int row = nci * KHW, RS = kRepackT * KHW + 1;   // odd row stride: no bank conflicts across rows
  const int valid = (Cin - ci0) * KHW;                  // row entries with a real input channel
  // twelve loads in flight per thread before any is stored
  constexpr int U = 12;
  const int nld = nco * row;
  for (int b = threadIdx.x; b < nld; b += 256 * U) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int idx = b + u * 256, co = idx / row, j = idx - co * row;
      v[u] = idx < nld && j < valid ? st[r.src + ((long)(co0 + co) * Cin + ci0) * KHW + j] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int idx = b + u * 256, co = idx / row, j = idx - co * row;
      if (idx < nld) s[co * RS + j] = v[u];
    }
  }
  __syncthreads();
  // Both layouts are written in 16-byte runs (VS consecutive channels per
  // thread): channel counts are multiples of the vector width and every
  // layout offset is a multiple of its run length.
  constexpr int VS = TT<T>::VW;
  // forward layout [Cout][KHW][Cin_p]: consecutive input channels
  const int nciv = nci / VS;
  for (int idx = threadIdx.x; idx < nco * KHW * nciv; idx += 256) {
    const int cv = idx % nciv, rest = idx / nciv, tap = rest % KHW, co = rest / KHW;
    float v[VS];
#pragma unroll
    for (int e = 0; e < VS; ++e) v[e] = s[co * RS + (cv * VS + e) * KHW + tap];
    *(uint4*)(wf + r.dst_f + ((long)(co0 + co) * KHW + tap) * Cin_p + ci0 + cv * VS) = pack<T>(v);
  }
  // data-gradient layout [Cin_p][KHW][Cout]: consecutive output channels
  if (r.dst_d >= 0) {
    const int ncov = nco / VS;
    for (int idx = threadIdx.x; idx < nci * KHW * ncov; idx += 256) {
      const int cv = idx % ncov, rest = idx / ncov, tap = rest % KHW, ci = rest / KHW;
      float v[VS];
#pragma unroll
      for (int e = 0; e < VS; ++e) v[e] = s[(cv * VS + e) * RS + ci * KHW + tap];
      *(uint4*)(wd + r.dst_d + ((long)(ci0 + ci) * KHW + tap) * Cout + co0 + cv * VS) = pack<T>(v);
    }
  }
}

// ------------------------------------------------------------------ dropout
// Philox4x32-10 (Salmon et al., SC'11): ten rounds of two 32x32 -> 64-bit
// products mixed with the other counter words and the key, the key bumped by
// the Weyl constants between rounds.
__device__ inline void philox4x32_10(uint32_t (&c)[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0], p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0, n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = (uint32_t)p1;
    c[2] = n2;
    c[3] = (uint32_t)p0;
  }
}

// In-place dropout of n fp32 values, four per counter: group q draws one
// Philox output (counter (q, step), key seed); value 4q + w is kept iff the
// top 24 bits of word w are >= thresh, and kept values are scaled. A ragged
// last group (n not a multiple of 4) uses the leading words of its output.
__global__ void dropout_kernel(float* __restrict__ x, long n, uint32_t k0, uint32_t k1, uint32_t s0, uint32_t s1,
                               uint32_t thresh, float scale) {
  const long n4 = (n + 3) / 4;
  for (long q = blockIdx.x * (long)blockDim.x + threadIdx.x; q < n4; q += (long)gridDim.x * blockDim.x) {
    uint32_t c[4] = {(uint32_t)q, (uint32_t)(q >> 32), s0, s1};
    philox4x32_10(c, k0, k1);
    if (4 * q + 4 <= n) {
      float4 v = ((float4*)x)[q];
      v.x = (c[0] >> 8) >= thresh ? v.x * scale : 0.f;
      v.y = (c[1] >> 8) >= thresh ? v.y * scale : 0.f;
      v.z = (c[2] >> 8) >= thresh ? v.z * scale : 0.f;
      v.w = (c[3] >> 8) >= thresh ? v.w * scale : 0.f;
      ((float4*)x)[q] = v;
    } else {
      for (int w = 0; w < 4 && 4 * q + w < n; ++w) x[4 * q + w] = (c[w] >> 8) >= thresh ? x[4 * q + w] * scale : 0.f;
    }
  }
}

// ------------------------------------------------------------------ max pool 3x3 s2 p1
template <typename T>
__global__ void maxpool_fwd_kernel(const T* __restrict__ x, T* __restrict__ y, uint8_t* __restrict__ arg, int N,
                                   int H, int W, int C, int Ho, int Wo) {
  constexpr int VW = TT<T>::VW;
  const int cpr = C / VW;
  const int total = N * Ho * Wo * cpr;
  for (int q = blockIdx.x * 256 + threadIdx.x; q < total; q += gridDim.x * 256) {
    const int pix = q / cpr, cc = q - pix * cpr;
    const int t2 = pix / Wo, j = pix - t2 * Wo;
    const int n = t2 / Ho, i = t2 - n * Ho;
    float best[VW];
    uint8_t bi[VW];
    pool_max_window<T>(x, n, i, j, cc, H, W, C, [](float*) {}, best, bi);
    ((uint4*)y)[q] = pack<T>(best);
    ArgVec<VW>::store(arg + (long)q * VW, bi);
  }
}

// Gather form over 2x2 quads of input pixels (deterministic: no atomics).
template <typename T>
__global__ void maxpool_bwd_kernel(const T* __restrict__ dy, const uint8_t* __restrict__ arg, T* __restrict__ dx,
                                   int N, int H, int W, int C, int Ho, int Wo) {
  constexpr int VW = TT<T>::VW;
  const int cpr = C / VW;
  const int Hq = (H + 1) / 2, Wq = (W + 1) / 2;
  const int total = N * Hq * Wq * cpr;
  for (int q = blockIdx.x * 256 + threadIdx.x; q < total; q += gridDim.x * 256) {
    const int quad = q / cpr, cc = q - quad * cpr;
    const int t2 = quad / Wq, qj = quad - t2 * Wq;
    const int n = t2 / Hq, qi = t2 - n * Hq;
    float acc[4][VW];
    pool_grad_quad<T>(dy, arg, n, qi, qj, cc, cpr, Ho, Wo, acc);
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int h = 2 * qi + (p >> 1), w = 2 * qj + (p & 1);
      if (h < H && w < W) ((uint4*)dx)[((n * H + h) * W + w) * cpr + cc] = pack<T>(acc[p]);
    }
  }
}

// ------------------------------------------------------------------ avg pool
template <typename T>
__global__ void avgpool_fwd_kernel(const T* __restrict__ x, float* __restrict__ f, int N, int HW, int C) {
  constexpr int VW = TT<T>::VW;
  const int cpr = C / VW;
  const long total = (long)N * cpr;
  for (long q = blockIdx.x * 256l + threadIdx.x; q < total; q += (long)gridDim.x * 256) {
    const int cc = (int)(q % cpr);
    const long n = q / cpr;
    float s[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) s[e] = 0.f;
    for (int p = 0; p < HW; ++p) {
      float v[VW];
      unpack<T>(*(const uint4*)(x + (n * HW + p) * C + cc * VW), v);
#pragma unroll
      for (int e = 0; e < VW; ++e) s[e] += v[e];
    }
    const float inv = 1.0f / (float)HW;
#pragma unroll
    for (int e = 0; e < VW; ++e) f[n * C + cc * VW + e] = s[e] * inv;
  }
}

template <typename T>
__global__ void avgpool_bwd_kernel(const float* __restrict__ df, T* __restrict__ dx, int N, int HW, int C) {
  constexpr int VW = TT<T>::VW;
  const int cpr = C / VW;
  const long total = (long)N * HW * cpr;
  const float inv = 1.0f / (float)HW;
  for (long q = blockIdx.x * 256l + threadIdx.x; q < total; q += (long)gridDim.x * 256) {
    const int cc = (int)(q % cpr);
    const long n = q / cpr / HW;
    float v[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) v[e] = df[n * C + cc * VW + e] * inv;
    ((uint4*)dx)[q] = pack<T>(v);
  }
}

// ------------------------------------------------------------------ fp32 GEMM (classifier)
// C[M][N] = A B (+ bias) with A(m,k) = A[m*sam + k*sak], B(k,n) = B[k*sbk + n*sbn].
// The classifier GEMMs are small (M, N <= 1000) and long in K, so K is split
// over blockIdx.z; with several splits each writes its partial product to
// P[z][M][N] and gemm_splitk_reduce_kernel adds them in split order
// (deterministic). Tiles are loaded along whichever operand stride is 1.
// They are latency-bound: a block takes its K range in passes of GK rows,
// issuing every global load of a pass before the first is used (16 per
// operand and thread), so each pass costs one memory round trip.
constexpr int GK = 64;
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, long sam, long sak,
                                                       const float* __restrict__ B, long sbk, long sbn,
                                                       const float* __restrict__ bias, float* __restrict__ C,
                                                       int M, int N, int K, int kchunk, float* __restrict__ P) {
  __shared__ float As[GK][65], Bs[GK][65];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const int kb = blockIdx.z * kchunk, ke = min(K, kb + kchunk);
  float acc[4][4] = {};
  for (int k0 = kb; k0 < ke; k0 += GK) {
    float ra[16], rb[16];
#pragma unroll
    for (int l = 0; l < 16; ++l) {
      const int e = tid + 256 * l;
      const int mm = sak == 1 ? e >> 6 : e & 63, kk = sak == 1 ? e & 63 : e >> 6;
      ra[l] = (m0 + mm < M && k0 + kk < ke) ? A[(long)(m0 + mm) * sam + (long)(k0 + kk) * sak] : 0.f;
      const int nn = sbk == 1 ? e >> 6 : e & 63, kq = sbk == 1 ? e & 63 : e >> 6;
      rb[l] = (n0 + nn < N && k0 + kq < ke) ? B[(long)(k0 + kq) * sbk + (long)(n0 + nn) * sbn] : 0.f;
    }
    __syncthreads();   // the previous pass's reads of the tiles are done
#pragma unroll
    for (int l = 0; l < 16; ++l) {
      const int e = tid + 256 * l;
      const int mm = sak == 1 ? e >> 6 : e & 63, kk = sak == 1 ? e & 63 : e >> 6;
      As[kk][mm] = ra[l];
      const int nn = sbk == 1 ? e >> 6 : e & 63, kq = sbk == 1 ? e & 63 : e >> 6;
      Bs[kq][nn] = rb[l];
    }
    __syncthreads();
#pragma unroll 16
    for (int kk = 0; kk < GK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { a[i] = As[kk][ty * 4 + i]; b[i] = Bs[kk][tx * 4 + i]; }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
    }
  }
  float* __restrict__ out = P ? P + (long)blockIdx.z * M * N : C;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n < N) out[(long)m * N + n] = acc[i][j] + (!P && bias ? bias[n] : 0.f);
    }
  }
}

__global__ void gemm_splitk_reduce_kernel(const float* __restrict__ P, int splits, long MN, int N,
                                          const float* __restrict__ bias, float* __restrict__ C) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < MN; i += (long)gridDim.x * blockDim.x) {
    float v = 0.f;
    for (int z = 0; z < splits; ++z) v += P[z * MN + i];
    C[i] = v + (bias ? bias[i % N] : 0.f);
  }
}

// Column sums of A [M][N]: a block covers 64 columns with 4 row groups
// (rows g, g+4, ...); the four group sums are added in order.
__global__ __launch_bounds__(256) void colsum_kernel(const float* __restrict__ A, int M, int N,
                                                     float* __restrict__ out) {
  __shared__ float part[4][64];
  const int c = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int n = blockIdx.x * 64 + c;
  float s = 0.f;
  if (n < N)
    for (int m = q; m < M; m += 4) s += A[(long)m * N + n];
  part[q][c] = s;
  __syncthreads();
  if (q == 0 && n < N) out[n] = ((part[0][c] + part[1][c]) + part[2][c]) + part[3][c];
}

// ------------------------------------------------------------------ softmax cross-entropy
__device__ inline float block_reduce(float v, float* sh, bool is_max) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) sh[tid] = is_max ? fmaxf(sh[tid], sh[tid + s]) : sh[tid] + sh[tid + s];
    __syncthreads();
  }
  const float r = sh[0];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(256) void softmax_ce_kernel(const float* __restrict__ z, const int32_t* __restrict__ y,
                                                         int N, int C, float* __restrict__ dz,
                                                         float* __restrict__ row_loss, unsigned* err,
                                                         const LossScale* __restrict__ ls) {
  __shared__ float sh[256];
  const int n = blockIdx.x;
  const float* zr = z + (long)n * C;
  float* dr = dz + (long)n * C;
  const int lab = y[n];
  const bool bad = lab < 0 || lab >= C;
  float mx = -INFINITY;
  for (int c = threadIdx.x; c < C; c += 256) mx = fmaxf(mx, zr[c]);
  mx = block_reduce(mx, sh, true);
  float s = 0.f;
  for (int c = threadIdx.x; c < C; c += 256) s += expf(zr[c] - mx);
  s = block_reduce(s, sh, false);
  const float inv_s = 1.0f / s, inv_n = 1.0f / (float)N;
  // loss scaling: the backward pass starts from (scale x loss); the scale
  // is a power of two, so the product is exact
  const float sc = ls ? ls->scale : 1.0f;
  for (int c = threadIdx.x; c < C; c += 256) {
    const float p = expf(zr[c] - mx) * inv_s;
    dr[c] = bad ? 0.f : (p - (c == lab ? 1.f : 0.f)) * inv_n * sc;
  }
  if (threadIdx.x == 0) {
    if (bad) {
      atomicOr(err, (unsigned)DEVERR_LABEL);
      row_loss[n] = 0.f;
    } else {
      row_loss[n] = logf(s) + mx - zr[lab];
    }
  }
}

__global__ __launch_bounds__(256) void loss_reduce_kernel(const float* __restrict__ row_loss, int N,
                                                          float* __restrict__ loss, unsigned* err) {
  __shared__ double sh[256];
  double a = 0.0;
  for (int i = threadIdx.x; i < N; i += 256) a += (double)row_loss[i];
  sh[threadIdx.x] = a;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float l = (float)(sh[0] / (double)N);
    if (loss) loss[0] = l;
    if (!isfinite(l)) atomicOr(err, (unsigned)DEVERR_NONFINITE);
  }
}

// ------------------------------------------------------------------ flat fp32 streams
// With loss scaling (ls != NULL) the gradient holds scale x g: the update is
// skipped when the finiteness check found a non-finite value, else the
// gradient is multiplied by 1/scale (exact, a power of two) first.
__global__ void sgd_kernel(float* __restrict__ w, const float* __restrict__ g, float* __restrict__ v, long n,
                           float lr, float mom, float wd, const LossScale* __restrict__ ls) {
  float inv = 1.0f;
  if (ls) {
    if (ls->overflow) return;
    inv = ls->inv_scale;
  }
  const long n4 = n >> 2;
  for (long i = blockIdx.x * 256l + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
    float4 ww = ((float4*)w)[i], gg = ((const float4*)g)[i], vv = ((float4*)v)[i];
    gg.x *= inv; gg.y *= inv; gg.z *= inv; gg.w *= inv;
    vv.x = mom * vv.x + (gg.x + wd * ww.x); ww.x -= lr * vv.x;
    vv.y = mom * vv.y + (gg.y + wd * ww.y); ww.y -= lr * vv.y;
    vv.z = mom * vv.z + (gg.z + wd * ww.z); ww.z -= lr * vv.z;
    vv.w = mom * vv.w + (gg.w + wd * ww.w); ww.w -= lr * vv.w;
    ((float4*)w)[i] = ww;
    ((float4*)v)[i] = vv;
  }
  for (long i = (n4 << 2) + blockIdx.x * 256l + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
    const float vv = mom * v[i] + (g[i] * inv + wd * w[i]);
    v[i] = vv;
    w[i] -= lr * vv;
  }
}

// Finiteness of the scaled gradient: any Inf or NaN sets ls->overflow (a
// vector atomic from one lane per wave that found one).
__global__ void grad_check_kernel(const float* __restrict__ g, long n, LossScale* ls) {
  bool bad = false;
  const long n4 = n >> 2;
  for (long i = blockIdx.x * 256l + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
    const float4 x = ((const float4*)g)[i];
    bad |= !(__builtin_isfinite(x.x) && __builtin_isfinite(x.y) && __builtin_isfinite(x.z) && __builtin_isfinite(x.w));
  }
  for (long i = (n4 << 2) + blockIdx.x * 256l + threadIdx.x; i < n; i += (long)gridDim.x * 256)
    bad |= !__builtin_isfinite(g[i]);
  if (__any(bad) && (threadIdx.x & 63) == __ffsll(__ballot(bad)) - 1) atomicOr(&ls->overflow, 1u);
}

// Dynamic loss scale after a step: halve it (and count a skipped step)
// after an overflow, double it after `interval` steps in a row without one.
__global__ void loss_scale_update_kernel(LossScale* ls) {
  if (threadIdx.x != 0) return;
  LossScale x = *ls;
  if (x.overflow) {
    x.scale = fmaxf(x.scale * 0.5f, 1.0f);
    x.good = 0;
    ++x.skipped;
  } else if (++x.good >= x.interval) {
    x.scale = fminf(x.scale * 2.0f, 16777216.0f);
    x.good = 0;
  }
  x.inv_scale = 1.0f / x.scale;
  x.overflow = 0;
  *ls = x;
}

__global__ void merge_kernel(float* __restrict__ p, const float* __restrict__ ds, const float* __restrict__ dl,
                             long n, float f) {
  const long n4 = n >> 2;
  for (long i = blockIdx.x * 256l + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
    float4 pp = ((float4*)p)[i];
    const float4 a = ((const float4*)ds)[i], b = ((const float4*)dl)[i];
    pp.x -= b.x + f * a.x; pp.y -= b.y + f * a.y; pp.z -= b.z + f * a.z; pp.w -= b.w + f * a.w;
    ((float4*)p)[i] = pp;
  }
  for (long i = (n4 << 2) + blockIdx.x * 256l + threadIdx.x; i < n; i += (long)gridDim.x * 256)
    p[i] -= dl[i] + f * ds[i];
}

__global__ void delta_kernel(const float* __restrict__ a, const float* __restrict__ b, float* __restrict__ d,
                             long n) {
  const long n4 = n >> 2;
  for (long i = blockIdx.x * 256l + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
    const float4 x = ((const float4*)a)[i], y = ((const float4*)b)[i];
    ((float4*)d)[i] = make_float4(x.x - y.x, x.y - y.y, x.z - y.z, x.w - y.w);
  }
  for (long i = (n4 << 2) + blockIdx.x * 256l + threadIdx.x; i < n; i += (long)gridDim.x * 256) d[i] = a[i] - b[i];
}

__global__ void round_bf16_kernel(const float* __restrict__ x, bf16_t* __restrict__ y, long nchunks) {
  for (long q = blockIdx.x * 256l + threadIdx.x; q < nchunks; q += (long)gridDim.x * 256) {
    float v[8];
    unpack<float>(((const uint4*)x)[2 * q], v);
    unpack<float>(((const uint4*)x)[2 * q + 1], v + 4);
    ((uint4*)y)[q] = pack<bf16_t>(v);
  }
}

__global__ void fill_zero_kernel(uint32_t* __restrict__ p, long nwords) {
  for (long i = blockIdx.x * 256l + threadIdx.x; i < nwords; i += (long)gridDim.x * 256) p[i] = 0u;
}

}  // namespace

int ingest_launch(int prec, const float* img, void* x, int N, int H, int W, int Cp, unsigned* err, hipStream_t s) {
  const long npix = (long)N * H * W;
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(ingest_kernel<T>, dim3(grid_for(npix)), dim3(256), 0, s, img, (T*)x, npix, H * W, Cp,
                       err);
    return ok();
  });
}

int ingest_s2d_launch(int prec, const float* img, void* x, int N, int H, int W, unsigned* err, hipStream_t s) {
  if (H % 2 || W % 2) return -1;
  const long npix = (long)N * (H / 2) * (W / 2);
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(ingest_s2d_kernel<T>, dim3(grid_for(npix)), dim3(256), 0, s, img, (T*)x, npix, H, W,
                       err);
    return ok();
  });
}

int round_bf16_launch(const float* x, uint16_t* y, long n, hipStream_t s) {
  if (n % 8) return -1;
  hipLaunchKernelGGL(round_bf16_kernel, dim3(grid_for(n / 8)), dim3(256), 0, s, x, (bf16_t*)y, n / 8);
  return ok();
}

int repack_launch(int prec, const float* state, void* wf, void* wd, const RepackEntry* tab, int nent, long total,
                  hipStream_t s) {
  if (nent > 24) return -1;
  if (total <= 0) return 0;
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(repack_kernel<T>, dim3(grid_for(total)), dim3(256), 0, s, state, (T*)wf,
                       (T*)wd, tab, nent, total);
    return ok();
  });
}

int repack_tiled_launch(int prec, const float* state, void* wf, void* wd, const RepackEntry* tab, int nent,
                        int ntiles, hipStream_t s) {
  if (nent > 24) return -1;
  if (ntiles <= 0) return 0;
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(repack_tiled_kernel<T>, dim3(ntiles), dim3(256), 0, s, state, (T*)wf, (T*)wd,
                       tab, nent);
    return ok();
  });
}

bool repack_tiled_fits(int khw) { return khw <= kRepackMaxKHW; }
int repack_tiles(int cout, int cin_p) {
  return ((cout + kRepackT - 1) / kRepackT) * ((cin_p + kRepackT - 1) / kRepackT);
}

int maxpool_fwd_launch(int prec, const void* x, void* y, uint8_t* arg, int N, int H, int W, int C, int Ho, int Wo,
                       hipStream_t s) {
  const int vw = prec_vw(prec);
  const long work = (long)N * Ho * Wo * (C / vw);
  if ((long)N * H * W * C >= (1l << 31)) return -1;  // 32-bit chunk indices
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(maxpool_fwd_kernel<T>, dim3(grid_for(work)), dim3(256), 0, s, (const T*)x,
                       (T*)y, arg, N, H, W, C, Ho, Wo);
    return ok();
  });
}

int maxpool_bwd_launch(int prec, const void* dy, const uint8_t* arg, void* dx, int N, int H, int W, int C, int Ho,
                       int Wo, hipStream_t s) {
  const int vw = prec_vw(prec);
  const long work = (long)N * ((H + 1) / 2) * ((W + 1) / 2) * (C / vw);
  if ((long)N * H * W * C >= (1l << 31)) return -1;  // 32-bit chunk indices
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(maxpool_bwd_kernel<T>, dim3(grid_for(work)), dim3(256), 0, s, (const T*)dy, arg,
                       (T*)dx, N, H, W, C, Ho, Wo);
    return ok();
  });
}

int avgpool_fwd_launch(int prec, const void* x, float* f, int N, int HW, int C, hipStream_t s) {
  const int vw = prec_vw(prec);
  const long work = (long)N * (C / vw);
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(avgpool_fwd_kernel<T>, dim3(grid_for(work)), dim3(256), 0, s, (const T*)x, f, N, HW,
                       C);
    return ok();
  });
}

int avgpool_bwd_launch(int prec, const float* df, void* dx, int N, int HW, int C, hipStream_t s) {
  const int vw = prec_vw(prec);
  const long work = (long)N * HW * (C / vw);
  return with_prec(prec, [&](auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(avgpool_bwd_kernel<T>, dim3(grid_for(work)), dim3(256), 0, s, df, (T*)dx, N, HW, C);
    return ok();
  });
}

int gemm_f32_splits(int M, int N, int K) {
  const long tiles = (long)ceil_div(N, 64) * ceil_div(M, 64);
  int splits = 1;
  // at least 512 blocks or K ranges of one pass (GK) each
  while (tiles * splits < 512 && K > GK * splits) splits *= 2;
  return splits;
}

size_t gemm_f32_workspace(int M, int N, int K) {
  const int s = gemm_f32_splits(M, N, K);
  return s > 1 ? (size_t)s * M * N * 4 : 0;
}

int gemm_f32_launch(const float* A, long sam, long sak, const float* B, long sbk, long sbn, const float* bias,
                    float* C, int M, int N, int K, float* part, hipStream_t s) {
  if (M <= 0 || N <= 0) return 0;
  int splits = part ? gemm_f32_splits(M, N, K) : 1;
  const int kchunk = splits > 1 ? (ceil_div(K, splits) + 15) / 16 * 16 : (K > 0 ? K : 1);
  splits = K > 0 ? ceil_div(K, kchunk) : 1;
  hipLaunchKernelGGL(gemm_f32_kernel, dim3(ceil_div(N, 64), ceil_div(M, 64), splits), dim3(256), 0, s, A, sam, sak,
                     B, sbk, sbn, bias, C, M, N, K, kchunk, splits > 1 ? part : nullptr);
  if (splits > 1) {
    const long mn = (long)M * N;
    hipLaunchKernelGGL(gemm_splitk_reduce_kernel, dim3(grid_for(mn, 256, 1024)), dim3(256), 0, s, part, splits, mn,
                       N, bias, C);
  }
  return ok();
}

int colsum_launch(const float* A, int M, int N, float* out, hipStream_t s) {
  hipLaunchKernelGGL(colsum_kernel, dim3(ceil_div(N, 64)), dim3(256), 0, s, A, M, N, out);
  return ok();
}

int softmax_ce_launch(const float* z, const int32_t* labels, int N, int C, float* dz, float* row_loss, float* loss,
                      unsigned* err, hipStream_t s, const LossScale* ls) {
  hipLaunchKernelGGL(softmax_ce_kernel, dim3(N), dim3(256), 0, s, z, labels, N, C, dz, row_loss, err, ls);
  hipLaunchKernelGGL(loss_reduce_kernel, dim3(1), dim3(256), 0, s, row_loss, N, loss, err);
  return ok();
}

int dropout_launch(float* x, long n, uint64_t seed, uint64_t step, uint32_t thresh, float scale, hipStream_t s) {
  if (n < 0 || ((uintptr_t)x & 15)) return -1;
  const long n4 = (n + 3) / 4;
  if (n4 == 0) return 0;
  long blocks = (n4 + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(dropout_kernel, dim3(blocks), dim3(256), 0, s, x, n, (uint32_t)seed, (uint32_t)(seed >> 32),
                     (uint32_t)step, (uint32_t)(step >> 32), thresh, scale);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int sgd_launch(float* w, const float* g, float* v, long n, float lr, float mom, float wd, hipStream_t s,
               const LossScale* ls) {
  if (((uintptr_t)w | (uintptr_t)g | (uintptr_t)v) & 15) return -1;   // float4 accesses
  hipLaunchKernelGGL(sgd_kernel, dim3(grid_for((n + 3) / 4, 256, 8192)), dim3(256), 0, s, w, g, v, n, lr, mom, wd,
                     ls);
  return ok();
}

int grad_check_launch(const float* g, long n, LossScale* ls, hipStream_t s) {
  if ((uintptr_t)g & 15) return -1;
  hipLaunchKernelGGL(grad_check_kernel, dim3(grid_for((n + 3) / 4, 256, 4096)), dim3(256), 0, s, g, n, ls);
  return ok();
}

int loss_scale_update_launch(LossScale* ls, hipStream_t s) {
  hipLaunchKernelGGL(loss_scale_update_kernel, dim3(1), dim3(64), 0, s, ls);
  return ok();
}

int merge_launch(float* p, const float* ds, const float* dl, long n, float f, hipStream_t s) {
  hipLaunchKernelGGL(merge_kernel, dim3(grid_for((n + 3) / 4, 256, 8192)), dim3(256), 0, s, p, ds, dl, n, f);
  return ok();
}

int delta_launch(const float* a, const float* b, float* d, long n, hipStream_t s) {
  hipLaunchKernelGGL(delta_kernel, dim3(grid_for((n + 3) / 4, 256, 8192)), dim3(256), 0, s, a, b, d, n);
  return ok();
}

int fill_zero_launch(void* p, size_t bytes, hipStream_t s) {
  const long nw = (long)(bytes / 4);
  if (nw <= 0) return 0;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(nw, 256, 8192)), dim3(256), 0, s, (uint32_t*)p, nw);
  return ok();
}

}  // namespace rn18
