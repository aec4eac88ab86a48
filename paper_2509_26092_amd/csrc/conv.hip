// Convolutions of the ResNet-18 training step as implicit GEMMs on CDNA4 MFMA.
//
// Layout: activations NHWC (channels innermost), weights [Cout][KH*KW][Cin]
// for the forward pass and [Cin][KH*KW][Cout] for the data gradient; Cin is
// padded to a multiple of the 16-byte vector width (4 fp32 / 8 bf16).
//
// One kernel family ("gather") computes the forward pass and the data
// gradient. A GEMM row is an output pixel, a GEMM column an output channel,
// and the reduction runs over (tap, input channel). The data gradient of a
// stride-1 conv is a forward conv of dY with the taps mirrored; a stride-2
// conv's data gradient is split by the parity of the output pixel into four
// sub-convolutions, each with only its own taps, so no zero-inserted MACs are
// done (the tap arithmetic is parameterised: offset and step per axis).
//
// Tiles of K are staged through LDS as rows of 128 bytes (one or more 16-byte
// chunks of consecutive channels of one tap). Each MFMA lane supplies one
// 16-byte chunk of A and the matching chunk of B; the order of the K index
// inside an MFMA does not change the dot product, so fp32 (16x16x4) and bf16
// (16x16x32) share the LDS layout and the loaders.
//
// The weight gradient reduces over pixels. Its dY and im2col X tiles are
// staged as they lie in memory (one pixel's 128 bytes of channels per LDS row)
// and the pixel-major MFMA operands are built on the way out of LDS (gfx950
// transpose reads for bf16, 4-byte reads for fp32). The older kernel for
// 16-channel outputs transposes in registers instead. Partial sums of a split
// of the pixel range go to a scratch buffer that is summed in a fixed order
// (deterministic, no float atomics).
#include "kernels.h"

#include <cstdio>
#include <mutex>
#include <set>
#include <string>

namespace rn18 {

namespace {

constexpr int RSTR = 9;  // LDS row stride in 16-byte units: 8 data chunks + 1 pad

__device__ inline int xcd_remap(int b, int nb) {
  // Blocks are dealt round-robin to the 8 XCDs; give each XCD a contiguous
  // range of logical tiles so neighbouring tiles share its L2.
  int per = nb >> 3, rem = nb & 7;
  int x = b & 7, r = b >> 3;
  return x * per + (x < rem ? x : rem) + r;
}

template <typename T> struct Mma;
template <> struct Mma<bf16_t> {
  static constexpr int SUB = 1;
  __device__ static inline void run(floatx4_t& acc, const uint4& a, const uint4& b, int) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
  }
};
template <> struct Mma<float> {
  static constexpr int SUB = 4;
  __device__ static inline float el(const uint4& q, int t) {
    return __builtin_bit_cast(float, t == 0 ? q.x : t == 1 ? q.y : t == 2 ? q.z : q.w);
  }
  __device__ static inline void run(floatx4_t& acc, const uint4& a, const uint4& b, int t) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(el(a, t), el(b, t), acc, 0, 0, 0);
  }
};

// One 128-byte K stage: two groups of four 16-byte chunks (one per lane group).
template <typename T, int FM, int FN>
__device__ inline void mma_stage(floatx4_t (&acc)[FM][FN], const uint4* As, const uint4* Bs,
                                 int arow0, int brow0, int lane) {
#pragma unroll
  for (int kg = 0; kg < 2; ++kg) {
    const int ch = kg * 4 + (lane >> 4);
    uint4 a[FM], b[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) a[i] = As[(arow0 + i * 16 + (lane & 15)) * RSTR + ch];
#pragma unroll
    for (int j = 0; j < FN; ++j) b[j] = Bs[(brow0 + j * 16 + (lane & 15)) * RSTR + ch];
#pragma unroll
    for (int t = 0; t < Mma<T>::SUB; ++t)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) Mma<T>::run(acc[i][j], a[i], b[j], t);
  }
}

// ---------------------------------------------------------------------------
// Gather conv, pipelined: the K loop streams 128-byte row stages from global
// memory straight into an LDS ring of STAGES buffers (gfx950
// global_load_lds_dwordx4, one 16-byte chunk per lane, written lane-contiguous
// at the instruction's LDS base), so STAGES-1 stages are in flight while one
// is multiplied. Rows are 128 bytes without padding; the chunk of row r that
// goes to slot q is q ^ (r & 7), which spreads the 16 rows of an MFMA operand
// read over all LDS banks. Taps outside the image and K beyond the end load
// from a zero page. When Cin is a multiple of the stage width, a stage is one
// tap and a contiguous block of channels, and the tap arithmetic is uniform.
// ---------------------------------------------------------------------------
__device__ uint4 g_zero_page[8];  // zero-initialised at load; never written

typedef __attribute__((address_space(3))) void* lds_void_t;

// 16-byte global -> LDS copy of each lane's chunk, written lane-contiguous at
// the wave-uniform LDS byte address `lds`. Issued as inline assembly so that
// the compiler's wait-count insertion does not treat every later LDS read as
// dependent on it; completion is tracked by explicit vmcnt waits instead.
__device__ inline void lds_dma16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds) : "memory", "m0");
}
// Buffer resource of a raw byte range [base, base + bytes): a buffer load at
// a byte offset >= bytes is out of range and returns zeros (written to LDS
// as zeros by the DMA form), which is how padding taps are filled.
typedef int i32x4_t __attribute__((ext_vector_type(4)));
__device__ inline i32x4_t buffer_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  i32x4_t r;
  r[0] = (int)(uint32_t)a;
  r[1] = (int)(uint32_t)(a >> 32);  // stride 0
  r[2] = (int)bytes;
  r[3] = 0x00020000;                // raw 32-bit dwords, no swizzle
  return r;
}
constexpr uint32_t kOutOfRange = 0x80000000u;  // byte offset beyond every buffer used here

// 16-byte buffer -> LDS copy of each lane's chunk at byte offset `voff` of
// the buffer `rsrc`, written lane-contiguous at the wave-uniform LDS byte
// address `lds`.
__device__ inline void lds_dma16_buf(uint32_t voff, i32x4_t rsrc, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff), "s"(rsrc), "s"(lds)
               : "memory", "m0");
}

__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(lds_void_t)p;
}

// Workgroup barrier without the memory fence __syncthreads() implies (the
// fence would wait for every outstanding LDS-DMA stage, not just the one
// about to be read).
__device__ inline void barrier_only() { asm volatile("s_barrier" ::: "memory"); }

template <int N>
__device__ inline void wait_vmcnt() {
  // s_waitcnt vmcnt(N), expcnt and lgkmcnt left at their maximum
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <int IPW>
__device__ inline void wait_stage(int later_issued) {
  // wait until only `later_issued` stages of IPW loads each are outstanding
  if (later_issued >= 2) wait_vmcnt<2 * IPW>();
  else if (later_issued == 1) wait_vmcnt<IPW>();
  else wait_vmcnt<0>();
}

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES, bool UNI>
__global__ __launch_bounds__(64 * WGM * WGN) void conv_gather2_kernel(ConvGather g) {
  constexpr int NW = WGM * WGN, NT = 64 * NW;
  constexpr int VW = TT<T>::VW;
  constexpr int KT = 128 / (int)sizeof(T);
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int AI = BM / 8, BI = BN / 8;          // 8-row load instructions per stage
  constexpr int NI = AI + BI, IPW = NI / NW;       // per wave
  constexpr int STAGE_U4 = (BM + BN) * 8;
  constexpr int SM_LOOP = STAGES * STAGE_U4;
  constexpr int WSTR = WTN + 4;                    // epilogue strip row stride (floats)
  constexpr int SM_EPI = NW * 16 * WSTR / 4;       // one 16-row strip per wave
  constexpr int ST_F = 2 * VW;                     // per-lane BN partial: VW shifted sums, VW squares
  constexpr int SM_ST = SM_EPI + (BN + NW * 64 * ST_F + 3) / 4;
  __shared__ uint4 smem[SM_LOOP > SM_ST ? SM_LOOP : SM_ST];
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
  static_assert(NI % NW == 0 && BN % 8 == 0, "whole load instructions per wave");
  static_assert(STAGES >= 2 && STAGES <= 4, "stages");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int tiles_n = (g.Cols + BN - 1) / BN;
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (t / tiles_n) * BM, n0 = (t % tiles_n) * BN;
  const T* __restrict__ A = (const T*)g.A;
  const T* __restrict__ B = (const T*)g.B;
  const int HWm = g.Hm * g.Wm;
  const int c = (lane & 7) ^ (lane >> 3);          // chunk this lane loads (slot lane&7, row lane>>3)
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t smem_lds = lds_addr(smem);
  const void* const zero = g.zero;

  // Per load instruction of this wave: the row it fills and that row's geometry.
  bool isA[IPW], ok[IPW];
  int pix[IPW], hb[IPW], wb[IPW];
  long boff[IPW];
#pragma unroll
  for (int u = 0; u < IPW; ++u) {
    const int j = wave_u + NW * u;
    isA[u] = j < AI;
    if (isA[u]) {
      const int m = m0 + j * 8 + (lane >> 3);
      ok[u] = m < g.M;
      const int mm = ok[u] ? m : 0;
      const int n = (int)g.fd_hw.div(mm), rem = mm - n * HWm;
      const int i = (int)g.fd_w.div(rem), jj = rem - i * g.Wm;
      hb[u] = i * g.is - g.ip;
      wb[u] = jj * g.is - g.ip;
      pix[u] = (n * g.Hin + hb[u]) * g.Win + wb[u];
      boff[u] = 0;
    } else {
      const int col = n0 + (j - AI) * 8 + (lane >> 3);
      ok[u] = col < g.Cols;
      boff[u] = (long)(ok[u] ? col : 0) * g.KHW * g.Cin;
      hb[u] = wb[u] = pix[u] = 0;
    }
  }
  const int CB = UNI ? (g.Cin >= KT ? g.Cin / KT : 1) : 1;

  // Uniform path: per-lane byte offsets and tap-validity masks are fixed for
  // the whole K loop; a stage only adds the wave-uniform offset of its tap
  // and channel block, kept incrementally in scalars. A 128-byte row is one
  // tap and KT channels when Cin >= KT; with fewer channels it holds RT =
  // KT / Cin consecutive taps along w (consecutive pixels, contiguous in
  // NHWC), and each lane's chunk sits at its own pixel of the row.
  constexpr int UA = AI / NW, UB = BI / NW;        // A and B load instructions per wave
  static_assert(AI % NW == 0 && BI % NW == 0, "loads split evenly between A and B");
  const int es = (int)sizeof(T);
  const int RT = UNI && g.Cin < KT ? KT / g.Cin : 1;   // taps per row
  const int ntw_g = g.ntw / RT;                        // row groups along w
  uint32_t uoff[UNI ? IPW : 1];
  uint32_t umask[UNI ? UA : 1];
  i32x4_t rsA, rsB;
  int st_ti = 0, st_th = 0, st_tw = 0, st_cb = 0;  // tap (th, tw group), channel block of the next stage issued
  if (UNI) {
    rsA = buffer_rsrc(A, (uint32_t)((long)g.N * g.Hin * g.Win * g.Cin * es));
    rsB = buffer_rsrc(B, (uint32_t)((long)g.Cols * g.KHW * g.Cin * es));
    const int lane_px = (c * VW) / g.Cin;              // pixel of this lane's chunk within a row
#pragma unroll
    for (int u = 0; u < UA; ++u) {
      // valid tap rows x valid tap-group columns, as bit vectors
      uint32_t vh = 0, vw = 0, m = 0;
      for (int th = 0; th < g.nth; ++th)
        vh |= (unsigned)(hb[u] + g.dh0 + th * g.dhs) < (unsigned)g.Hin ? 1u << th : 0u;
      for (int tg = 0; tg < ntw_g; ++tg)
        vw |= (unsigned)(wb[u] + g.dw0 + (tg * RT + lane_px) * g.dws) < (unsigned)g.Win ? 1u << tg : 0u;
      for (int th = 0; th < g.nth; ++th) m |= (vh >> th) & 1u ? vw << (th * ntw_g) : 0u;
      umask[u] = ok[u] ? m : 0u;
      uoff[u] = (uint32_t)(pix[u] * g.Cin * es + c * 16);
    }
#pragma unroll
    for (int u = UA; u < IPW; ++u) uoff[u] = ok[u] ? (uint32_t)(boff[u] * es + c * 16) : kOutOfRange;
  }
  auto issue_uni = [&](int buf) {
    const int dh = g.dh0 + st_th * g.dhs, dw = g.dw0 + st_tw * RT * g.dws;
    const int wt = (g.wkh0 + st_th * g.wkhs) * g.KW + g.wkw0 + st_tw * RT * g.wkws;
    const uint32_t sa = (uint32_t)((dh * g.Win + dw) * g.Cin * es + st_cb * 128);
    const uint32_t sb = (uint32_t)(wt * g.Cin * es + st_cb * 128);
    const uint32_t base = smem_lds + (uint32_t)(buf * STAGE_U4 * 16);
#pragma unroll
    for (int u = 0; u < UA; ++u) {
      const uint32_t v = (umask[u] >> st_ti) & 1u ? uoff[u] + sa : kOutOfRange;
      lds_dma16_buf(v, rsA, base + (uint32_t)((wave_u + NW * u) * 1024));
    }
#pragma unroll
    for (int u = UA; u < IPW; ++u) {
      const uint32_t v = uoff[u] == kOutOfRange ? kOutOfRange : uoff[u] + sb;
      lds_dma16_buf(v, rsB, base + (uint32_t)((AI + wave_u + NW * (u - UA)) * 1024));
    }
    if (++st_cb == CB) {
      st_cb = 0;
      ++st_ti;
      if (++st_tw == ntw_g) { st_tw = 0; ++st_th; }
    }
  };

  // General path (channel chunks of different taps in one row): per-lane tap
  // arithmetic and 64-bit addresses, padding read from the zero page.
  auto issue = [&](int s, int buf) {
    const int k = s * KT + c * VW;
    const bool kok = k < g.K;
    const int tap = kok ? k / g.Cin : 0;
    const int ci = k - tap * g.Cin;
    const int th = tap / g.ntw, tw = tap - th * g.ntw;
    const int dh = g.dh0 + th * g.dhs;
    const int dw = g.dw0 + tw * g.dws;
    const int wt = (g.wkh0 + th * g.wkhs) * g.KW + g.wkw0 + tw * g.wkws;
    const uint32_t base = smem_lds + (uint32_t)(buf * STAGE_U4 * 16);
#pragma unroll
    for (int u = 0; u < IPW; ++u) {
      const int j = wave_u + NW * u;
      const void* src;
      if (isA[u]) {
        const bool in = kok && ok[u] && (unsigned)(hb[u] + dh) < (unsigned)g.Hin &&
                        (unsigned)(wb[u] + dw) < (unsigned)g.Win;
        src = in ? (const void*)(A + (long)(pix[u] + dh * g.Win + dw) * g.Cin + ci) : zero;
      } else {
        src = kok && ok[u] ? (const void*)(B + boff[u] + (long)wt * g.Cin + ci) : zero;
      }
      lds_dma16(src, base + (uint32_t)(j * 1024));
    }
  };

  floatx4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  const int S = (g.K + KT - 1) / KT;
#pragma unroll
  for (int p = 0; p < STAGES - 1; ++p)
    if (p < S) {
      if (UNI) issue_uni(p);
      else issue(p, p);
    }
  const int arow0 = wm * WTM, brow0 = wn * WTN;
  const int sw = lane & 7;
  for (int s = 0; s < S; ++s) {
    const int later = min(STAGES - 2, S - 1 - s);
    wait_stage<IPW>(later);
    barrier_only();
    if (s + STAGES - 1 < S) {
      if (UNI) issue_uni((s + STAGES - 1) % STAGES);
      else issue(s + STAGES - 1, (s + STAGES - 1) % STAGES);
    }
    const uint4* As = smem + (s % STAGES) * STAGE_U4;
    const uint4* Bs = As + BM * 8;
    // both 64-byte halves of the stage's rows are read before any MFMA, so
    // the second half's LDS latency hides behind the first half's MFMAs
    uint4 a[2][FM], b[2][FN];
#pragma unroll
    for (int kg = 0; kg < 2; ++kg) {
      const int slot = (kg * 4 + (lane >> 4)) ^ sw;
#pragma unroll
      for (int i = 0; i < FM; ++i) a[kg][i] = As[(arow0 + i * 16 + (lane & 15)) * 8 + slot];
#pragma unroll
      for (int j = 0; j < FN; ++j) b[kg][j] = Bs[(brow0 + j * 16 + (lane & 15)) * 8 + slot];
    }
    __builtin_amdgcn_sched_barrier(0);   // keep every LDS read ahead of the MFMAs
#pragma unroll
    for (int kg = 0; kg < 2; ++kg)
#pragma unroll
      for (int tt = 0; tt < Mma<T>::SUB; ++tt)
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j) Mma<T>::run(acc[i][j], a[kg][i], b[kg][j], tt);
  }
  wait_vmcnt<0>();
  __syncthreads();

  // Epilogue per wave, one 16-row strip at a time: the strip's accumulators
  // go through a wave-private LDS buffer and leave as 16-byte chunks of
  // consecutive output channels. With g.stats set (forward pass followed by
  // batch norm), the stored (rounded) values also feed per-channel partial
  // statistics of the tile: sums of v - shift and (v - shift)^2, with the
  // tile's first row as the shift (a sample of the channel keeps the sums
  // well conditioned), summed over lanes and waves in a fixed order and
  // written to g.stats[tile_m][col] as (rows, shift, sum, sum of squares).
  float* Ws = (float*)smem + wave_u * 16 * WSTR;
  constexpr int CPW = WTN / VW;                    // chunks per strip row; a lane's chunk column is lane % CPW
  static_assert(64 % CPW == 0, "lane chunk column fixed across strips");
  T* __restrict__ Cg = (T*)g.C;
  const bool stats = g.stats != nullptr;
  float* Sh = (float*)smem + SM_EPI * 4;           // [BN] shifts, then [NW][64][ST_F] lane sums
  float* St = Sh + BN;
  float ssh[VW], ss1[VW], ss2[VW];
#pragma unroll
  for (int e = 0; e < VW; ++e) ssh[e] = ss1[e] = ss2[e] = 0.f;
  if (stats) {
    // tile row 0 sits in strip 0, register 0 of lanes 0..15 of the waves with wm == 0
    if (wm == 0 && lane < 16) {
#pragma unroll
      for (int j = 0; j < FN; ++j) Sh[brow0 + j * 16 + lane] = TT<T>::to_f(TT<T>::from_f(acc[0][j][0]));
    }
    __syncthreads();
    const int cc = lane % CPW;
#pragma unroll
    for (int e = 0; e < VW; ++e) ssh[e] = Sh[brow0 + cc * VW + e];
  }
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) Ws[(4 * (lane >> 4) + r) * WSTR + j * 16 + (lane & 15)] = acc[i][j][r];
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    for (int idx = lane; idx < 16 * CPW; idx += 64) {
      const int row = idx / CPW, cc = idx - row * CPW;
      const int m = m0 + arow0 + i * 16 + row, col = n0 + brow0 + cc * VW;
      if (m >= g.M || col >= g.Cols) continue;
      const int n = (int)g.fd_hw.div(m), rem = m - n * HWm;
      const int ii = (int)g.fd_w.div(rem), jj = rem - ii * g.Wm;
      const uint32_t off = ((uint32_t)((n * g.Hout + ii * g.os + g.oph) * g.Wout + jj * g.os + g.opw)) * g.Cols + col;
      float v[VW];
#pragma unroll
      for (int e = 0; e < VW; ++e) v[e] = Ws[row * WSTR + cc * VW + e];
      if (g.mode == 1) {
        float o[VW];
        unpack<T>(*(const uint4*)(Cg + off), o);
#pragma unroll
        for (int e = 0; e < VW; ++e) v[e] += o[e];
      } else if (g.mode == 2) {
        float rr[VW], mk[VW];
        unpack<T>(*(const uint4*)((const T*)g.R + off), rr);
        unpack<T>(*(const uint4*)((const T*)g.Rm + off), mk);
#pragma unroll
        for (int e = 0; e < VW; ++e) v[e] += mk[e] > 0.f ? rr[e] : 0.f;
      }
      const uint4 pk = pack<T>(v);
      *(uint4*)(Cg + off) = pk;
      if (stats) {
        float vr[VW];
        unpack<T>(pk, vr);
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          const float d = vr[e] - ssh[e];
          ss1[e] += d;
          ss2[e] = __builtin_fmaf(d, d, ss2[e]);
        }
      }
    }
  }
  if (!stats) return;
  {
    float* o = St + (wave_u * 64 + lane) * ST_F;
#pragma unroll
    for (int e = 0; e < VW; ++e) { o[e] = ss1[e]; o[VW + e] = ss2[e]; }
  }
  __syncthreads();
  const int rows = min(BM, g.M - m0);
  for (int cl = tid; cl < BN; cl += NT) {
    const int col = n0 + cl;
    if (col >= g.Cols) continue;
    const int wn_c = cl / WTN, cw = cl - wn_c * WTN, cc = cw / VW, e = cw - cc * VW;
    float a1 = 0.f, a2 = 0.f;
    for (int wmi = 0; wmi < WGM; ++wmi)
      for (int k = 0; k < 64 / CPW; ++k) {
        const float* p = St + ((wmi * WGN + wn_c) * 64 + cc + CPW * k) * ST_F;
        a1 += p[e];
        a2 += p[VW + e];
      }
    float4* out = (float4*)g.stats + ((long)(m0 / BM) * g.Cols + col);
    *out = make_float4((float)rows, Sh[cl], a1, a2);
  }
}

// ---------------------------------------------------------------------------
// Weight gradient
// ---------------------------------------------------------------------------
template <typename T> struct Tr;
template <> struct Tr<bf16_t> {
  // 8 pixels x 8 channels (bf16) -> 8 channels x 8 pixels
  __device__ static inline void run(const uint4 (&in)[8], uint4 (&out)[8]) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      uint32_t x[8];
#pragma unroll
      for (int p = 0; p < 8; ++p) x[p] = d == 0 ? in[p].x : d == 1 ? in[p].y : d == 2 ? in[p].z : in[p].w;
      uint32_t lo[4], hi[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        lo[q] = (x[2 * q] & 0xffffu) | (x[2 * q + 1] << 16);
        hi[q] = (x[2 * q] >> 16) | (x[2 * q + 1] & 0xffff0000u);
      }
      out[2 * d] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
      out[2 * d + 1] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
    }
  }
};
template <> struct Tr<float> {
  __device__ static inline void run(const uint4 (&in)[4], uint4 (&out)[4]) {
    out[0] = make_uint4(in[0].x, in[1].x, in[2].x, in[3].x);
    out[1] = make_uint4(in[0].y, in[1].y, in[2].y, in[3].y);
    out[2] = make_uint4(in[0].z, in[1].z, in[2].z, in[3].z);
    out[3] = make_uint4(in[0].w, in[1].w, in[2].w, in[3].w);
  }
};

template <typename T, int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(256) void conv_wgrad_kernel(ConvWgrad g) {
  constexpr int VW = TT<T>::VW;
  constexpr int KTP = 128 / (int)sizeof(T);  // pixels per stage
  constexpr int PG = KTP / VW;               // pixel groups per stage (8)
  constexpr int NA = PG * (BM / VW), NB = PG * (BN / VW);
  constexpr int NBLK = (NA + NB + 255) / 256;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int STAGE = (BM + BN) * RSTR;
  __shared__ uint4 smem[2 * STAGE];
  static_assert(WGM * WGN == 4, "4 waves");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  // One-dimensional grid over (split, tile), tile fastest; the XCD remap
  // keeps all tiles of a pixel split on one XCD, so the split's dY and X rows
  // are fetched from HBM once and re-read from that XCD's L2.
  const int tiles_n = (g.Kcols + BN - 1) / BN;
  const int tiles = ((g.Cout + BM - 1) / BM) * tiles_n;
  const int lt = xcd_remap(blockIdx.x, gridDim.x);
  const int split = lt / tiles, t = lt - split * tiles;
  const int co0 = (t / tiles_n) * BM, k0 = (t % tiles_n) * BN;
  const int p_begin = split * g.pix_per_split;
  const int p_end = min(g.Mpix, p_begin + g.pix_per_split);
  const int HWo = g.Ho * g.Wo;

  const T* __restrict__ DY = (const T*)g.DY;
  const T* __restrict__ X = (const T*)g.X;

  uint4 rv[NBLK][VW];
  auto load = [&](int p0) {
#pragma unroll
    for (int u = 0; u < NBLK; ++u) {
      const int b = tid + 256 * u;
      if (b < NA) {
        const int cg = b % (BM / VW), pg = b / (BM / VW);
        const int co = co0 + cg * VW;
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          const int p = p0 + pg * VW + e;
          uint4 v = make_uint4(0, 0, 0, 0);
          if (p < p_end && co < g.Cout) v = *(const uint4*)(DY + (long)p * g.Cout + co);
          rv[u][e] = v;
        }
      } else if (b < NA + NB) {
        const int bb = b - NA;
        const int cc = bb % (BN / VW), pg = bb / (BN / VW);
        const int kc = k0 + cc * VW;
        const bool kok = kc < g.Kcols;
        const int tap = kok ? kc / g.Cin : 0;
        const int ci = kc - tap * g.Cin;
        const int kh = tap / g.KW, kw = tap - kh * g.KW;
        int p = p0 + pg * VW;
        const int pc = p < g.Mpix ? p : 0;
        int n = pc / HWo, rem = pc - n * HWo;
        int ho = rem / g.Wo, wo = rem - ho * g.Wo;
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          uint4 v = make_uint4(0, 0, 0, 0);
          const int hi = ho * g.stride - g.pad + kh, wi = wo * g.stride - g.pad + kw;
          if (kok && p + e < p_end && (unsigned)hi < (unsigned)g.H && (unsigned)wi < (unsigned)g.W)
            v = *(const uint4*)(X + ((long)(n * g.H + hi) * g.W + wi) * g.Cin + ci);
          rv[u][e] = v;
          if (++wo == g.Wo) { wo = 0; if (++ho == g.Ho) { ho = 0; ++n; } }
        }
      }
    }
  };
  auto store = [&](int buf) {
    uint4* As = smem + buf * STAGE;
    uint4* Bs = As + BM * RSTR;
#pragma unroll
    for (int u = 0; u < NBLK; ++u) {
      const int b = tid + 256 * u;
      uint4 o[VW];
      if (b < NA) {
        const int cg = b % (BM / VW), pg = b / (BM / VW);
        Tr<T>::run(rv[u], o);
#pragma unroll
        for (int e = 0; e < VW; ++e) As[(cg * VW + e) * RSTR + pg] = o[e];
      } else if (b < NA + NB) {
        const int bb = b - NA;
        const int cc = bb % (BN / VW), pg = bb / (BN / VW);
        Tr<T>::run(rv[u], o);
#pragma unroll
        for (int e = 0; e < VW; ++e) Bs[(cc * VW + e) * RSTR + pg] = o[e];
      }
    }
  };

  floatx4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  const int S = p_end > p_begin ? (p_end - p_begin + KTP - 1) / KTP : 0;
  if (S > 0) {
    load(p_begin);
    store(0);
  }
  __syncthreads();
  for (int s = 0; s < S; ++s) {
    if (s + 1 < S) load(p_begin + (s + 1) * KTP);
    const uint4* As = smem + (s & 1) * STAGE;
    mma_stage<T, FM, FN>(acc, As, As + BM * RSTR, wm * WTM, wn * WTN, lane);
    if (s + 1 < S) store((s + 1) & 1);
    __syncthreads();
  }

  float* __restrict__ P = g.P + (long)split * g.Cout * g.Kcols;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int kc = k0 + wn * WTN + j * 16 + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = co0 + wm * WTM + i * 16 + 4 * (lane >> 4) + r;
        if (co < g.Cout && kc < g.Kcols) P[(long)co * g.Kcols + kc] = acc[i][j][r];
      }
    }
}

// ---------------------------------------------------------------------------
// Weight gradient, pipelined. Both operand tiles are staged exactly as they
// lie in memory, one pixel per 128-byte LDS row (dY: that pixel's output
// channels; X: the input channels its tap reads, or the 16-byte chunks of
// several taps when Cin is smaller than a row), loaded by the same LDS-DMA
// ring as the gather kernel. The reduction runs over pixels, so the MFMA
// operands need several pixels of one channel per lane: bf16 reads them with
// the gfx950 LDS transpose read (ds_read_b64_tr_b16, four lanes' 8-byte row
// pieces transposed across a 16-lane group), fp32 with one 4-byte read per
// pixel. Partial sums of a pixel split go to a scratch buffer summed in a
// fixed order afterwards.
// ---------------------------------------------------------------------------
typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_char_t;

template <typename T> struct WOp;
template <> struct WOp<bf16_t> {
  static constexpr int KP = 64;      // pixels per stage
  static constexpr int KSTEPS = 2;   // MFMA k-steps (32 pixels each) per stage
  typedef uint4 frag_t;
  // 16 channels [ch0, ch0+16) of a 64-channel sub-tile, pixels kk*32 + 8*(lane/16) + 0..7
  __device__ static inline uint4 frag(const lds_char_t* sub, int ch0, int kk, int lane) {
    const int r = lane & 15, kq = lane >> 4;
    const int ch = ch0 + 4 * (r & 3);
    const int c = ch >> 3, bo = (ch & 7) << 1;
    int p = kk * 32 + 8 * kq + (r >> 2);
    const lds_char_t* a1 = sub + p * 128 + ((c ^ (p & 7)) << 4) + bo;
    p += 4;
    const lds_char_t* a2 = sub + p * 128 + ((c ^ (p & 7)) << 4) + bo;
    const v4i16_t x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16_t*)a1);
    const v4i16_t y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16_t*)a2);
    uint4 q;
    q.x = (uint32_t)(uint16_t)x[0] | ((uint32_t)(uint16_t)x[1] << 16);
    q.y = (uint32_t)(uint16_t)x[2] | ((uint32_t)(uint16_t)x[3] << 16);
    q.z = (uint32_t)(uint16_t)y[0] | ((uint32_t)(uint16_t)y[1] << 16);
    q.w = (uint32_t)(uint16_t)y[2] | ((uint32_t)(uint16_t)y[3] << 16);
    return q;
  }
  __device__ static inline void mma(floatx4_t& acc, const uint4& a, const uint4& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                  acc, 0, 0, 0);
  }
};
template <> struct WOp<float> {
  static constexpr int KP = 32;      // pixels per stage
  static constexpr int KSTEPS = 8;   // MFMA k-steps (4 pixels each) per stage
  typedef float frag_t;
  // channel ch0 + lane%16 of a 32-channel sub-tile, pixel kk*4 + lane/16
  __device__ static inline float frag(const lds_char_t* sub, int ch0, int kk, int lane) {
    const int ch = ch0 + (lane & 15), p = kk * 4 + (lane >> 4);
    const int c = ch >> 2;
    return *(const __attribute__((address_space(3))) float*)(sub + p * 128 + ((c ^ (p & 7)) << 4) + ((ch & 3) << 2));
  }
  __device__ static inline void mma(floatx4_t& acc, float a, float b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
  }
};

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES>
__global__ __launch_bounds__(64 * WGM * WGN) void conv_wgrad2_kernel(ConvWgrad g) {
  typedef WOp<T> O;
  constexpr int NW = WGM * WGN;
  constexpr int VW = TT<T>::VW;
  constexpr int CPS = 128 / (int)sizeof(T);     // channels per LDS row
  constexpr int KP = O::KP;
  constexpr int SA = BM / CPS, SB = BN / CPS;   // 128-byte-wide sub-tiles of each operand
  constexpr int RI = KP / 8;                    // load instructions per sub-tile
  constexpr int NI = (SA + SB) * RI, IPW = NI / NW;
  constexpr int SUB_B = KP * 128, STAGE_B = (SA + SB) * SUB_B;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  __shared__ uint4 smem[STAGES * STAGE_B / 16];
  static_assert(NI % NW == 0 && BM % CPS == 0 && BN % CPS == 0, "tile shape");
  static_assert(RI % NW == 0 || NW % RI == 0, "load rows");
  static_assert(STAGES >= 2 && STAGES <= 4, "stages");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave_u = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave_u / WGN, wn = wave_u % WGN;
  // One-dimensional grid over (split, tile), tile fastest; the XCD remap
  // keeps all tiles of a pixel split on one XCD, so the split's dY and X rows
  // are fetched from HBM once and re-read from that XCD's L2.
  const int tiles_n = (g.Kcols + BN - 1) / BN;
  const int tiles = ((g.Cout + BM - 1) / BM) * tiles_n;
  const int lt = xcd_remap(blockIdx.x, gridDim.x);
  const int split = lt / tiles, t = lt - split * tiles;
  const int co0 = (t / tiles_n) * BM, k0 = (t % tiles_n) * BN;
  const int p_begin = split * g.pix_per_split;
  const int p_end = min(g.Mpix, p_begin + g.pix_per_split);
  const int HWo = g.Ho * g.Wo;
  const T* __restrict__ DY = (const T*)g.DY;
  const T* __restrict__ X = (const T*)g.X;
  const int c = (lane & 7) ^ (lane >> 3);
  const uint32_t smem_lds = lds_addr(smem);

  // Fixed geometry of each load instruction of this wave: its LDS row (a
  // pixel of the stage), and the channel chunk it copies. The pixel of a
  // lane's row advances by KP per stage; its (n, ho, wo) coordinates are
  // carried incrementally, so no stage divides.
  const int es = (int)sizeof(T);
  const i32x4_t rsA = buffer_rsrc(DY, (uint32_t)((long)g.Mpix * g.Cout * es));
  const i32x4_t rsB = buffer_rsrc(X, (uint32_t)((long)g.N * g.H * g.W * g.Cin * es));
  // When NW is a multiple of RI every load of a wave fills the same LDS row
  // (pixel), so one set of pixel coordinates serves all of them.
  constexpr bool ONE_ROW = NW % RI == 0;
  constexpr int NR = ONE_ROW ? 1 : IPW;
  bool isA[IPW];
  int row[IPW];
  uint32_t coff[IPW];   // A: channel byte offset; B: tap + channel byte offset; or out of range
  int tdh[IPW], tdw[IPW];
  int pn[NR], pho[NR], pwo[NR];
#pragma unroll
  for (int u = 0; u < IPW; ++u) {
    // load j = wave_u + NW*u fills row j % RI of sub-tile j / RI; written so
    // that the sub-tile (and with it A or B) is a compile-time constant
    // whenever NW divides RI
    const int sub = RI % NW == 0 ? NW * u / RI : (NW / RI) * u + wave_u / RI;
    row[u] = (RI % NW == 0 ? NW * u % RI + wave_u : wave_u % RI) * 8 + (lane >> 3);
    isA[u] = sub < SA;
    tdh[u] = tdw[u] = 0;
    if (isA[u]) {
      const int co = co0 + sub * CPS + c * VW;
      coff[u] = co < g.Cout ? (uint32_t)(co * es) : kOutOfRange;
    } else {
      const int kc = k0 + (sub - SA) * CPS + c * VW;
      if (kc < g.Kcols) {
        const int tap = kc / g.Cin, ci = kc - tap * g.Cin;
        const int kh = tap / g.KW, kw = tap - kh * g.KW;
        tdh[u] = kh - g.pad;
        tdw[u] = kw - g.pad;
        coff[u] = (uint32_t)(((kh - g.pad) * g.W + (kw - g.pad)) * g.Cin * es + ci * es);
      } else {
        coff[u] = kOutOfRange;
      }
    }
  }
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int p = p_begin + row[r];
    pn[r] = p / HWo;
    const int rem = p - pn[r] * HWo;
    pho[r] = rem / g.Wo;
    pwo[r] = rem - pho[r] * g.Wo;
  }
  // advance of a pixel index by KP in (n, ho, wo) digits
  const int adv_n = KP / HWo, adv_r = KP - adv_n * HWo;
  const int adv_ho = adv_r / g.Wo, adv_wo = adv_r - adv_ho * g.Wo;
  const int cin_es = g.Cin * es, cout_es = g.Cout * es;

  int s_issue = 0;  // next stage to issue
  auto issue = [&](int buf) {
    const int p0 = p_begin + s_issue * KP;
    const int lim = p_end - p0;   // rows < lim are pixels of this split
    const uint32_t base = smem_lds + (uint32_t)(buf * STAGE_B);
#pragma unroll
    for (int u = 0; u < IPW; ++u) {
      const int r = ONE_ROW ? 0 : u;
      const int sub = RI % NW == 0 ? NW * u / RI : (NW / RI) * u + wave_u / RI;
      const int rq = RI % NW == 0 ? NW * u % RI + wave_u : wave_u % RI;
      uint32_t v;
      if (isA[u]) {
        const bool in = (row[u] < lim) & (coff[u] != kOutOfRange);
        v = in ? (uint32_t)((p0 + row[u]) * cout_es) + coff[u] : kOutOfRange;
      } else {
        const int hs = pho[r] * g.stride, ws = pwo[r] * g.stride;
        const bool in = (row[u] < lim) & (coff[u] != kOutOfRange) & ((unsigned)(hs + tdh[u]) < (unsigned)g.H) &
                        ((unsigned)(ws + tdw[u]) < (unsigned)g.W);
        v = in ? (uint32_t)(((pn[r] * g.H + hs) * g.W + ws) * cin_es) + coff[u] : kOutOfRange;
      }
      lds_dma16_buf(v, isA[u] ? rsA : rsB, base + (uint32_t)(sub * SUB_B + rq * 1024));
    }
    // carry the pixel coordinates to the next stage
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      int wo = pwo[r] + adv_wo, ho = pho[r] + adv_ho, n = pn[r] + adv_n;
      const bool cw = wo >= g.Wo;
      wo = cw ? wo - g.Wo : wo;
      ho = cw ? ho + 1 : ho;
      const bool ch = ho >= g.Ho;
      pwo[r] = wo;
      pho[r] = ch ? ho - g.Ho : ho;
      pn[r] = ch ? n + 1 : n;
    }
    ++s_issue;
  };

  floatx4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  const int S = p_end > p_begin ? (p_end - p_begin + KP - 1) / KP : 0;
#pragma unroll
  for (int q = 0; q < STAGES - 1; ++q)
    if (q < S) issue(q);
  const lds_char_t* lds = (const lds_char_t*)(lds_void_t)smem;
  // wave tile rows: channels [wm*WTM, +WTM) of the A sub-tiles; cols: [wn*WTN, +WTN) of B
  for (int s = 0; s < S; ++s) {
    wait_stage<IPW>(min(STAGES - 2, S - 1 - s));
    barrier_only();
    if (s + STAGES - 1 < S) issue((s + STAGES - 1) % STAGES);
    const lds_char_t* st = lds + (s % STAGES) * STAGE_B;
    // every operand read of the stage issues before its MFMAs, so later
    // k-steps' LDS latency hides behind earlier k-steps' MFMAs
    typename O::frag_t a[O::KSTEPS][FM], b[O::KSTEPS][FN];
#pragma unroll
    for (int kk = 0; kk < O::KSTEPS; ++kk) {
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int ch = wm * WTM + i * 16;
        a[kk][i] = O::frag(st + (ch / CPS) * SUB_B, ch % CPS, kk, lane);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int ch = wn * WTN + j * 16;
        b[kk][j] = O::frag(st + (SA + ch / CPS) * SUB_B, ch % CPS, kk, lane);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < O::KSTEPS; ++kk)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) O::mma(acc[i][j], a[kk][i], b[kk][j]);
  }
  wait_vmcnt<0>();

  float* __restrict__ P = g.P + (long)split * g.Cout * g.Kcols;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int kc = k0 + wn * WTN + j * 16 + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = co0 + wm * WTM + i * 16 + 4 * (lane >> 4) + r;
        if (co < g.Cout && kc < g.Kcols) P[(long)co * g.Kcols + kc] = acc[i][j][r];
      }
    }
}

// Sum of the split partials in a fixed order, written in OIHW order. A block
// covers 256 consecutive (co, tap, ci) elements as 64 float4 columns with 4
// groups of 64 threads; group q sums splits q, q+4, ... and the four sums are
// added in order, so the result is deterministic and the split axis is read
// in parallel with 16-byte loads.
__device__ inline void wgrad_store(float* __restrict__ out, long idx, float sum, int KHW, int Cin, int Cin_real,
                                   int s2d) {
  const int ci = (int)(idx % Cin);
  const long rest = idx / Cin;
  const int tap = (int)(rest % KHW);
  const int co = (int)(rest / KHW);
  if (s2d) {
    // 4x4 tap (a, b), channel (2*dy + dx)*3 + c  ->  7x7 tap (2a+dy-1, 2b+dx-1) of channel c
    if (ci < 12) {
      const int q = ci / 3, c = ci - 3 * q;
      const int kh = 2 * (tap >> 2) + (q >> 1) - 1, kw = 2 * (tap & 3) + (q & 1) - 1;
      if (kh >= 0 && kw >= 0) out[(((long)co * 3 + c) * 7 + kh) * 7 + kw] = sum;
    }
  } else if (ci < Cin_real) {
    out[((long)co * Cin_real + ci) * KHW + tap] = sum;
  }
}

__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float* __restrict__ P, int splits, int Cout,
                                                           int KHW, int Cin, int Cin_real, float* __restrict__ out,
                                                           int s2d) {
  __shared__ float4 part[4][64];
  const long total4 = (long)Cout * KHW * Cin / 4;   // Cin is a multiple of 4
  const int e = threadIdx.x & 63, q = threadIdx.x >> 6;
  const float4* __restrict__ P4 = (const float4*)P;
  for (long base = blockIdx.x * 64l; base < total4; base += (long)gridDim.x * 64) {
    const long idx = base + e;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (idx < total4) {
      int z = q;
      for (; z + 12 < splits; z += 16) {
        const float4 a = P4[z * total4 + idx], b = P4[(z + 4) * total4 + idx];
        const float4 c = P4[(z + 8) * total4 + idx], d = P4[(z + 12) * total4 + idx];
        acc.x += a.x; acc.y += a.y; acc.z += a.z; acc.w += a.w;
        acc.x += b.x; acc.y += b.y; acc.z += b.z; acc.w += b.w;
        acc.x += c.x; acc.y += c.y; acc.z += c.z; acc.w += c.w;
        acc.x += d.x; acc.y += d.y; acc.z += d.z; acc.w += d.w;
      }
      for (; z < splits; z += 4) {
        const float4 a = P4[z * total4 + idx];
        acc.x += a.x; acc.y += a.y; acc.z += a.z; acc.w += a.w;
      }
    }
    part[q][e] = acc;
    __syncthreads();
    if (q == 0 && idx < total4) {
      const float4 a = part[0][e], b = part[1][e], c = part[2][e], d = part[3][e];
      const float sum[4] = {((a.x + b.x) + c.x) + d.x, ((a.y + b.y) + c.y) + d.y, ((a.z + b.z) + c.z) + d.z,
                            ((a.w + b.w) + c.w) + d.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) wgrad_store(out, idx * 4 + k, sum[k], KHW, Cin, Cin_real, s2d);
    }
    __syncthreads();
  }
}

const void* zero_page() {
  static const void* zp[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  if (!zp[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_zero_page)) != hipSuccess) return nullptr;
    zp[dev] = p;
  }
  return zp[dev];
}

// The uniform K loop needs whole 128-byte channel blocks per tap, at most 32
// taps (one validity bit each) and buffers addressable with 31-bit offsets.
// With fewer channels than a row (kt), a row must be whole consecutive taps
// along w of a forward-ordered, stride-1 tap walk.
bool gather_uniform(const ConvGather& g, int kt) {
  const long es = 128 / kt;
  const int vw = 16 / (int)es;
  bool rows_ok;
  int groups = g.nth * g.ntw;
  if (g.Cin % kt == 0) {
    rows_ok = true;
  } else {
    const int rt = kt / g.Cin;
    rows_ok = g.Cin % vw == 0 && kt % g.Cin == 0 && g.ntw % rt == 0 && g.dws == 1 && g.wkws == 1;
    groups = g.nth * (g.ntw / (rows_ok ? rt : 1));
  }
  return rows_ok && groups <= 32 && (long)g.N * g.Hin * g.Win * g.Cin * es < (1l << 31) &&
         (long)g.Cols * g.KHW * g.Cin * es < (1l << 31);
}

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES>
int launch_gather2(const ConvGather& g0, hipStream_t s) {
  ConvGather g = g0;
  g.fd_hw = FastDiv((uint32_t)(g.Hm * g.Wm));
  g.fd_w = FastDiv((uint32_t)g.Wm);
  if ((long)g.N * g.Hout * g.Wout * g.Cols >= (1l << 31)) return -1;  // 32-bit output offsets
  g.zero = zero_page();
  if (!g.zero) return -4;
  const int tiles = ceil_div(g.M, BM) * ceil_div(g.Cols, BN);
  const int kt = 128 / (int)sizeof(T);
  const int nt = 64 * WGM * WGN;
  if (gather_uniform(g, kt))
    hipLaunchKernelGGL((conv_gather2_kernel<T, BM, BN, WGM, WGN, STAGES, true>), dim3(tiles), dim3(nt), 0, s, g);
  else
    hipLaunchKernelGGL((conv_gather2_kernel<T, BM, BN, WGM, WGN, STAGES, false>), dim3(tiles), dim3(nt), 0, s, g);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// Kernel configurations: id -> (BM, BN, waves along M, waves along N, stages).
#define RN18_GATHER_CONFIGS(X)                                                                   \
  X(1, 64, 32, 2, 2, 3) X(2, 64, 64, 2, 2, 3) X(3, 128, 64, 2, 2, 3) X(4, 128, 128, 2, 2, 3)     \
  X(5, 256, 128, 4, 2, 3) X(6, 256, 128, 2, 2, 3) X(7, 256, 64, 4, 2, 3) X(8, 128, 128, 2, 4, 3) \
  X(9, 256, 64, 4, 1, 3) X(10, 128, 128, 2, 2, 2) X(11, 256, 128, 4, 2, 2) X(12, 128, 64, 2, 2, 4) \
  X(13, 128, 64, 2, 2, 2) X(14, 64, 64, 2, 2, 2) X(15, 256, 64, 4, 2, 2) X(16, 128, 128, 2, 4, 2) \
  X(17, 256, 128, 2, 2, 2) X(18, 512, 64, 4, 1, 2) X(19, 256, 128, 2, 2, 3) X(20, 128, 128, 2, 2, 4) \
  X(21, 256, 64, 4, 1, 2) X(22, 256, 64, 2, 2, 2)
constexpr int kGatherCfgs = 22;
int g_gather_override = 0;

struct GatherCfg { int bm, bn, wgm, wgn, stages; };
constexpr GatherCfg kGather[kGatherCfgs + 1] = {
    {0, 0, 0, 0, 0},
#define RN18_X(id, bm, bn, wgm, wgn, st) {bm, bn, wgm, wgn, st},
    RN18_GATHER_CONFIGS(RN18_X)
#undef RN18_X
};

// Choice measured on MI355X over the ResNet-18 shapes (bf16 224x224 batch 256,
// fp32 32x32 batch 128): two-stage rings with two or more blocks per CU beat
// deeper rings with one block; 8-wave blocks for the large tiles.
int gather_cfg(const ConvGather& g) {
  if (g_gather_override) return g_gather_override;
  if (g.Cols <= 32) return 1;
  if (g.Cols <= 64) return g.M >= 131072 ? 15 : g.M >= 65536 ? 13 : 14;
  return (long)ceil_div(g.M, 128) * ceil_div(g.Cols, 128) >= 256 ? 16 : 14;
}

int gather_tile(const ConvGather& g) {
  const int id = gather_cfg(g);
  return id >= 1 && id <= kGatherCfgs ? kGather[id].bm * 1000 + kGather[id].bn : 0;
}

template <typename T>
int gather_dispatch(const ConvGather& g, hipStream_t s) {
  switch (gather_cfg(g)) {
#define RN18_X(id, bm, bn, wgm, wgn, st) \
  case id: return launch_gather2<T, bm, bn, wgm, wgn, st>(g, s);
    RN18_GATHER_CONFIGS(RN18_X)
#undef RN18_X
    default: return -1;
  }
}

template <typename T, int BM, int BN, int WGM, int WGN>
int launch_wgrad(const ConvWgrad& g, hipStream_t s) {
  const int tiles = ceil_div(g.Cout, BM) * ceil_div(g.Kcols, BN);
  hipLaunchKernelGGL((conv_wgrad_kernel<T, BM, BN, WGM, WGN>), dim3(tiles * g.splits), dim3(256), 0, s, g);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES>
int launch_wgrad2(const ConvWgrad& g, hipStream_t s) {
  const int tiles = ceil_div(g.Cout, BM) * ceil_div(g.Kcols, BN);
  hipLaunchKernelGGL((conv_wgrad2_kernel<T, BM, BN, WGM, WGN, STAGES>), dim3(tiles * g.splits), dim3(64 * WGM * WGN),
                     0, s, g);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// Weight-gradient configurations: id -> kernel, BM (output channels) x BN
// (tap x input channel columns), waves, stages.
//   1-3: register-transposing kernel 16x64, 64x64, 128x128
//   4: 64x128 1x4 s2   5: 64x128 2x2 s2   6: 128x128 2x2 s2   7: 128x128 2x2 s3
//   8: 64x64 2x2 s2    9: 128x64 2x2 s2  10: 128x128 2x4 s2
constexpr int kWgradCfgs = 10;
int g_wgrad_override = 0;

// Choice measured on MI355X (bf16 224x224 batch 256, fp32 32x32 batch 128).
int wgrad_cfg(int prec, int Cout, int Kcols) {
  if (g_wgrad_override) return g_wgrad_override;
  if (Cout <= 16) return 1;
  if (prec == PREC_BF16) {
    if (Cout <= 64) return 4;
    return Kcols <= 576 ? 9 : 10;
  }
  return Cout <= 64 ? 8 : 6;
}

void wgrad_tile(int prec, int Cout, int Kcols, int* bm, int* bn) {
  static const int tile[kWgradCfgs + 1][2] = {{0, 0},   {16, 64},  {64, 64},  {128, 128}, {64, 128}, {64, 128},
                                              {128, 128}, {128, 128}, {64, 64}, {128, 64},  {128, 128}};
  const int id = wgrad_cfg(prec, Cout, Kcols);
  *bm = tile[id][0];
  *bn = tile[id][1];
}

template <typename T>
int wgrad_dispatch(const ConvWgrad& g, hipStream_t s) {
  switch (wgrad_cfg(sizeof(T) == 2 ? PREC_BF16 : PREC_F32, g.Cout, g.Kcols)) {
    case 1: return launch_wgrad<T, 16, 64, 1, 4>(g, s);
    case 2: return launch_wgrad<T, 64, 64, 2, 2>(g, s);
    case 3: return launch_wgrad<T, 128, 128, 2, 2>(g, s);
    case 4: return launch_wgrad2<T, 64, 128, 1, 4, 2>(g, s);
    case 5: return launch_wgrad2<T, 64, 128, 2, 2, 2>(g, s);
    case 6: return launch_wgrad2<T, 128, 128, 2, 2, 2>(g, s);
    case 7: return launch_wgrad2<T, 128, 128, 2, 2, 3>(g, s);
    case 8: return launch_wgrad2<T, 64, 64, 2, 2, 2>(g, s);
    case 9: return launch_wgrad2<T, 128, 64, 2, 2, 2>(g, s);
    case 10: return launch_wgrad2<T, 128, 128, 2, 4, 2>(g, s);
    default: return -1;
  }
}

}  // namespace

namespace {

// Instance names as a profiler prints them (namespace dropped, the bf16
// storage type uint16_t written as bf16), interned for the life of the process.
const char* intern_name(const std::string& s) {
  static std::mutex mu;
  static std::set<std::string> names;
  std::lock_guard<std::mutex> lock(mu);
  return names.insert(s).first->c_str();
}

const char* type_name(int prec) { return prec == PREC_BF16 ? "bf16" : "float"; }

}  // namespace

const char* conv_gather_kernel_name(int prec, const ConvGather& g) {
  const int id = gather_cfg(g);
  if (id < 1 || id > kGatherCfgs) return "conv_gather2_kernel";
  const GatherCfg& c = kGather[id];
  const int kt = prec == PREC_BF16 ? 64 : 32;
  char buf[128];
  snprintf(buf, sizeof buf, "conv_gather2_kernel<%s, %d, %d, %d, %d, %d, %s>", type_name(prec), c.bm, c.bn, c.wgm,
           c.wgn, c.stages, gather_uniform(g, kt) ? "true" : "false");
  return intern_name(buf);
}

const char* conv_wgrad_kernel_name(int prec, int Cout, int Kcols) {
  static const int cfg[kWgradCfgs + 1][6] = {
      {0, 0, 0, 0, 0, 0},     {1, 16, 64, 1, 4, 0},   {1, 64, 64, 2, 2, 0},  {1, 128, 128, 2, 2, 0},
      {2, 64, 128, 1, 4, 2},  {2, 64, 128, 2, 2, 2},  {2, 128, 128, 2, 2, 2}, {2, 128, 128, 2, 2, 3},
      {2, 64, 64, 2, 2, 2},   {2, 128, 64, 2, 2, 2},  {2, 128, 128, 2, 4, 2}};
  const int id = wgrad_cfg(prec, Cout, Kcols);
  if (id < 1 || id > kWgradCfgs) return "conv_wgrad_kernel";
  const int* c = cfg[id];
  char buf[128];
  if (c[0] == 1)
    snprintf(buf, sizeof buf, "conv_wgrad_kernel<%s, %d, %d, %d, %d>", type_name(prec), c[1], c[2], c[3], c[4]);
  else
    snprintf(buf, sizeof buf, "conv_wgrad2_kernel<%s, %d, %d, %d, %d, %d>", type_name(prec), c[1], c[2], c[3], c[4],
             c[5]);
  return intern_name(buf);
}

const char* kernel_instance_name(const char* base, int prec) {
  return intern_name(std::string(base) + "<" + type_name(prec) + ">");
}

int conv_gather_tile(const ConvGather& g) { return gather_tile(g); }

int conv_gather_override(int id) {
  if (id < 0 || id > kGatherCfgs) return -1;
  g_gather_override = id;
  return 0;
}

int conv_wgrad_override(int id) {
  if (id < 0 || id > kWgradCfgs) return -1;
  g_wgrad_override = id;
  return 0;
}

int conv_wgrad_tile(int prec, int Cout, int Kcols) {
  int bm, bn;
  wgrad_tile(prec, Cout, Kcols, &bm, &bn);
  return bm * 1000 + bn;
}

int conv_gather_launch(int prec, const ConvGather& g, hipStream_t s) {
  if (g.M <= 0) return 0;
  return prec == PREC_BF16 ? gather_dispatch<bf16_t>(g, s) : gather_dispatch<float>(g, s);
}

int conv_wgrad_splits(int prec, int Cout, int Kcols, long Mpix, int* pix_per_split) {
  const int ktp = prec == PREC_BF16 ? 64 : 32;
  int bm, bn;
  wgrad_tile(prec, Cout, Kcols, &bm, &bn);
  const long tiles = (long)ceil_div(Cout, bm) * ceil_div(Kcols, bn);
  long splits = (1024 + tiles - 1) / tiles;
  const long per_split_bytes = (long)Cout * Kcols * 4;
  long max_by_bytes = (32l << 20) / per_split_bytes;
  if (max_by_bytes < 1) max_by_bytes = 1;
  long max_by_len = Mpix / (ktp * 8);
  if (max_by_len < 1) max_by_len = 1;
  if (splits > max_by_bytes) splits = max_by_bytes;
  if (splits > max_by_len) splits = max_by_len;
  if (splits < 1) splits = 1;
  long pps = (Mpix + splits - 1) / splits;
  pps = (pps + ktp - 1) / ktp * ktp;
  splits = (Mpix + pps - 1) / pps;
  if (splits < 1) splits = 1;
  *pix_per_split = (int)pps;
  return (int)splits;
}

int conv_wgrad_launch(int prec, const ConvWgrad& g, hipStream_t s) {
  // the pipelined kernels address both operands with 31-bit byte offsets
  const long es = prec == PREC_BF16 ? 2 : 4;
  if ((long)g.Mpix * g.Cout * es >= (1l << 31) || (long)g.N * g.H * g.W * g.Cin * es >= (1l << 31)) return -1;
  return prec == PREC_BF16 ? wgrad_dispatch<bf16_t>(g, s) : wgrad_dispatch<float>(g, s);
}

int wgrad_reduce_launch(const float* P, int splits, int Cout, int KHW, int Cin, int Cin_real,
                        float* out_oihw, int s2d, hipStream_t s) {
  if (s2d && (KHW != 16 || Cin != 16 || Cin_real != 3)) return -1;
  if (Cin % 4) return -1;
  const long total4 = (long)Cout * KHW * Cin / 4;
  int blocks = (int)((total4 + 63) / 64);
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(blocks), dim3(256), 0, s, P, splits, Cout, KHW, Cin, Cin_real,
                     out_oihw, s2d);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // namespace rn18
