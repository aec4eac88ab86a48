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
#include "pool.h"

#include <cstdio>
#include <mutex>
#include <set>
#include <string>

namespace rn18 {

namespace {

constexpr int RSTR = 9;  // LDS row stride in 16-byte units: 8 data chunks + 1 pad

template <typename T> struct Mma;
template <> struct Mma<bf16_t> {
  static constexpr int SUB = 1;
  __device__ static inline void run(floatx4_t& acc, const uint4& a, const uint4& b, int) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
  }
};
template <> struct Mma<f16_t> {
  static constexpr int SUB = 1;
  __device__ static inline void run(floatx4_t& acc, const uint4& a, const uint4& b, int) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), acc,
                                                 0, 0, 0);
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
// is multiplied. Rows are 128 bytes without padding; the chunk q of row r
// goes to slot q ^ ((r / 2) & 7). Consecutive rows sit in alternate halves of
// the 64 banks, so this puts the 16 rows of an MFMA operand read on 16
// distinct 16-byte bank groups (q ^ (r & 7) would pair rows r and r + 8 on
// one group). Taps outside the image and K beyond the end load
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

// One stored 16-byte output chunk (pk, at element offset off, channels c0 ..)
// into the BN backward partials of g.bstats: g = the stored value where the
// BN's ReLU passed, s1 += g, s2 += g * (y - mean) * rstd, the arithmetic of
// the standalone BN backward reduction.
template <typename T>
__device__ inline void bwd_partial_add(const ConvGather& g, const uint4& pk, uint32_t off, int c0,
                                       float (&s1)[TT<T>::VW], float (&s2)[TT<T>::VW]) {
  constexpr int VW = TT<T>::VW;
  float vr[VW], yy[VW];
  unpack<T>(pk, vr);
  unpack<T>(*(const uint4*)((const T*)g.by + off), yy);
  const uint32_t mb = g.bmask ? g.bmask[off / VW] : 0u;
  // four channels at a time: their constants as one 16-byte load each (c0 is a
  // multiple of VW), few registers live in the epilogue
#pragma unroll
  for (int q = 0; q < VW / 4; ++q) {
    const float4 mu = ((const float4*)(g.bmean + c0))[q], rs = ((const float4*)(g.brstd + c0))[q];
    const float m4[4] = {mu.x, mu.y, mu.z, mu.w}, r4[4] = {rs.x, rs.y, rs.z, rs.w};
    uint32_t mk = mb >> (4 * q);
    if (!g.bmask) {
      const float4 sc = ((const float4*)(g.bsc + c0))[q], sf = ((const float4*)(g.bsf + c0))[q];
      const float c4[4] = {sc.x, sc.y, sc.z, sc.w}, f4[4] = {sf.x, sf.y, sf.z, sf.w};
      mk = 0u;
#pragma unroll
      for (int t = 0; t < 4; ++t) mk |= relu_stored<T>(yy[4 * q + t], c4[t], f4[t]) > 0.f ? 1u << t : 0u;
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int e = 4 * q + t;
      const float gv = (mk >> t) & 1u ? vr[e] : 0.f;
      s1[e] += gv;
      s2[e] += gv * ((yy[e] - m4[t]) * r4[t]);
    }
  }
}

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES, bool UNI, bool RP>
__device__ inline void gather_impl(const ConvGather& g) {
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
  // split-K: logical block = range * tiles + tile, so the tiles of one K
  // range sit together on an XCD (they share operand rows of that range)
  const int ksplit = g.ksplit > 1 ? g.ksplit : 1;
  const int tiles = ((g.M + BM - 1) / BM) * tiles_n;
  const int tk = xcd_remap(blockIdx.x, gridDim.x);
  const int ks = ksplit > 1 ? tk / tiles : 0;
  const int t = tk - ks * tiles;
  const int m0 = (t / tiles_n) * BM, n0 = (t % tiles_n) * BN;
  const int S_all = (g.K + KT - 1) / KT;
  const int s_lo = ks * S_all / ksplit;            // this block's stages [s_lo, s_lo + S)
  const T* __restrict__ A = (const T*)g.A;
  const T* __restrict__ B = (const T*)g.B;
  const int HWm = g.Hm * g.Wm;
  // chunk this lane loads into slot lane & 7 of row 8 j + lane / 8 (j = wave
  // + NW u, of the wave's parity as NW and the A rows per stage are even)
  const int c = (lane & 7) ^ (((wave & 1) << 2) | (lane >> 4));
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
    // stage s is channel block s / (nth ntw_g), tap s % (nth ntw_g) (w group fastest)
    const int per_cb = g.nth * ntw_g;
    st_cb = s_lo / per_cb;
    st_ti = s_lo - st_cb * per_cb;
    st_th = st_ti / ntw_g;
    st_tw = st_ti - st_th * ntw_g;
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
    // taps inner, channel blocks outer: consecutive stages of a channel block
    // read input rows shifted by one tap, which L2 (and at times L1) still holds
    ++st_ti;
    if (++st_tw == ntw_g) {
      st_tw = 0;
      if (++st_th == g.nth) { st_th = 0; st_ti = 0; ++st_cb; }
    }
  };

  // General path (channel chunks of different taps in one row): per-lane tap
  // arithmetic and 64-bit addresses, padding read from the zero page.
  auto issue = [&](int s, int buf) {
    const int k = (s_lo + s) * KT + c * VW;
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

  const int S = (ks + 1) * S_all / ksplit - s_lo;
  const int arow0 = wm * WTM, brow0 = wn * WTN;
  const int sw = (lane >> 1) & 7;                 // (row / 2) % 8 of the operand rows
  if constexpr (RP) {
    // Register-prefetched loop: the operand fragments of stage s+1 are read
    // from LDS while the MFMAs of stage s run from registers, and a ring
    // buffer is refilled as soon as every wave has read it (before its
    // MFMAs), so all STAGES buffers are in flight.
    auto read_stage = [&](int s, uint4(&a)[2][FM], uint4(&b)[2][FN]) {
      const uint4* As = smem + (s % STAGES) * STAGE_U4;
      const uint4* Bs = As + BM * 8;
#pragma unroll
      for (int kg = 0; kg < 2; ++kg) {
        const int slot = (kg * 4 + (lane >> 4)) ^ sw;
#pragma unroll
        for (int i = 0; i < FM; ++i) a[kg][i] = As[(arow0 + i * 16 + (lane & 15)) * 8 + slot];
#pragma unroll
        for (int j = 0; j < FN; ++j) b[kg][j] = Bs[(brow0 + j * 16 + (lane & 15)) * 8 + slot];
      }
    };
    auto mma_regs = [&](const uint4(&a)[2][FM], const uint4(&b)[2][FN]) {
#pragma unroll
      for (int kg = 0; kg < 2; ++kg)
#pragma unroll
        for (int tt = 0; tt < Mma<T>::SUB; ++tt)
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) Mma<T>::run(acc[i][j], a[kg][i], b[kg][j], tt);
    };
    auto body = [&](int s, const uint4(&ac)[2][FM], const uint4(&bc)[2][FN], uint4(&an)[2][FM],
                    uint4(&bn)[2][FN]) {
      // stage s+1 must have landed; the stages after it may stay in flight
      if (s + 1 < S) wait_stage<IPW>(min(STAGES - 2, S - 2 - s));
      // this wave's reads of stage s are complete (s_waitcnt lgkmcnt(0))
      __builtin_amdgcn_s_waitcnt(0xC07F);
      barrier_only();
      if (s + STAGES < S) {
        if (UNI) issue_uni(s % STAGES);
        else issue(s + STAGES, s % STAGES);
      }
      if (s + 1 < S) read_stage(s + 1, an, bn);
      __builtin_amdgcn_sched_barrier(0);
      mma_regs(ac, bc);
      __builtin_amdgcn_sched_barrier(0);
    };
#pragma unroll
    for (int p = 0; p < STAGES; ++p)
      if (p < S) {
        if (UNI) issue_uni(p);
        else issue(p, p);
      }
    uint4 a0[2][FM], b0[2][FN], a1[2][FM], b1[2][FN];
    if (S > 0) {
      wait_stage<IPW>(min(STAGES - 1, S - 1));
      barrier_only();
      read_stage(0, a0, b0);
    }
    for (int s = 0; s < S; s += 2) {
      body(s, a0, b0, a1, b1);
      if (s + 1 < S) body(s + 1, a1, b1, a0, b0);
    }
  } else {
#pragma unroll
  for (int p = 0; p < STAGES - 1; ++p)
    if (p < S) {
      if (UNI) issue_uni(p);
      else issue(p, p);
    }
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
  // With g.bstats set (a data gradient entering a BN's backward pass), they
  // feed that BN's backward partials instead: sum g and sum g * xhat of the
  // stored values g where its ReLU passed, written as g.bstats[tile_m][col].
  float* Ws = (float*)smem + wave_u * 16 * WSTR;
  if (ksplit > 1) {
    // split-K: the raw fp32 tile of this K range, row m at m * Cols
    float* __restrict__ P = g.part + (size_t)ks * g.M * g.Cols;
    constexpr int C4 = WTN / 4;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) Ws[(4 * (lane >> 4) + r) * WSTR + j * 16 + (lane & 15)] = acc[i][j][r];
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      for (int idx = lane; idx < 16 * C4; idx += 64) {
        const int row = idx / C4, c4 = idx - row * C4;
        const int m = m0 + arow0 + i * 16 + row, col = n0 + brow0 + c4 * 4;
        if (m >= g.M || col >= g.Cols) continue;
        *(float4*)(P + (size_t)m * g.Cols + col) = *(const float4*)(Ws + row * WSTR + c4 * 4);
      }
    }
    return;
  }
  constexpr int CPW = WTN / VW;                    // chunks per strip row; a lane's chunk column is lane % CPW
  static_assert(64 % CPW == 0, "lane chunk column fixed across strips");
  T* __restrict__ Cg = (T*)g.C;
  const bool stats = g.stats != nullptr;
  const bool bstats = g.bstats != nullptr;
  float* Sh = (float*)smem + SM_EPI * 4;           // [BN] shifts, then [NW][64][ST_F] lane sums
  float* St = Sh + BN;
  float ssh[VW], ss1[VW], ss2[VW];
#pragma unroll
  for (int e = 0; e < VW; ++e) ssh[e] = ss1[e] = ss2[e] = 0.f;
  const int bc0 = n0 + brow0 + (lane % CPW) * VW;  // first channel of this lane's chunk column
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
        float rr[VW];
        unpack<T>(*(const uint4*)((const T*)g.R + off), rr);
        const uint32_t mk = ((const uint8_t*)g.Rm)[off / VW];    // mask byte of this 16-byte chunk
#pragma unroll
        for (int e = 0; e < VW; ++e) v[e] += (mk >> e) & 1u ? rr[e] : 0.f;
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
      } else if (bstats) {
        bwd_partial_add<T>(g, pk, off, bc0, ss1, ss2);
      }
    }
  }
  if (!stats && !bstats) return;
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
    if (bstats) ((float2*)g.bstats)[(long)(m0 / BM) * g.Cols + col] = make_float2(a1, a2);
    else ((float4*)g.stats)[(long)(m0 / BM) * g.Cols + col] = make_float4((float)rows, Sh[cl], a1, a2);
  }
}

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES, bool UNI>
__global__ __launch_bounds__(64 * WGM * WGN) void conv_gather2_kernel(ConvGather g) {
  gather_impl<T, BM, BN, WGM, WGN, STAGES, UNI, false>(g);
}
// Split-K reduce: the ksplit fp32 partial tiles of a gather launch summed in
// range order, then the gather epilogue on the sum (mode 0 store, 1
// accumulate, 2 masked residual; storage rounding). With g.stats set, the BN
// partials are written per block of SK_ROWS rows as (rows, shift, sum of
// v - shift, sum of squares), the shift being the block's first stored value
// of the channel, like the gather kernel's entries per tile; with g.bstats
// set, the BN backward partials of the stored values per block of rows.
constexpr int SK_ROWS = 32;   // GEMM rows per block (and per BN partial entry)
constexpr int SK_COLS = 64;   // output channels per block
template <typename T>
__global__ __launch_bounds__(256) void gather_splitk_reduce_kernel(ConvGather g) {
  constexpr int VW = TT<T>::VW;
  constexpr int CC = SK_COLS / VW;    // chunks per row
  constexpr int RL = 256 / CC;        // row lanes
  static_assert(RL <= SK_ROWS && SK_ROWS % RL == 0, "row lanes");
  __shared__ float red[RL][SK_COLS][2];
  __shared__ float shs[SK_COLS];
  const int tid = threadIdx.x, cc = tid % CC, rl = tid / CC;
  const int tiles_n = (g.Cols + SK_COLS - 1) / SK_COLS;
  const int bm = blockIdx.x / tiles_n, bn = blockIdx.x - bm * tiles_n;
  const int m0 = bm * SK_ROWS, col = bn * SK_COLS + cc * VW;
  const int rows = min(SK_ROWS, g.M - m0);
  const bool cok = col < g.Cols;
  const size_t slice = (size_t)g.M * g.Cols;
  const int HWm = g.Hm * g.Wm;
  T* __restrict__ Cg = (T*)g.C;
  auto sum_row = [&](int m, float (&v)[VW]) {
    const float* p = g.part + (size_t)m * g.Cols + col;
#pragma unroll
    for (int e = 0; e < VW; ++e) v[e] = 0.f;
    for (int k = 0; k < g.ksplit; ++k, p += slice) {
#pragma unroll
      for (int q = 0; q < VW / 4; ++q) {
        const float4 f = *(const float4*)(p + 4 * q);
        v[4 * q] += f.x; v[4 * q + 1] += f.y; v[4 * q + 2] += f.z; v[4 * q + 3] += f.w;
      }
    }
  };
  const bool stats = g.stats != nullptr, bstats = g.bstats != nullptr;
  float ssh[VW], s1[VW], s2[VW];
#pragma unroll
  for (int e = 0; e < VW; ++e) ssh[e] = s1[e] = s2[e] = 0.f;
  if (stats && cok) {
    float v[VW];
    sum_row(m0, v);
    unpack<T>(pack<T>(v), ssh);
  }
  if (cok) {
    for (int r = rl; r < rows; r += RL) {
      const int m = m0 + r;
      float v[VW];
      sum_row(m, v);
      const int n = (int)g.fd_hw.div(m), rem = m - n * HWm;
      const int ii = (int)g.fd_w.div(rem), jj = rem - ii * g.Wm;
      const uint32_t off = ((uint32_t)((n * g.Hout + ii * g.os + g.oph) * g.Wout + jj * g.os + g.opw)) * g.Cols + col;
      if (g.mode == 1) {
        float o[VW];
        unpack<T>(*(const uint4*)(Cg + off), o);
#pragma unroll
        for (int e = 0; e < VW; ++e) v[e] += o[e];
      } else if (g.mode == 2) {
        float rr[VW];
        unpack<T>(*(const uint4*)((const T*)g.R + off), rr);
        const uint32_t mk = ((const uint8_t*)g.Rm)[off / VW];
#pragma unroll
        for (int e = 0; e < VW; ++e) v[e] += (mk >> e) & 1u ? rr[e] : 0.f;
      }
      const uint4 pk = pack<T>(v);
      *(uint4*)(Cg + off) = pk;
      if (bstats) bwd_partial_add<T>(g, pk, off, col, s1, s2);
      if (stats) {
        float vr[VW];
        unpack<T>(pk, vr);
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          const float d = vr[e] - ssh[e];
          s1[e] += d;
          s2[e] = __builtin_fmaf(d, d, s2[e]);
        }
      }
    }
  }
  if (!stats && !bstats) return;
#pragma unroll
  for (int e = 0; e < VW; ++e) {
    red[rl][cc * VW + e][0] = s1[e];
    red[rl][cc * VW + e][1] = s2[e];
    if (rl == 0) shs[cc * VW + e] = ssh[e];
  }
  __syncthreads();
  if (tid < SK_COLS && bn * SK_COLS + tid < g.Cols) {
    float a1 = 0.f, a2 = 0.f;
    for (int k = 0; k < RL; ++k) { a1 += red[k][tid][0]; a2 += red[k][tid][1]; }
    const long at = (long)bm * g.Cols + bn * SK_COLS + tid;
    if (bstats) ((float2*)g.bstats)[at] = make_float2(a1, a2);
    else ((float4*)g.stats)[at] = make_float4((float)rows, shs[tid], a1, a2);
  }
}

// Blocks per CU that the LDS ring of a configuration allows (160 KB per CU),
// and the waves per SIMD they make; the register allocation of the kernels
// that use this is bounded to match.
constexpr int gather_blocks_per_cu(int bm, int bn, int stages) {
  const int b = 163840 / (stages * (bm + bn) * 128);
  return b < 1 ? 1 : b > 4 ? 4 : b;
}
constexpr int gather_occupancy(int bm, int bn, int nw, int stages) {
  const int w = gather_blocks_per_cu(bm, bn, stages) * nw / 4;
  return w < 1 ? 1 : w > 8 ? 8 : w;
}
template <typename T, int BM, int BN, int WGM, int WGN, int STAGES, bool UNI>
__global__ __launch_bounds__(64 * WGM * WGN, gather_occupancy(BM, BN, WGM * WGN, STAGES)) void conv_gather_rp_kernel(
    ConvGather g) {
  gather_impl<T, BM, BN, WGM, WGN, STAGES, UNI, true>(g);
}

// ---------------------------------------------------------------------------
// Persistent gather conv. A grid of at most as many blocks as fit on the chip
// walks a list of tiles (of up to four sub-problems of one launch, e.g. the
// four parity phases of a stride-2 data gradient): block b takes logical
// tiles b', b' + G, b' + 2G, ... (b' its XCD-contiguous slot). The K stages
// of consecutive tiles form one stream through the LDS ring, so the first
// stages of the next tile are loading while the current tile finishes its
// MFMAs and its epilogue. The epilogue stages its strips in the ring buffer
// of the stage consumed last, which no load targets until the next barrier.
// Only the uniform row layout (whole 128-byte channel blocks per tap, or
// whole groups of consecutive w taps) is handled here.
// ---------------------------------------------------------------------------
struct GatherSet {
  ConvGather p[4];
  int np;
  int tile_begin[5];  // sub-problem i owns logical tiles [tile_begin[i], tile_begin[i+1])
};

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES>
__global__ __launch_bounds__(64 * WGM * WGN, gather_occupancy(BM, BN, WGM * WGN, STAGES)) void conv_gather_ps_kernel(
    GatherSet gs) {
  constexpr int NW = WGM * WGN, NT = 64 * NW;
  constexpr int VW = TT<T>::VW;
  constexpr int KT = 128 / (int)sizeof(T);
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int AI = BM / 8, BI = BN / 8;
  constexpr int NI = AI + BI, IPW = NI / NW;
  constexpr int UA = AI / NW;
  constexpr int STAGE_U4 = (BM + BN) * 8;
  constexpr int WSTR = WTN + 4;
  constexpr int CPW = WTN / VW;
  constexpr int EPI_F = NW * 16 * WSTR + BN + NW * WTN * 2;
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
  static_assert(NI % NW == 0 && AI % NW == 0 && BN % 8 == 0, "whole load instructions per wave");
  static_assert(STAGES >= 2 && STAGES <= 4, "stages");
  static_assert(EPI_F * 4 <= STAGE_U4 * 16, "epilogue fits in one ring buffer");
  static_assert(64 % CPW == 0, "lane chunk column fixed across strips");
  __shared__ uint4 smem[STAGES * STAGE_U4];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave_u = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave_u / WGN, wn = wave_u % WGN;
  const int c = (lane & 7) ^ (((wave_u & 1) << 2) | (lane >> 4));   // see gather_impl
  const uint32_t smem_lds = lds_addr(smem);
  const int G = gridDim.x;
  const int slot = xcd_remap(blockIdx.x, G);
  const int total = gs.tile_begin[gs.np];
  const int es = (int)sizeof(T);
  const int arow0 = wm * WTM, brow0 = wn * WTN;
  const int sw = (lane >> 1) & 7;                 // (row / 2) % 8 of the operand rows

  // ---- issue side: the tile whose stages are being loaded
  constexpr int UB = IPW - UA;
  int is_tile = slot - G, is_s = 0, is_S = 0, is_S1 = 0;
  uint32_t uoff[IPW], umask[UA];
  uint32_t uoff2[UB], umask2 = 0;   // second K segment: B2 offsets, A2 row validity (bit u)
  i32x4_t rsA, rsB, rsA2, rsB2;
  int st_ti = 0, st_th = 0, st_tw = 0, st_cb = 0;
  int q_dh0 = 0, q_dhs = 0, q_dw0 = 0, q_dws = 0, q_wkh0 = 0, q_wkhs = 0, q_wkw0 = 0, q_wkws = 0;
  int q_KW = 0, q_Win = 0, q_Cin = 0, q_RT = 1, q_ntwg = 1, q_CB = 1;
  auto find_prob = [&](int t) {
    int pr = 0;
    while (pr + 1 < gs.np && t >= gs.tile_begin[pr + 1]) ++pr;
    return pr;
  };
  // advance the issue side to its next tile with at least one stage
  auto next_issue_tile = [&]() -> bool {
    for (;;) {
      is_tile += G;
      if (is_tile >= total) return false;
      const ConvGather& g = gs.p[find_prob(is_tile)];
      is_S1 = (g.K + KT - 1) / KT;
      is_S = is_S1 + g.K2 / KT;
      is_s = 0;
      if (is_S == 0) continue;
      const int pr = find_prob(is_tile);
      const int lt = is_tile - gs.tile_begin[pr];
      const int tiles_n = (g.Cols + BN - 1) / BN;
      const int m0 = (lt / tiles_n) * BM, n0 = (lt - (lt / tiles_n) * tiles_n) * BN;
      const int HWm = g.Hm * g.Wm;
      q_dh0 = g.dh0; q_dhs = g.dhs; q_dw0 = g.dw0; q_dws = g.dws;
      q_wkh0 = g.wkh0; q_wkhs = g.wkhs; q_wkw0 = g.wkw0; q_wkws = g.wkws;
      q_KW = g.KW; q_Win = g.Win; q_Cin = g.Cin;
      q_CB = g.Cin >= KT ? g.Cin / KT : 1;
      q_RT = g.Cin < KT ? KT / g.Cin : 1;
      q_ntwg = g.ntw / q_RT;
      rsA = buffer_rsrc(g.A, (uint32_t)((long)g.N * g.Hin * g.Win * g.Cin * es));
      rsB = buffer_rsrc(g.B, (uint32_t)((long)g.Cols * g.KHW * g.Cin * es));
      const int lane_px = (c * VW) / g.Cin;
      umask2 = 0;
#pragma unroll
      for (int u = 0; u < UA; ++u) {
        const int m = m0 + (wave_u + NW * u) * 8 + (lane >> 3);
        const bool ok = m < g.M;
        const int mm = ok ? m : 0;
        const int n = (int)g.fd_hw.div(mm), rem = mm - n * HWm;
        const int i = (int)g.fd_w.div(rem), jj = rem - i * g.Wm;
        const int hb = i * g.is - g.ip, wb = jj * g.is - g.ip;
        uint32_t vh = 0, vw = 0, msk = 0;
        for (int th = 0; th < g.nth; ++th)
          vh |= (unsigned)(hb + g.dh0 + th * g.dhs) < (unsigned)g.Hin ? 1u << th : 0u;
        for (int tg = 0; tg < q_ntwg; ++tg)
          vw |= (unsigned)(wb + g.dw0 + (tg * q_RT + lane_px) * g.dws) < (unsigned)g.Win ? 1u << tg : 0u;
        for (int th = 0; th < g.nth; ++th) msk |= (vh >> th) & 1u ? vw << (th * q_ntwg) : 0u;
        umask[u] = ok ? msk : 0u;
        uoff[u] = (uint32_t)(((n * g.Hin + hb) * g.Win + wb) * g.Cin * es + c * 16);
        if (ok && (unsigned)hb < (unsigned)g.Hin && (unsigned)wb < (unsigned)g.Win) umask2 |= 1u << u;
      }
#pragma unroll
      for (int u = UA; u < IPW; ++u) {
        const int col = n0 + (wave_u + NW * u - AI) * 8 + (lane >> 3);
        uoff[u] = col < g.Cols ? (uint32_t)((long)col * g.KHW * g.Cin * es + c * 16) : kOutOfRange;
        uoff2[u - UA] = col < g.Cols ? (uint32_t)((long)col * g.Cin * es + c * 16) : kOutOfRange;
      }
      if (g.K2 > 0) {
        rsA2 = buffer_rsrc(g.A2, (uint32_t)((long)g.N * g.Hin * g.Win * g.Cin * es));
        rsB2 = buffer_rsrc(g.B2, (uint32_t)((long)g.Cols * g.Cin * es));
      }
      st_ti = st_th = st_tw = st_cb = 0;
      return true;
    }
  };
  int n_issued = 0;
  bool more = next_issue_tile();
  // issue the next stage of the stream into its ring buffer; false when the stream has ended
  auto issue_next = [&]() {
    if (!more) return;
    const uint32_t base =
        __builtin_amdgcn_readfirstlane(smem_lds + (uint32_t)((n_issued % STAGES) * STAGE_U4 * 16));
    if (is_s >= is_S1) {
      // second K segment: channel block is_s - is_S1 of A2 at the row's own pixel, and of B2
      const uint32_t s2 = (uint32_t)((is_s - is_S1) * 128);
#pragma unroll
      for (int u = 0; u < UA; ++u) {
        const uint32_t v = (umask2 >> u) & 1u ? uoff[u] + s2 : kOutOfRange;
        lds_dma16_buf(v, rsA2, base + (uint32_t)((wave_u + NW * u) * 1024));
      }
#pragma unroll
      for (int u = UA; u < IPW; ++u) {
        const uint32_t v = uoff2[u - UA] == kOutOfRange ? kOutOfRange : uoff2[u - UA] + s2;
        lds_dma16_buf(v, rsB2, base + (uint32_t)((AI + wave_u + NW * (u - UA)) * 1024));
      }
    } else {
      const int dh = q_dh0 + st_th * q_dhs, dw = q_dw0 + st_tw * q_RT * q_dws;
      const int wt = (q_wkh0 + st_th * q_wkhs) * q_KW + q_wkw0 + st_tw * q_RT * q_wkws;
      const uint32_t sa = (uint32_t)((dh * q_Win + dw) * q_Cin * es + st_cb * 128);
      const uint32_t sb = (uint32_t)(wt * q_Cin * es + st_cb * 128);
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
      if (++st_cb == q_CB) {
        st_cb = 0;
        ++st_ti;
        if (++st_tw == q_ntwg) { st_tw = 0; ++st_th; }
      }
    }
    ++n_issued;
    if (++is_s == is_S) more = next_issue_tile();
  };

  for (int p = 0; p < STAGES - 1; ++p) issue_next();

  // ---- compute side
  int q = 0;  // stages consumed so far
  for (int tile = slot; tile < total; tile += G) {
    const int pr = find_prob(tile);
    const ConvGather& g = gs.p[pr];
    const int S = (g.K + KT - 1) / KT + g.K2 / KT;
    floatx4_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < S; ++s, ++q) {
      wait_stage<IPW>(n_issued - 1 - q);
      barrier_only();
      while (more && n_issued < q + STAGES) issue_next();
      const uint4* As = smem + (q % STAGES) * STAGE_U4;
      const uint4* Bs = As + BM * 8;
      uint4 a[2][FM], b[2][FN];
#pragma unroll
      for (int kg = 0; kg < 2; ++kg) {
        const int sl = (kg * 4 + (lane >> 4)) ^ sw;
#pragma unroll
        for (int i = 0; i < FM; ++i) a[kg][i] = As[(arow0 + i * 16 + (lane & 15)) * 8 + sl];
#pragma unroll
        for (int j = 0; j < FN; ++j) b[kg][j] = Bs[(brow0 + j * 16 + (lane & 15)) * 8 + sl];
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kg = 0; kg < 2; ++kg)
#pragma unroll
        for (int tt = 0; tt < Mma<T>::SUB; ++tt)
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) Mma<T>::run(acc[i][j], a[kg][i], b[kg][j], tt);
    }

    // ---- epilogue of this tile, staged in the ring buffer of the last consumed stage
    const int lt = tile - gs.tile_begin[pr];
    const int tiles_n = (g.Cols + BN - 1) / BN;
    const int tm = lt / tiles_n;
    const int m0 = tm * BM, n0 = (lt - tm * tiles_n) * BN;
    const int HWm = g.Hm * g.Wm;
    float* E = (float*)(smem + ((q + STAGES - 1) % STAGES) * STAGE_U4);
    float* Ws = E + wave_u * 16 * WSTR;
    float* Sh = E + NW * 16 * WSTR;
    float* Sp = Sh + BN;
    T* __restrict__ Cg = (T*)g.C;
    const bool stats = g.stats != nullptr, bstats = g.bstats != nullptr;
    barrier_only();  // every wave is done with the stage data in E
    float ssh[VW], ss1[VW], ss2[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) ssh[e] = ss1[e] = ss2[e] = 0.f;
    const int cc = lane % CPW;
    if (stats) {
      if (wm == 0 && lane < 16) {
#pragma unroll
        for (int j = 0; j < FN; ++j) Sh[brow0 + j * 16 + lane] = TT<T>::to_f(TT<T>::from_f(acc[0][j][0]));
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      barrier_only();
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
        const int row = idx / CPW;
        const int m = m0 + arow0 + i * 16 + row, col = n0 + brow0 + cc * VW;
        if (m >= g.M || col >= g.Cols) continue;
        const int n = (int)g.fd_hw.div(m), rem = m - n * HWm;
        const int ii = (int)g.fd_w.div(rem), jj = rem - ii * g.Wm;
        const uint32_t off =
            ((uint32_t)((n * g.Hout + ii * g.os + g.oph) * g.Wout + jj * g.os + g.opw)) * g.Cols + col;
        float v[VW];
#pragma unroll
        for (int e = 0; e < VW; ++e) v[e] = Ws[row * WSTR + cc * VW + e];
        if (g.mode == 1) {
          float o[VW];
          unpack<T>(*(const uint4*)(Cg + off), o);
#pragma unroll
          for (int e = 0; e < VW; ++e) v[e] += o[e];
        } else if (g.mode == 2) {
          float rr[VW];
          unpack<T>(*(const uint4*)((const T*)g.R + off), rr);
          const uint32_t mk = ((const uint8_t*)g.Rm)[off / VW];  // mask byte of this 16-byte chunk
#pragma unroll
          for (int e = 0; e < VW; ++e) v[e] += (mk >> e) & 1u ? rr[e] : 0.f;
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
        } else if (bstats) {
          bwd_partial_add<T>(g, pk, off, col, ss1, ss2);
        }
      }
    }
    if (stats || bstats) {
      // lanes with the same chunk column hold the same channels: butterfly sum
#pragma unroll
      for (int d = CPW; d < 64; d <<= 1)
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          ss1[e] += __shfl_xor(ss1[e], d);
          ss2[e] += __shfl_xor(ss2[e], d);
        }
      if (lane < CPW) {
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          Sp[(wave_u * WTN + lane * VW + e) * 2] = ss1[e];
          Sp[(wave_u * WTN + lane * VW + e) * 2 + 1] = ss2[e];
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      barrier_only();
      const int rows = min(BM, g.M - m0);
      for (int cl = tid; cl < BN; cl += NT) {
        const int col = n0 + cl;
        if (col >= g.Cols) continue;
        const int wn_c = cl / WTN, cw = cl - wn_c * WTN;
        float a1 = 0.f, a2 = 0.f;
        for (int wmi = 0; wmi < WGM; ++wmi) {
          a1 += Sp[((wmi * WGN + wn_c) * WTN + cw) * 2];
          a2 += Sp[((wmi * WGN + wn_c) * WTN + cw) * 2 + 1];
        }
        if (bstats) {
          // the sub-problems' row tiles follow one another in the entries
          const long row = gs.tile_begin[pr] / tiles_n + tm;
          ((float2*)g.bstats)[row * g.Cols + col] = make_float2(a1, a2);
        } else {
          ((float4*)g.stats)[(long)tm * g.Cols + col] = make_float4((float)rows, Sh[cl], a1, a2);
        }
      }
    }
  }
  wait_vmcnt<0>();
}

// ---------------------------------------------------------------------------
// Halo conv for the 64 -> 64 channel 3x3 stride-1 convolutions (bf16): the
// forward pass and the data gradient of the first stage. The whole weight
// matrix [9 taps][64 columns][64 channels] (72 KB) stays in LDS for the
// launch. A tile is up to TH whole output rows of one image (up to 512
// pixels); its input patch, (TH + 2) x (W + 2) pixels with a zero halo, is
// loaded into LDS one 32-channel half at a time and all nine taps read it
// at a fixed pixel offset, so an input pixel crosses from L2 about
// (TH + 2)(W + 2) / (TH W) times instead of nine. Half-patches are
// double-buffered: the next one loads while the current one is multiplied.
// Eight waves (two per SIMD, for LDS throughput) each own 64 pixels x 64
// columns; the operand fragments of the next K step are read while the
// MFMAs of the current one run.
// LDS rows are swizzled so that an MFMA operand read (16 consecutive rows,
// four 16-byte chunks of each) runs without bank conflicts: 128-byte weight
// rows by (row / 2) mod 8, 64-byte patch rows by (row / 2) mod 4. (Measured
// with ds_read_b128 on gfx950 at 8 waves per CU: these take 5.1-5.2 cycles
// per read at every row offset; the (row / 4) mod 4 patch swizzle, or none,
// takes 8.)
// The MFMAs take the weights as their first operand, so a lane's
// accumulators are 4 consecutive output channels of one pixel: the epilogue
// stores them as 8-byte chunks straight from registers. The BN partial
// statistics of the stored values accumulate per lane over all of a wave's
// tiles and are reduced over the lanes once at the end: one statistics entry
// per wave of the grid.
// ---------------------------------------------------------------------------
struct ConvHalo {
  ConvGather g;
  int TH;          // output rows per tile
  int PH, PW;      // patch rows and columns
  int tiles_img;   // ceil(Hm / TH)
  int tiles;       // N * tiles_img
};

constexpr int HALO_PROWS = 640;  // patch pixels per half-patch buffer
constexpr int HALO_WAVES = 8;    // waves per block = statistics entries per block
constexpr int HALO_BM = 64 * HALO_WAVES;

template <typename T, int MODE, bool STATS>
__global__ __launch_bounds__(64 * HALO_WAVES, 1) void conv_halo_kernel(ConvHalo h) {
  constexpr int NW = HALO_WAVES, FM = 4, FN = 4;
  constexpr int B_U4 = 9 * 64 * 8;                  // resident weights, uint4 units (128-byte rows)
  constexpr int P_U4 = HALO_PROWS * 4;              // one half-patch buffer (64-byte rows)
  constexpr int PI = HALO_PROWS / 16 / NW;          // half-patch load instructions per wave (16 rows each)
  constexpr int BI = 9 * 64 / 8 / NW;               // weight load instructions per wave (8 rows each)
  constexpr int kResidualLoads = MODE == 0 ? 0 : FM * FN * (MODE == 2 ? 2 : 1);   // per wave and tile
  static_assert(kResidualLoads < 64, "vmcnt range");
  __shared__ uint4 smem[B_U4 + 2 * P_U4];
  static_assert((B_U4 + 2 * P_U4) * 16 <= 163840, "LDS");
  static_assert(HALO_PROWS % (16 * NW) == 0 && (9 * 64) % (8 * NW) == 0, "whole load instructions per wave");
  const ConvGather& g = h.g;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t smem_lds = lds_addr(smem);
  const int rowb = g.Cin * 2;                        // 128 bytes per pixel or weight tap
  const i32x4_t rsA = buffer_rsrc(g.A, (uint32_t)((long)g.N * g.Hin * g.Win * rowb));
  const i32x4_t rsB = buffer_rsrc(g.B, (uint32_t)((long)g.Cols * g.KHW * rowb));
  const int G = gridDim.x;
  const int slot = xcd_remap(blockIdx.x, G);

  // weights: row r = tap * 64 + column (tap = th * 3 + tw in the walk
  // order); the lane's 16 bytes go to slot lane % 8 and hold chunk
  // (lane % 8) ^ ((r / 2) % 8)
#pragma unroll
  for (int u = 0; u < BI; ++u) {
    const int r = (wave + NW * u) * 8 + (lane >> 3);
    const int t = r >> 6, col = r & 63, th = t / 3, tw = t - th * 3;
    const int wt = (g.wkh0 + th * g.wkhs) * g.KW + g.wkw0 + tw * g.wkws;
    const int c = (lane & 7) ^ ((r >> 1) & 7);
    lds_dma16_buf((uint32_t)((col * g.KHW + wt) * rowb + c * 16), rsB,
                  smem_lds + (uint32_t)((wave + NW * u) * 1024));
  }
  // half-patch load geometry: row p = patch pixel; the lane's 16 bytes go to
  // slot lane % 4 and hold chunk (lane % 4) ^ ((p / 2) % 4) of the half
  int prel[PI], prow[PI];
#pragma unroll
  for (int u = 0; u < PI; ++u) {
    const int p = (wave + NW * u) * 16 + (lane >> 2);
    const int pr = p / h.PW, pc = p - pr * h.PW;
    const int ir = -g.ip + g.dh0 + pr, ic = -g.ip + g.dw0 + pc;   // input row (relative to i0) and column
    const bool ok = p < h.PH * h.PW && (unsigned)ic < (unsigned)g.Win;
    const int c = (lane & 3) ^ ((p >> 1) & 3);
    prel[u] = (ir * g.Win + ic) * rowb + c * 16;
    prow[u] = ok ? ir : -0x40000000;
  }
  auto issue_patch = [&](int tile, int half, int buf) {
    const int n = tile / h.tiles_img, i0 = (tile - n * h.tiles_img) * h.TH;
    const int base = (n * g.Hin + i0) * g.Win * rowb + half * 64;
    const uint32_t lbase = smem_lds + (uint32_t)((B_U4 + buf * P_U4) * 16);
#pragma unroll
    for (int u = 0; u < PI; ++u) {
      const bool ok = (unsigned)(i0 + prow[u]) < (unsigned)g.Hin;
      lds_dma16_buf(ok ? (uint32_t)(base + prel[u]) : kOutOfRange, rsA, lbase + (uint32_t)((wave + NW * u) * 1024));
    }
  };
  // A operand rows of this lane: tile pixel q -> patch pixel of tap (0, 0)
  int abase[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int q = wave * 64 + i * 16 + (lane & 15);
    const int ti = (int)g.fd_w.div(q);
    abase[i] = ti * h.PW + (q - ti * g.Wm);
  }
  const int kq = lane >> 4;
  const int chl = 4 * (lane >> 4);                   // first of this lane's 4 channels within a 16-column block
  const int wsw = (lane >> 1) & 7;                   // weight rows: (row / 2) % 8 == (lane % 16) / 2
  T* __restrict__ Cg = (T*)g.C;
  // output and residual operands as buffers: lanes of pixels beyond the tile
  // use an out-of-range offset (loads read zeros, stores are dropped), so
  // every tile issues the same number of vector memory instructions
  const uint32_t out_bytes = (uint32_t)((long)g.N * g.Hout * g.Wout * g.Cols * 2);
  const __amdgpu_buffer_rsrc_t rsC = __builtin_amdgcn_make_buffer_rsrc(g.C, 0, out_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsR = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(g.mode == 1 || !g.R ? (const void*)g.C : g.R), 0, out_bytes, 0x00020000);
  // ReLU mask bytes of the residual: one byte per 8 output elements
  const __amdgpu_buffer_rsrc_t rsRm = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(g.Rm ? g.Rm : (const void*)g.C), 0, out_bytes / 16, 0x00020000);

  // running BN partial statistics of this lane's 16 channels over the wave's pixels
  float s1[FN][4], s2[FN][4], sh[FN][4];
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) s1[j][e] = s2[j][e] = sh[j][e] = 0.f;
  bool have_shift = false;
  int rows_acc = 0;

  // phases: (tile, half) in order; phase k uses buffer k % 2
  if (slot < h.tiles) issue_patch(slot, 0, 0);
  int buf = 0;
  for (int tile = slot; tile < h.tiles; tile += G) {
    const int n = tile / h.tiles_img, i0 = (tile - n * h.tiles_img) * h.TH;
    const int npx = min(h.TH, g.Hm - i0) * g.Wm;    // output pixels of this tile
    const long m0 = ((long)n * g.Hm + i0) * g.Wm;    // GEMM row of the tile's first pixel
    uint32_t obase[FM];
    bool okq[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int q = wave * 64 + i * 16 + (lane & 15);
      okq[i] = q < npx;
      obase[i] = (uint32_t)((m0 + (okq[i] ? q : 0)) * g.Cols) + chl;
    }
    // residual operands of modes 1 and 2, requested during the first half so
    // that they have landed by the epilogue
    typedef int i32x2_t __attribute__((ext_vector_type(2)));
    i32x2_t ld0[MODE ? FM : 1][FN];
    uint32_t ld1[MODE == 2 ? FM : 1][FN];
    floatx4_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int half = 0; half < 2; ++half, buf ^= 1) {
      // this half-patch has landed. Vector memory operations complete in
      // issue order. After the first half of a tile was requested, only the
      // previous tile's epilogue issued vector memory instructions: exactly
      // FM * FN stores, which may stay in flight. After the second half was
      // requested, only the tile's own residual loads were issued: at least
      // kResidualLoads instructions (their addresses are 32 and 2 bytes apart,
      // so none merge; the compiler splits some masked ones in two), so
      // waiting down to that many leaves the patch landed.
      if (half == 0 && tile != slot) wait_vmcnt<FM * FN>();
      else if (half == 1) wait_vmcnt<kResidualLoads>();
      else wait_vmcnt<0>();
      barrier_only();
      if (half == 0) {
        issue_patch(tile, 1, buf ^ 1);
        if constexpr (MODE != 0) {
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) {
              const uint32_t ob = okq[i] ? (obase[i] + j * 16) * 2 : kOutOfRange;
              ld0[i][j] = __builtin_amdgcn_raw_buffer_load_b64(rsR, ob, 0, 0);
              if constexpr (MODE == 2)
                ld1[i][j] = __builtin_amdgcn_raw_buffer_load_b8(
                    rsRm, okq[i] ? (obase[i] + j * 16) >> 3 : kOutOfRange, 0, 0);
            }
        }
      } else if (tile + G < h.tiles) {
        issue_patch(tile + G, 0, buf ^ 1);
      }
      const uint4* P = smem + B_U4 + buf * P_U4;
      // the patch width is made opaque here so that the operand addresses are
      // recomputed per phase rather than held in registers across phases
      int pw = h.PW;
      asm volatile("" : "+s"(pw));
      // K step t: tap t (th, tw), this half's 32 channels
      auto read_step = [&](int t, uint4(&a)[FM], uint4(&b)[FN]) {
        const int th = t / 3, tw = t - th * 3;
        const int off = th * pw + tw;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          const int pix = abase[i] + off;
          a[i] = P[pix * 4 + (kq ^ ((pix >> 1) & 3))];
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) b[j] = smem[(t * 64 + j * 16 + (lane & 15)) * 8 + ((half * 4 + kq) ^ wsw)];
      };
      uint4 a0[FM], b0[FN], a1[FM], b1[FN];
      read_step(0, a0, b0);
#pragma unroll
      for (int t = 0; t < 9; t += 2) {
        if (t + 1 < 9) read_step(t + 1, a1, b1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j) Mma<T>::run(acc[i][j], b0[j], a0[i], 0);
        __builtin_amdgcn_sched_barrier(0);
        if (t + 1 < 9) {
          if (t + 2 < 9) read_step(t + 2, a0, b0);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) Mma<T>::run(acc[i][j], b1[j], a1[i], 0);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    // every wave must be done with the patch buffers before they are reloaded
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");

    // ---- epilogue straight from registers
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        float x[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        if constexpr (MODE != 0) {
          const uint32_t rw[2] = {(uint32_t)ld0[i][j].x, (uint32_t)ld0[i][j].y};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float rv = s16_to_f<T>((uint16_t)(e & 1 ? rw[e >> 1] >> 16 : rw[e >> 1] & 0xffffu));
            if constexpr (MODE == 2) {
              // this lane's 4 channels are the low or high half of the byte
              x[e] += (ld1[i][j] >> ((chl & 4) + e)) & 1u ? rv : 0.f;
            } else {
              x[e] += rv;
            }
          }
        }
        const uint2 pk = make_uint2(pack2<T>(x[0], x[1]), pack2<T>(x[2], x[3]));
        __builtin_amdgcn_raw_buffer_store_b64(i32x2_t{(int)pk.x, (int)pk.y}, rsC,
                                              okq[i] ? (obase[i] + j * 16) * 2 : kOutOfRange, 0, 0);
        if constexpr (STATS) {
          const float vr[4] = {s16_to_f<T>((uint16_t)(pk.x & 0xffffu)), s16_to_f<T>((uint16_t)(pk.x >> 16)),
                               s16_to_f<T>((uint16_t)(pk.y & 0xffffu)), s16_to_f<T>((uint16_t)(pk.y >> 16))};
          if (!have_shift && i == 0) {
            // the wave's first pixel (of its first tile) is its statistics shift
#pragma unroll
            for (int e = 0; e < 4; ++e) sh[j][e] = __shfl(vr[e], lane & 48, 64);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float d = okq[i] ? vr[e] - sh[j][e] : 0.f;
            s1[j][e] += d;
            s2[j][e] = __builtin_fmaf(d, d, s2[j][e]);
          }
        }
      }
    if (wave * 64 < npx) {
      have_shift = true;
      rows_acc += min(64, npx - wave * 64);
    }
  }
  if (STATS && slot < h.tiles) {
    // one entry per wave: its pixels over all of its tiles, shifted by the
    // first one; the sums over the 16 pixels of a lane row are shuffled
    // together, then each lane writes one channel
    const int kk = lane & 15, jj = kk >> 2, rr = kk & 3;
    float o1 = 0.f, o2 = 0.f, osh = 0.f;
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float a1 = s1[j][r], a2 = s2[j][r];
#pragma unroll
        for (int dd = 1; dd < 16; dd <<= 1) {
          a1 += __shfl_xor(a1, dd, 16);
          a2 += __shfl_xor(a2, dd, 16);
        }
        if (j == jj && r == rr) { o1 = a1; o2 = a2; osh = sh[j][r]; }
      }
    float4* out = (float4*)g.stats + ((long)(blockIdx.x * NW + wave) * g.Cols + jj * 16 + chl + rr);
    *out = rows_acc > 0 ? make_float4((float)rows_acc, osh, o1, o2) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  wait_vmcnt<0>();
}

// ---------------------------------------------------------------------------
// Halo conv for the space-to-depth stem: 16 input channels (32-byte pixels),
// a 4x4 stride-1 forward tap walk, 64 output channels (bf16). Same scheme as
// the 64-channel halo kernel: the weights [16 taps][64 columns][16 channels]
// (32 KB) stay in LDS, a tile is up to 256 pixels of whole output rows, and
// its input patch (TH + 3) x (W + 3) pixels is loaded once (double-buffered)
// for all sixteen taps. Blocks of 4 waves use 72 KB of LDS, so two share a
// CU and one block's epilogue (stores and statistics) overlaps the other's
// MFMAs. A K step of 32 covers two taps of the same tap row;
// the lane group kq reads tap 2 * (step % 2) + kq / 2, channels 8 (kq % 2) ..
// +8. LDS rows of 32 bytes are not swizzled: an operand read (16 consecutive
// rows, both halves) is conflict-free as laid out (measured on gfx950 with
// ds_read_b128 at 8 waves per CU: 5.1-5.2 cycles per read at every row
// offset, where a (row / 8) mod 2 swizzle takes 8).
// ---------------------------------------------------------------------------
constexpr int HALO16_PROWS = 640;   // patch pixels per buffer
constexpr int HALO16_WAVES = 4;     // waves per block; two blocks per CU overlap each other's epilogues
constexpr int HALO16_BM = 64 * HALO16_WAVES;

template <typename T, bool STATS>
__global__ __launch_bounds__(64 * HALO16_WAVES, 2) void conv_halo16_kernel(ConvHalo h) {
  typedef int i32x2_t __attribute__((ext_vector_type(2)));
  constexpr int NW = HALO16_WAVES, FM = 4, FN = 4;
  constexpr int B_U4 = 16 * 64 * 2;                 // resident weights, uint4 units (32-byte rows)
  constexpr int P_U4 = HALO16_PROWS * 2;            // one patch buffer
  constexpr int PI = HALO16_PROWS / 32 / NW;        // patch load instructions per wave (32 rows each)
  constexpr int BI = 16 * 64 / 32 / NW;             // weight load instructions per wave
  __shared__ uint4 smem[B_U4 + 2 * P_U4];
  static_assert((B_U4 + 2 * P_U4) * 16 * 2 <= 163840, "two blocks per CU");
  static_assert(HALO16_PROWS % (32 * NW) == 0 && (16 * 64) % (32 * NW) == 0, "whole load instructions per wave");
  const ConvGather& g = h.g;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t smem_lds = lds_addr(smem);
  const i32x4_t rsA = buffer_rsrc(g.A, (uint32_t)((long)g.N * g.Hin * g.Win * 32));
  const i32x4_t rsB = buffer_rsrc(g.B, (uint32_t)((long)g.Cols * 16 * 32));
  const int G = gridDim.x;
  const int slot = xcd_remap(blockIdx.x, G);

  // weights: row r = tap * 64 + column; the lane's 16 bytes go to slot
  // lane % 2 and hold half lane % 2 of the tap's channels
#pragma unroll
  for (int u = 0; u < BI; ++u) {
    const int r = (wave + NW * u) * 32 + (lane >> 1);
    const int t = r >> 6, col = r & 63;
    const int c = lane & 1;
    lds_dma16_buf((uint32_t)((col * 16 + t) * 32 + c * 16), rsB, smem_lds + (uint32_t)((wave + NW * u) * 1024));
  }
  int prel[PI], prow[PI];
#pragma unroll
  for (int u = 0; u < PI; ++u) {
    const int p = (wave + NW * u) * 32 + (lane >> 1);
    const int pr = p / h.PW, pc = p - pr * h.PW;
    const int ir = -g.ip + pr, ic = -g.ip + pc;      // input row (relative to i0) and column
    const bool ok = p < h.PH * h.PW && (unsigned)ic < (unsigned)g.Win;
    const int c = lane & 1;
    prel[u] = (ir * g.Win + ic) * 32 + c * 16;
    prow[u] = ok ? ir : -0x40000000;
  }
  auto issue_patch = [&](int tile, int buf) {
    const int n = tile / h.tiles_img, i0 = (tile - n * h.tiles_img) * h.TH;
    const int base = (n * g.Hin + i0) * g.Win * 32;
    const uint32_t lbase = smem_lds + (uint32_t)((B_U4 + buf * P_U4) * 16);
#pragma unroll
    for (int u = 0; u < PI; ++u) {
      const bool ok = (unsigned)(i0 + prow[u]) < (unsigned)g.Hin;
      lds_dma16_buf(ok ? (uint32_t)(base + prel[u]) : kOutOfRange, rsA, lbase + (uint32_t)((wave + NW * u) * 1024));
    }
  };
  int abase[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int q = wave * 64 + i * 16 + (lane & 15);
    const int ti = (int)g.fd_w.div(q);
    abase[i] = ti * h.PW + (q - ti * g.Wm);
  }
  const int kq = lane >> 4, kh = kq & 1, kt = kq >> 1;
  const int chl = 4 * (lane >> 4);
  const uint32_t out_bytes = (uint32_t)((long)g.N * g.Hout * g.Wout * g.Cols * 2);
  const __amdgpu_buffer_rsrc_t rsC = __builtin_amdgcn_make_buffer_rsrc(g.C, 0, out_bytes, 0x00020000);

  float s1[FN][4], s2[FN][4], sh[FN][4];
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) s1[j][e] = s2[j][e] = sh[j][e] = 0.f;
  bool have_shift = false;
  int rows_acc = 0;

  if (slot < h.tiles) issue_patch(slot, 0);
  int buf = 0;
  for (int tile = slot; tile < h.tiles; tile += G, buf ^= 1) {
    // this tile's patch has landed (vector memory operations complete in
    // issue order; the previous tile issued exactly FM * FN stores after it)
    if (tile == slot) wait_vmcnt<0>();
    else wait_vmcnt<FM * FN>();
    barrier_only();
    if (tile + G < h.tiles) issue_patch(tile + G, buf ^ 1);
    const int n = tile / h.tiles_img, i0 = (tile - n * h.tiles_img) * h.TH;
    const int npx = min(h.TH, g.Hm - i0) * g.Wm;
    const uint4* P = smem + B_U4 + buf * P_U4;
    floatx4_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    // the patch width is made opaque here so that the operand addresses are
    // recomputed per tile rather than held in registers across tiles
    int pw = h.PW;
    asm volatile("" : "+s"(pw));
    // K step s: tap row s / 2, taps 2 (s % 2) and 2 (s % 2) + 1 of it
    auto read_step = [&](int s, uint4(&a)[FM], uint4(&b)[FN]) {
      const int th = s >> 1, tw = 2 * (s & 1) + kt;
      const int off = th * pw + tw;
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int pix = abase[i] + off;
        a[i] = P[pix * 2 + kh];
      }
      const int t = th * 4 + tw;
#pragma unroll
      for (int j = 0; j < FN; ++j) b[j] = smem[(t * 64 + j * 16 + (lane & 15)) * 2 + kh];
    };
    uint4 a0[FM], b0[FN], a1[FM], b1[FN];
    read_step(0, a0, b0);
#pragma unroll
    for (int s = 0; s < 8; s += 2) {
      read_step(s + 1, a1, b1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) Mma<T>::run(acc[i][j], b0[j], a0[i], 0);
      __builtin_amdgcn_sched_barrier(0);
      if (s + 2 < 8) read_step(s + 2, a0, b0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) Mma<T>::run(acc[i][j], b1[j], a1[i], 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");

    // ---- epilogue straight from registers (as in the 64-channel kernel)
    const long m0 = ((long)n * g.Hm + i0) * g.Wm;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int q = wave * 64 + i * 16 + (lane & 15);
      const bool ok = q < npx;
      const uint32_t ob = (uint32_t)((m0 + (ok ? q : 0)) * g.Cols) + chl;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const uint2 pk = make_uint2(pack2<T>(acc[i][j][0], acc[i][j][1]), pack2<T>(acc[i][j][2], acc[i][j][3]));
        __builtin_amdgcn_raw_buffer_store_b64(i32x2_t{(int)pk.x, (int)pk.y}, rsC, ok ? (ob + j * 16) * 2 : kOutOfRange,
                                              0, 0);
        if constexpr (STATS) {
          const float vr[4] = {s16_to_f<T>((uint16_t)(pk.x & 0xffffu)), s16_to_f<T>((uint16_t)(pk.x >> 16)),
                               s16_to_f<T>((uint16_t)(pk.y & 0xffffu)), s16_to_f<T>((uint16_t)(pk.y >> 16))};
          if (!have_shift && i == 0) {
#pragma unroll
            for (int e = 0; e < 4; ++e) sh[j][e] = __shfl(vr[e], lane & 48, 64);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float d = ok ? vr[e] - sh[j][e] : 0.f;
            s1[j][e] += d;
            s2[j][e] = __builtin_fmaf(d, d, s2[j][e]);
          }
        }
      }
    }
    if (wave * 64 < npx) {
      have_shift = true;
      rows_acc += min(64, npx - wave * 64);
    }
  }
  if (STATS && slot < h.tiles) {
    const int kk = lane & 15, jj = kk >> 2, rr = kk & 3;
    float o1 = 0.f, o2 = 0.f, osh = 0.f;
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float a1 = s1[j][r], a2 = s2[j][r];
#pragma unroll
        for (int dd = 1; dd < 16; dd <<= 1) {
          a1 += __shfl_xor(a1, dd, 16);
          a2 += __shfl_xor(a2, dd, 16);
        }
        if (j == jj && r == rr) { o1 = a1; o2 = a2; osh = sh[j][r]; }
      }
    float4* out = (float4*)g.stats + ((long)(blockIdx.x * NW + wave) * g.Cols + jj * 16 + chl + rr);
    *out = rows_acc > 0 ? make_float4((float)rows_acc, osh, o1, o2) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  wait_vmcnt<0>();
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
template <> struct Tr<f16_t> : Tr<bf16_t> {};
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
template <> struct WOp<f16_t> : WOp<bf16_t> {
  __device__ static inline void mma(floatx4_t& acc, const uint4& a, const uint4& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), acc,
                                                 0, 0, 0);
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

// ---------------------------------------------------------------------------
// Halo weight gradient for the 64 -> 64 channel 3x3 stride-1 convolutions
// (bf16). A block walks row strips (up to 256 output pixels of whole rows of
// one image); per strip it stages the strip's dY rows and the input patch
// (TH + 2) x PW with a zero halo in LDS (double-buffered), and all nine taps
// read the patch at a fixed pixel offset, so each input pixel crosses from
// L2 about (TH + 2) PW / (TH W) times instead of nine. Wave w owns input
// channels [16 w, 16 w + 16) of all nine taps: 64 x 144 fp32 accumulators
// (36 MFMA tiles). The pixel-major MFMA operands come from the gfx950
// transposing LDS read (ds_read_b64_tr_b16: in a 16-lane group, lane 4 j + q
// addresses the 8-byte piece of pixel j, channels 4 q .. 4 q + 3, and output
// lane 4 a + b receives channel 4 a + b of pixels 0..3). A block's sum over
// its strips is one split of the fixed-order split-K reduction.
// LDS rows are 128 bytes, swizzled by row mod 8; the patch width PW is a
// multiple of 8, so a tap-row shift keeps a row's swizzle and a K step (32
// pixels) keeps every dY row's: the per-step address arithmetic is a few
// adds.
// ---------------------------------------------------------------------------
struct WgradHalo {
  const void* DY;
  const void* X;
  float* P;
  int N, H, W, TH, PW, PH, strips_img, strips;
};

constexpr int WGH_PROWS = 384;   // patch rows per buffer
constexpr int WGH_YROWS = 256;   // dY rows per buffer

template <typename T>
__global__ __launch_bounds__(256, 1) void conv_wgrad_halo_kernel(WgradHalo h) {
  constexpr int P_U4 = WGH_PROWS * 8, Y_U4 = WGH_YROWS * 8;
  constexpr int BUF_U4 = P_U4 + Y_U4;
  constexpr int PI = WGH_PROWS / 8 / 4, YI = WGH_YROWS / 8 / 4;   // load instructions per wave
  __shared__ uint4 smem[2 * BUF_U4];
  static_assert(2 * BUF_U4 * 16 <= 163840, "LDS");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t smem_lds = lds_addr(smem);
  const i32x4_t rsX = buffer_rsrc(h.X, (uint32_t)((long)h.N * h.H * h.W * 128));
  const i32x4_t rsY = buffer_rsrc(h.DY, (uint32_t)((long)h.N * h.H * h.W * 128));
  const int G = gridDim.x;

  // load geometry of this lane: patch rows (pixel -> input offset relative to
  // the strip's first row, and its row for the bounds check) and dY rows
  int prel[PI], prow[PI];
#pragma unroll
  for (int u = 0; u < PI; ++u) {
    const int p = (wave + 4 * u) * 8 + (lane >> 3);
    const int pr = p / h.PW, pc = p - pr * h.PW;
    const int ir = pr - 1, ic = pc - 1;
    const bool ok = p < h.PH * h.PW && (unsigned)ic < (unsigned)h.W;
    const int c = (lane & 7) ^ (p & 7);
    prel[u] = (ir * h.W + ic) * 128 + c * 16;
    prow[u] = ok ? ir : -0x40000000;
  }
  auto issue_strip = [&](int strip, int buf) {
    const int n = strip / h.strips_img, i0 = (strip - n * h.strips_img) * h.TH;
    const int npx = min(h.TH, h.H - i0) * h.W;
    const int base = (n * h.H + i0) * h.W * 128;
    const uint32_t lb = smem_lds + (uint32_t)(buf * BUF_U4 * 16);
#pragma unroll
    for (int u = 0; u < PI; ++u) {
      const bool ok = (unsigned)(i0 + prow[u]) < (unsigned)h.H;
      lds_dma16_buf(ok ? (uint32_t)(base + prel[u]) : kOutOfRange, rsX, lb + (uint32_t)((wave + 4 * u) * 1024));
    }
#pragma unroll
    for (int u = 0; u < YI; ++u) {
      const int q = (wave + 4 * u) * 8 + (lane >> 3);
      const int c = (lane & 7) ^ (q & 7);
      lds_dma16_buf(q < npx ? (uint32_t)(base + q * 128 + c * 16) : kOutOfRange, rsY,
                    lb + (uint32_t)(P_U4 * 16 + (wave + 4 * u) * 1024));
    }
  };

  floatx4_t acc[4][9];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < 9; ++t) acc[i][t] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  const int j4 = (lane & 15) >> 2, qq = lane & 3, kq = lane >> 4;
  const int bo = (qq & 1) * 8;
  const int cx = 2 * wave + (qq >> 1);             // X chunk of this lane's 4 channels
  // dY rows of step s are 32 s + 8 kq + j4 + 4 h2: their row mod 8 is j4 + 4 h2,
  // so the byte offset of each fragment piece is fixed up to 4096 s
  int yoff[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      const int r = 8 * kq + j4 + 4 * h2;
      yoff[i][h2] = r * 128 + (((2 * i + (qq >> 1)) ^ (r & 7)) << 4) + bo;
    }
  auto tr = [&](const lds_char_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16_t*)p);
  };
  auto pack2 = [&](v4i16_t x, v4i16_t y) {
    uint4 r;
    r.x = (uint32_t)(uint16_t)x[0] | ((uint32_t)(uint16_t)x[1] << 16);
    r.y = (uint32_t)(uint16_t)x[2] | ((uint32_t)(uint16_t)x[3] << 16);
    r.z = (uint32_t)(uint16_t)y[0] | ((uint32_t)(uint16_t)y[1] << 16);
    r.w = (uint32_t)(uint16_t)y[2] | ((uint32_t)(uint16_t)y[3] << 16);
    return r;
  };

  int buf = 0;
  if (blockIdx.x < h.strips) issue_strip(blockIdx.x, 0);
  for (int strip = blockIdx.x; strip < h.strips; strip += G, buf ^= 1) {
    wait_vmcnt<0>();
    barrier_only();
    if (strip + G < h.strips) issue_strip(strip + G, buf ^ 1);
    const int n = strip / h.strips_img, i0 = (strip - n * h.strips_img) * h.TH;
    const int npx = min(h.TH, h.H - i0) * h.W;
    const lds_char_t* PX = (const lds_char_t*)(lds_void_t)(smem + buf * BUF_U4);
    const lds_char_t* PY = PX + P_U4 * 16;
    const int rowb = h.PW * 128;                     // one patch row of pixels, in bytes
    // patch pixel of tap (0, 0) of this lane's two pixels of step 0; pixels
    // beyond the strip read patch pixel 0 (their dY rows are zero)
    int ti[2], tj[2];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      const int q = 8 * kq + j4 + 4 * h2;
      ti[h2] = q / h.W;
      tj[h2] = q - ti[h2] * h.W;
    }
    auto read_step = [&](int s, uint4(&a)[4], uint4(&b)[9]) {
      const int ys = s * 4096;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v4i16_t x[2];
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) x[h2] = tr(PY + ys + yoff[i][h2]);
        a[i] = pack2(x[0], x[1]);
      }
      int pb[2][3];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const bool ok = 32 * s + 8 * kq + j4 + 4 * h2 < npx;
        const int pp = ok ? ti[h2] * h.PW + tj[h2] : 0;
#pragma unroll
        for (int tw = 0; tw < 3; ++tw) pb[h2][tw] = (pp + tw) * 128 + ((cx ^ ((pp + tw) & 7)) << 4) + bo;
      }
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        v4i16_t x[2];
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) x[h2] = tr(PX + (t / 3) * rowb + pb[h2][t % 3]);
        b[t] = pack2(x[0], x[1]);
      }
      // advance this lane's pixels by 32 for the next step
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        tj[h2] += 32;
        while (tj[h2] >= h.W) { tj[h2] -= h.W; ++ti[h2]; }
      }
    };
    auto mma_step = [&](const uint4(&a)[4], const uint4(&b)[9]) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int t = 0; t < 9; ++t)
          Mma<T>::run(acc[i][t], a[i], b[t], 0);
    };
    uint4 a0[4], b0[9], a1[4], b1[9];
    const int S = (npx + 31) / 32;
    read_step(0, a0, b0);
    for (int s = 0; s < S; s += 2) {
      if (s + 1 < S) read_step(s + 1, a1, b1);
      __builtin_amdgcn_sched_barrier(0);
      mma_step(a0, b0);
      __builtin_amdgcn_sched_barrier(0);
      if (s + 1 < S) {
        if (s + 2 < S) read_step(s + 2, a0, b0);
        __builtin_amdgcn_sched_barrier(0);
        mma_step(a1, b1);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
  // this block's split: P[block][co][tap * 64 + ci]
  float* __restrict__ P = h.P + (long)blockIdx.x * 64 * 576;
  const int ci = 16 * wave + (lane & 15);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < 9; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) P[(16 * i + 4 * kq + r) * 576 + t * 64 + ci] = acc[i][t][r];
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

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES, bool RP>
int launch_gather2(const ConvGather& g0, hipStream_t s) {
  ConvGather g = g0;
  g.fd_hw = FastDiv((uint32_t)(g.Hm * g.Wm));
  g.fd_w = FastDiv((uint32_t)g.Wm);
  if ((long)g.N * g.Hout * g.Wout * g.Cols >= (1l << 31)) return -1;  // 32-bit output offsets
  g.zero = zero_page();
  if (!g.zero) return -4;
  if (g.ksplit > 1 && (!g.part || ((uintptr_t)g.part & 15))) return -1;
  const int ks = g.ksplit > 1 ? g.ksplit : 1;
  const int tiles = ceil_div(g.M, BM) * ceil_div(g.Cols, BN);
  const int kt = 128 / (int)sizeof(T);
  const int nt = 64 * WGM * WGN;
  const dim3 grid(tiles * ks);
  if constexpr (RP) {
    if (gather_uniform(g, kt))
      hipLaunchKernelGGL((conv_gather_rp_kernel<T, BM, BN, WGM, WGN, STAGES, true>), grid, dim3(nt), 0, s, g);
    else
      hipLaunchKernelGGL((conv_gather_rp_kernel<T, BM, BN, WGM, WGN, STAGES, false>), grid, dim3(nt), 0, s, g);
  } else {
    if (gather_uniform(g, kt))
      hipLaunchKernelGGL((conv_gather2_kernel<T, BM, BN, WGM, WGN, STAGES, true>), grid, dim3(nt), 0, s, g);
    else
      hipLaunchKernelGGL((conv_gather2_kernel<T, BM, BN, WGM, WGN, STAGES, false>), grid, dim3(nt), 0, s, g);
  }
  if (ks > 1) {
    const int rb = ceil_div(g.M, SK_ROWS) * ceil_div(g.Cols, SK_COLS);
    hipLaunchKernelGGL(gather_splitk_reduce_kernel<T>, dim3(rb), dim3(256), 0, s, g);
  }
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int cu_count() {
  static int n[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (!n[dev] && hipDeviceGetAttribute(&n[dev], hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) n[dev] = 0;
  return n[dev];
}

// A second K segment must have whole channel blocks, A2 shaped like A and
// B2 [Cols][Cin], within the 32-bit buffer offsets.
bool gather_seg2_ok(const ConvGather& g, int kt) {
  const long es = 128 / kt;
  return g.A2 && g.B2 && g.K2 == g.Cin && g.Cin % kt == 0 &&
         (long)g.N * g.Hin * g.Win * g.Cin * es < (1l << 31) && (long)g.Cols * g.Cin * es < (1l << 31);
}

// One persistent launch over the tiles of np sub-problems (all of the uniform
// row layout); -1 if one is not, -2 if a second K segment cannot run.
template <typename T, int BM, int BN, int WGM, int WGN, int STAGES>
int launch_gather_ps(const ConvGather* probs, int np, hipStream_t s) {
  if (np < 1 || np > 4) return -1;
  GatherSet gs{};
  gs.np = np;
  const int kt = 128 / (int)sizeof(T);
  long total = 0;
  for (int i = 0; i < np; ++i) {
    ConvGather g = probs[i];
    if (!gather_uniform(g, kt)) return g.K2 ? -2 : -1;
    if ((long)g.N * g.Hout * g.Wout * g.Cols >= (1l << 31)) return -1;  // 32-bit output offsets
    if (g.K2 && !gather_seg2_ok(g, kt)) return -2;
    g.fd_hw = FastDiv((uint32_t)(g.Hm * g.Wm));
    g.fd_w = FastDiv((uint32_t)g.Wm);
    g.zero = nullptr;
    gs.p[i] = g;
    gs.tile_begin[i] = (int)total;
    if (g.M > 0) total += (long)ceil_div(g.M, BM) * ceil_div(g.Cols, BN);
  }
  if (total >= (1l << 30)) return -1;
  gs.tile_begin[np] = (int)total;
  if (total == 0) return 0;
  constexpr int NT = 64 * WGM * WGN;
  constexpr int occ = gather_blocks_per_cu(BM, BN, STAGES);  // registers are bounded to match
  const int cus = cu_count();
  if (cus < 1) return -4;
  const long grid = total < (long)occ * cus ? total : (long)occ * cus;
  hipLaunchKernelGGL((conv_gather_ps_kernel<T, BM, BN, WGM, WGN, STAGES>), dim3((unsigned)grid), dim3(NT), 0, s, gs);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// Tile height of the halo kernel for a launch, or 0 when the launch is not
// one it handles (bf16, 64 -> 64 channels, 3x3 taps walked forward with
// stride 1, output rows = GEMM rows, whole-row tiles that divide the image).
int halo_rows(int prec, const ConvGather& g) {
  if (prec == PREC_F32 || g.Cin != 64 || g.Cols != 64 || g.nth != 3 || g.ntw != 3 || g.KHW != 9 || g.K != 576)
    return 0;
  if (g.is != 1 || g.os != 1 || g.oph != 0 || g.opw != 0 || g.dhs != 1 || g.dws != 1) return 0;
  if (g.Hout != g.Hm || g.Wout != g.Wm || g.Hm < 1 || g.Wm < 1) return 0;
  if (g.mode < 0 || g.mode > 2 || (g.mode != 0 && g.stats)) return 0;
  if ((long)g.N * g.Hin * g.Win * 128 >= (1l << 31) || (long)g.N * g.Hout * g.Wout * g.Cols >= (1l << 31)) return 0;
  // as many whole rows as fit 512 pixels and a 640-pixel patch; at least
  // 256 pixels per tile keeps the per-wave statistics entries (8 per block,
  // blocks <= tiles) at most one per 32 GEMM rows
  int th = HALO_BM / g.Wm;
  if (th > g.Hm) th = g.Hm;
  while (th > 0 && (th + 2) * (g.Wm + 2) > HALO_PROWS) --th;
  if (th < 1 || th * g.Wm < 256) return 0;
  return th;
}

// Tile height of the stem halo kernel, or 0 when the launch is not one it
// handles (bf16, 16 -> 64 channels, a forward 4x4 stride-1 tap walk, mode 0).
int halo16_rows(int prec, const ConvGather& g) {
  if (prec == PREC_F32 || g.Cin != 16 || g.Cols != 64 || g.nth != 4 || g.ntw != 4 || g.KHW != 16 || g.KW != 4 ||
      g.K != 256)
    return 0;
  if (g.is != 1 || g.os != 1 || g.oph != 0 || g.opw != 0 || g.dh0 != 0 || g.dw0 != 0 || g.dhs != 1 || g.dws != 1 ||
      g.wkh0 != 0 || g.wkw0 != 0 || g.wkhs != 1 || g.wkws != 1 || g.mode != 0)
    return 0;
  if (g.Hout != g.Hm || g.Wout != g.Wm || g.Hm < 1 || g.Wm < 1) return 0;
  if ((long)g.N * g.Hin * g.Win * 32 >= (1l << 31) || (long)g.N * g.Hout * g.Wout * g.Cols * 2 >= (1l << 31)) return 0;
  // at least 128 pixels per tile keeps the per-wave statistics entries (4
  // per block, blocks <= tiles) at most one per 32 GEMM rows
  int th = HALO16_BM / g.Wm;
  if (th > g.Hm) th = g.Hm;
  while (th > 0 && (th + 3) * (g.Wm + 3) > HALO16_PROWS) --th;
  if (th < 1 || th * g.Wm < 128) return 0;
  return th;
}

template <typename T>
int launch_halo16(const ConvGather& g0, int th, hipStream_t s) {
  ConvHalo h{};
  h.g = g0;
  h.g.fd_hw = FastDiv((uint32_t)(g0.Hm * g0.Wm));
  h.g.fd_w = FastDiv((uint32_t)g0.Wm);
  h.TH = th;
  h.PH = th + 3;
  h.PW = g0.Wm + 3;
  h.tiles_img = (g0.Hm + th - 1) / th;
  h.tiles = g0.N * h.tiles_img;
  if (h.tiles <= 0) return 0;
  const int slots = 2 * cu_count();
  if (slots < 1) return -4;
  const int grid = h.tiles < slots ? h.tiles : slots;
  constexpr int NT = 64 * HALO16_WAVES;
  if (g0.stats) hipLaunchKernelGGL((conv_halo16_kernel<T, true>), dim3(grid), dim3(NT), 0, s, h);
  else hipLaunchKernelGGL((conv_halo16_kernel<T, false>), dim3(grid), dim3(NT), 0, s, h);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

template <typename T>
int launch_halo(const ConvGather& g0, int th, hipStream_t s) {
  ConvHalo h{};
  h.g = g0;
  h.g.fd_hw = FastDiv((uint32_t)(g0.Hm * g0.Wm));
  h.g.fd_w = FastDiv((uint32_t)g0.Wm);
  h.TH = th;
  h.PH = th + 2;
  h.PW = g0.Wm + 2;
  h.tiles_img = (g0.Hm + th - 1) / th;
  h.tiles = g0.N * h.tiles_img;
  if (h.tiles <= 0) return 0;
  const int cus = cu_count();
  if (cus < 1) return -4;
  const int grid = h.tiles < cus ? h.tiles : cus;
  const bool st = g0.stats != nullptr;
  constexpr int NT = 64 * HALO_WAVES;
  if (g0.mode == 0 && st) hipLaunchKernelGGL((conv_halo_kernel<T, 0, true>), dim3(grid), dim3(NT), 0, s, h);
  else if (g0.mode == 0) hipLaunchKernelGGL((conv_halo_kernel<T, 0, false>), dim3(grid), dim3(NT), 0, s, h);
  else if (g0.mode == 1 && !st) hipLaunchKernelGGL((conv_halo_kernel<T, 1, false>), dim3(grid), dim3(NT), 0, s, h);
  else if (g0.mode == 2 && !st) hipLaunchKernelGGL((conv_halo_kernel<T, 2, false>), dim3(grid), dim3(NT), 0, s, h);
  else return -1;
  return hipGetLastError() == hipSuccess ? 0 : -4;
}


// Kernel configurations: id -> (BM, BN, waves along M, waves along N, stages,
// kind: 0 plain loop, 1 register-prefetched loop, 2 persistent).
#define RN18_GATHER_CONFIGS(X)                                                                                  \
  X(1, 64, 32, 2, 2, 3, 0) X(2, 64, 64, 2, 2, 3, 0) X(3, 128, 64, 2, 2, 3, 0) X(4, 128, 128, 2, 2, 3, 0)        \
  X(5, 256, 128, 4, 2, 3, 0) X(6, 256, 128, 2, 2, 3, 0) X(7, 256, 64, 4, 2, 3, 0) X(8, 128, 128, 2, 4, 3, 0)    \
  X(9, 256, 64, 4, 1, 3, 0) X(10, 128, 128, 2, 2, 2, 0) X(11, 256, 128, 4, 2, 2, 0) X(12, 128, 64, 2, 2, 4, 0)  \
  X(13, 128, 64, 2, 2, 2, 0) X(14, 64, 64, 2, 2, 2, 0) X(15, 256, 64, 4, 2, 2, 0) X(16, 128, 128, 2, 4, 2, 0)   \
  X(17, 256, 128, 2, 2, 2, 0) X(18, 512, 64, 4, 1, 2, 0) X(19, 256, 128, 2, 2, 3, 0) X(20, 128, 128, 2, 2, 4, 0) \
  X(21, 256, 64, 4, 1, 2, 0) X(22, 256, 64, 2, 2, 2, 0) X(23, 128, 128, 2, 2, 2, 1) X(24, 256, 128, 4, 2, 2, 1) \
  X(25, 256, 64, 4, 1, 2, 1) X(26, 128, 128, 2, 4, 2, 1) X(27, 256, 64, 4, 2, 2, 1) X(28, 256, 128, 4, 2, 3, 1)  \
  X(29, 128, 128, 2, 2, 3, 1) X(30, 512, 64, 8, 1, 2, 1) X(31, 128, 256, 2, 4, 2, 1) X(32, 128, 64, 2, 2, 2, 1)  \
  X(33, 64, 64, 2, 2, 2, 1) X(34, 256, 64, 4, 1, 3, 1) X(35, 256, 64, 4, 2, 2, 2) X(36, 128, 128, 2, 4, 2, 2)   \
  X(37, 128, 64, 2, 2, 2, 2) X(38, 64, 64, 2, 2, 2, 2) X(39, 256, 128, 4, 2, 2, 2) X(40, 128, 128, 2, 2, 2, 2)  \
  X(41, 128, 256, 2, 4, 2, 2) X(42, 128, 128, 2, 4, 3, 2) X(43, 256, 64, 4, 2, 3, 2) X(44, 128, 64, 2, 2, 3, 2)
constexpr int kGatherCfgs = 44;
constexpr int kGatherHalo = 45;  // the halo kernel where it applies, else the automatic choice
int g_gather_override = 0;

struct GatherCfg { int bm, bn, wgm, wgn, stages, kind; };
constexpr GatherCfg kGather[kGatherCfgs + 1] = {
    {0, 0, 0, 0, 0, 0},
#define RN18_X(id, bm, bn, wgm, wgn, st, kind) {bm, bn, wgm, wgn, st, kind},
    RN18_GATHER_CONFIGS(RN18_X)
#undef RN18_X
};

// Choice measured on MI355X over the ResNet-18 shapes (bf16 224x224 batch 256,
// fp32 32x32 batch 128): two-stage rings with two or more blocks per CU beat
// deeper rings with one block; 8-wave blocks for the large tiles.
int gather_cfg(const ConvGather& g) {
  if (g_gather_override && g_gather_override != kGatherHalo) return g_gather_override;
  if (g.Cols <= 32) return 1;
  if (g.Cols <= 64) return g.M >= 131072 ? 15 : g.M >= 65536 ? 13 : 14;
  return (long)ceil_div(g.M, 128) * ceil_div(g.Cols, 128) >= 256 ? 16 : 14;
}

// Split-K for launches whose grid leaves CUs idle (fewer tiles than CUs:
// small batches at the late stages, e.g. 1024 GEMM rows x 512 channels at
// batch 64, 128x128 images): the K stages are cut into ranges of at least
// kSplitMinStages, for about kSplitBlocks blocks in all. Measured on MI355X,
// whole training steps: batch 64 at 128x128 2.07 -> 1.87 ms, at 160x160
// 2.27 -> 2.11 ms. Grids of 256..448 tiles, split, won alone but lost in the
// step beside the weight-gradient stream (batch 256 at 224x224 +0.1 ms,
// fp32 batch 128 at 32x32 +0.09 ms), so they stay whole. Only the
// non-persistent kernels split.
int g_gather_split = 0;
constexpr long kSplitBlocks = 640;
constexpr long kSplitMaxTiles = 255;
constexpr int kSplitMinStages = 8;

int gather_split_want(int prec, const ConvGather& g, int id) {
  if (id < 1 || id > kGatherCfgs || kGather[id].kind == 2 || g.K2 || g_gather_split == 1) return 1;
  const int S = ceil_div(g.K, 128 / prec_bytes(prec));
  int k;
  if (g_gather_split > 1) {
    k = g_gather_split;
  } else {
    const long tiles = (long)ceil_div(g.M, kGather[id].bm) * ceil_div(g.Cols, kGather[id].bn);
    if (tiles > kSplitMaxTiles) return 1;
    k = (int)((kSplitBlocks + tiles / 2) / tiles);
    if (k > S / kSplitMinStages) k = S / kSplitMinStages;
  }
  if (k > S) k = S;
  return k < 2 ? 1 : k;
}

// The split count a launch runs: the wanted one, cut to what the caller's
// scratch holds (none without scratch).
int gather_split(int prec, const ConvGather& g, int id) {
  int k = gather_split_want(prec, g, id);
  if (k < 2 || !g.ws || ((uintptr_t)g.ws & 15)) return 1;
  const size_t per = (size_t)g.M * g.Cols * 4;
  if (per == 0) return 1;
  if ((size_t)k > g.ws_bytes / per) k = (int)(g.ws_bytes / per);
  return k < 2 ? 1 : k;
}

bool use_halo(int prec, const ConvGather& g) {
  return (g_gather_override == 0 || g_gather_override == kGatherHalo) && halo_rows(prec, g) > 0;
}
bool use_halo16(int prec, const ConvGather& g) {
  return (g_gather_override == 0 || g_gather_override == kGatherHalo) && halo16_rows(prec, g) > 0;
}

int gather_tile(int prec, const ConvGather& g) {
  if (use_halo(prec, g)) return HALO_BM * 1000 + 64;
  if (use_halo16(prec, g)) return HALO16_BM * 1000 + 64;
  const int id = gather_cfg(g);
  return id >= 1 && id <= kGatherCfgs ? kGather[id].bm * 1000 + kGather[id].bn : 0;
}

// The sub-problems of one launch share the configuration chosen for the
// first; a persistent configuration takes them all in one grid when every
// one has the uniform row layout, the others launch one grid each.
// The parity phases of a stride-2 data gradient run in one persistent grid
// (measured on MI355X at bf16 224x224 batch 256: 256x64 tiles for up to 64
// columns, 128x128 for 128, 128x64 above).
// A launch with a second K segment always takes the persistent kernel (the
// only one that runs it), whatever configuration is forced.
bool gather_has_seg2(const ConvGather* g, int np) {
  for (int i = 0; i < np; ++i)
    if (g[i].K2) return true;
  return false;
}
int gather_cfg_multi(const ConvGather* g, int np) {
  if (!gather_has_seg2(g, np) && (g_gather_override || np < 2)) return gather_cfg(g[0]);
  return g[0].Cols <= 64 ? 35 : g[0].Cols <= 128 ? 36 : 37;
}

template <typename T>
int gather_dispatch(const ConvGather* g, int np, hipStream_t s) {
  const int prec = prec_of<T>();
  const bool seg2 = gather_has_seg2(g, np);
  if (g[0].bstats && !conv_gather_bwd_ok_multi(prec, g, np)) return -1;   // not computed on this path
  if constexpr (sizeof(T) == 2) {
    // the halo kernels are instantiated for the 16-bit storage types only
    if (!seg2 && np == 1 && use_halo(prec, g[0])) return launch_halo<T>(g[0], halo_rows(prec, g[0]), s);
    if (!seg2 && np == 1 && use_halo16(prec, g[0])) return launch_halo16<T>(g[0], halo16_rows(prec, g[0]), s);
  }
  switch (gather_cfg_multi(g, np)) {
#define RN18_X(id, bm, bn, wgm, wgn, st, kind)                                               \
  case id:                                                                                 \
    if constexpr (kind == 2) {                                                             \
      const int r = launch_gather_ps<T, bm, bn, wgm, wgn, st>(g, np, s);                   \
      if (r != -1 || seg2) return r;                                                       \
    }                                                                                      \
    for (int i = 0; i < np; ++i) {                                                         \
      if (g[i].M <= 0) continue;                                                           \
      ConvGather gi = g[i];                                                                \
      gi.ksplit = gather_split(prec, gi, id);                                              \
      gi.part = (float*)gi.ws;                                                             \
      const int r = launch_gather2<T, bm, bn, wgm, wgn, st, kind == 1>(gi, s);             \
      if (r) return r;                                                                     \
    }                                                                                      \
    return 0;
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
  if (prec != PREC_F32) {
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
  switch (wgrad_cfg(prec_of<T>(), g.Cout, g.Kcols)) {
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

// Strip height of the halo weight-gradient kernel, or 0 when the shape is not
// one it handles (bf16, 64 -> 64 channels, 3x3, stride 1, padding 1).
int wgrad_halo_pw(const ConvWgrad& g) { return (g.W + 2 + 7) / 8 * 8; }

int wgrad_halo_rows(int prec, const ConvWgrad& g) {
  if (prec == PREC_F32 || g.Cin != 64 || g.Cout != 64 || g.KH != 3 || g.KW != 3 || g.stride != 1 || g.pad != 1)
    return 0;
  if (g.Ho != g.H || g.Wo != g.W || g.H < 1 || g.W < 1 || g.W > 256) return 0;
  if ((long)g.N * g.H * g.W * 128 >= (1l << 31)) return 0;
  int th = WGH_YROWS / g.W;
  if (th > g.H) th = g.H;
  while (th > 0 && (th + 2) * wgrad_halo_pw(g) > WGH_PROWS) --th;
  return th;
}

bool use_wgrad_halo(int prec, const ConvWgrad& g) { return g_wgrad_override == 0 && wgrad_halo_rows(prec, g) > 0; }

int wgrad_halo_grid(int prec, const ConvWgrad& g) {
  const int th = wgrad_halo_rows(prec, g);
  const long strips = (long)g.N * ((g.H + th - 1) / th);
  const int cus = cu_count();
  return (int)(strips < cus ? strips : cus);
}

template <typename T>
int launch_wgrad_halo(const ConvWgrad& g, hipStream_t s) {
  WgradHalo h{};
  h.DY = g.DY; h.X = g.X; h.P = g.P;
  h.N = g.N; h.H = g.H; h.W = g.W;
  h.TH = wgrad_halo_rows(prec_of<T>(), g);
  h.PW = wgrad_halo_pw(g); h.PH = h.TH + 2;
  h.strips_img = (g.H + h.TH - 1) / h.TH;
  h.strips = g.N * h.strips_img;
  if (g.splits != wgrad_halo_grid(prec_of<T>(), g) || g.splits < 1) return -1;   // split count planned for this kernel
  hipLaunchKernelGGL(conv_wgrad_halo_kernel<T>, dim3(g.splits), dim3(256), 0, s, h);
  return hipGetLastError() == hipSuccess ? 0 : -4;
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

const char* type_name(int prec) { return prec == PREC_BF16 ? "bf16" : prec == PREC_F16 ? "_Float16" : "float"; }

}  // namespace

const char* gather_kernel_name(int prec, const ConvGather& g, int id);

const char* conv_gather_kernel_name(int prec, const ConvGather& g) {
  if (use_halo(prec, g)) {
    char buf[80];
    snprintf(buf, sizeof buf, "conv_halo_kernel<%s, %d, %s>", type_name(prec), g.mode, g.stats ? "true" : "false");
    return intern_name(buf);
  }
  if (use_halo16(prec, g)) {
    char buf[80];
    snprintf(buf, sizeof buf, "conv_halo16_kernel<%s, %s>", type_name(prec), g.stats ? "true" : "false");
    return intern_name(buf);
  }
  return gather_kernel_name(prec, g, gather_cfg(g));
}

const char* conv_gather_kernel_name_multi(int prec, const ConvGather* g, int np) {
  if (np == 1 && !g[0].K2) return conv_gather_kernel_name(prec, g[0]);
  return gather_kernel_name(prec, g[0], gather_cfg_multi(g, np));
}

const char* gather_kernel_name(int prec, const ConvGather& g, int id) {
  if (id < 1 || id > kGatherCfgs) return "conv_gather2_kernel";
  const GatherCfg& c = kGather[id];
  const int kt = 128 / prec_bytes(prec);
  char buf[128];
  if (c.kind == 2 && gather_uniform(g, kt))
    snprintf(buf, sizeof buf, "conv_gather_ps_kernel<%s, %d, %d, %d, %d, %d>", type_name(prec), c.bm, c.bn, c.wgm,
             c.wgn, c.stages);
  else
    snprintf(buf, sizeof buf, "%s<%s, %d, %d, %d, %d, %d, %s>",
             c.kind == 1 ? "conv_gather_rp_kernel" : "conv_gather2_kernel", type_name(prec), c.bm, c.bn, c.wgm, c.wgn,
             c.stages, gather_uniform(g, kt) ? "true" : "false");
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

int conv_gather_tile(int prec, const ConvGather& g) { return gather_tile(prec, g); }

int conv_gather_tile_multi(int prec, const ConvGather* g, int np) {
  if (np == 1 && !g[0].K2) return gather_tile(prec, g[0]);
  const int id = gather_cfg_multi(g, np);
  return id >= 1 && id <= kGatherCfgs ? kGather[id].bm * 1000 + kGather[id].bn : 0;
}

int conv_gather_stat_entries(int prec, const ConvGather& g) {
  if (use_halo(prec, g)) {
    const int th = halo_rows(prec, g);
    const int tiles = g.N * ((g.Hm + th - 1) / th), cus = cu_count();
    return (tiles < cus ? tiles : cus) * HALO_WAVES;
  }
  if (use_halo16(prec, g)) {
    const int th = halo16_rows(prec, g);
    const int tiles = g.N * ((g.Hm + th - 1) / th), slots = 2 * cu_count();
    return (tiles < slots ? tiles : slots) * HALO16_WAVES;
  }
  if (gather_split(prec, g, gather_cfg(g)) > 1) return ceil_div(g.M, SK_ROWS);
  const int bm = gather_tile(prec, g) / 1000;
  return bm > 0 ? ceil_div(g.M, bm) : 0;
}

int conv_gather_split_count(int prec, const ConvGather& g) {
  if (use_halo(prec, g) || use_halo16(prec, g)) return 1;
  return gather_split(prec, g, gather_cfg(g));
}

// The BN backward partials are computed by the non-persistent gather
// kernels and the split-K reduce (one launch of one sub-problem).
bool conv_gather_bwd_ok(int prec, const ConvGather& g) {
  if (g.K2 || use_halo(prec, g) || use_halo16(prec, g)) return false;
  const int id = gather_cfg(g);
  return id >= 1 && id <= kGatherCfgs && kGather[id].kind != 2;
}

int conv_gather_bwd_entries(int prec, const ConvGather& g) {
  if (!conv_gather_bwd_ok(prec, g)) return 0;
  const int id = gather_cfg(g);
  return gather_split(prec, g, id) > 1 ? ceil_div(g.M, SK_ROWS) : ceil_div(g.M, kGather[id].bm);
}

// Several sub-problems: the persistent kernel computes them when it runs the
// launch (its configuration, every sub-problem in the uniform row layout)
// and the output has more than 64 channels. Measured on MI355X at batch 256,
// 224x224: the 64-channel stride-2 data gradient of stage 2 (256x64 tiles,
// 3,136 per launch) took 164 -> 258 us with the epilogue reading y, more
// than the 44 us reduction it replaces; the 128- and 256-channel ones did not
// slow down.
bool conv_gather_bwd_ok_multi(int prec, const ConvGather* g, int np) {
  if (np == 1 && !g[0].K2) return conv_gather_bwd_ok(prec, g[0]);
  if (np < 1 || np > 4 || g[0].Cols <= 64) return false;
  const int id = gather_cfg_multi(g, np);
  if (id < 1 || id > kGatherCfgs || kGather[id].kind != 2) return false;
  const int kt = 128 / prec_bytes(prec);
  for (int i = 0; i < np; ++i)
    if (!gather_uniform(g[i], kt)) return false;
  return true;
}

int conv_gather_bwd_entries_multi(int prec, const ConvGather* g, int np) {
  if (np == 1 && !g[0].K2) return conv_gather_bwd_entries(prec, g[0]);
  if (!conv_gather_bwd_ok_multi(prec, g, np)) return 0;
  const int bm = kGather[gather_cfg_multi(g, np)].bm;
  int n = 0;
  for (int i = 0; i < np; ++i) n += g[i].M > 0 ? ceil_div(g[i].M, bm) : 0;
  return n;
}

int conv_gather_split_override(int k) {
  if (k < 0 || k > 64) return -1;
  g_gather_split = k;
  return 0;
}

int conv_gather_override(int id) {
  if (id < 0 || id > kGatherHalo) return -1;
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
  return with_prec(prec, [&](auto tag) { return gather_dispatch<decltype(tag)>(&g, 1, s); });
}

int conv_gather_launch_multi(int prec, const ConvGather* g, int np, hipStream_t s) {
  if (np < 1 || np > 4) return -1;
  return with_prec(prec, [&](auto tag) { return gather_dispatch<decltype(tag)>(g, np, s); });
}

int conv_wgrad_splits(int prec, int Cout, int Kcols, long Mpix, int* pix_per_split) {
  const int ktp = 128 / prec_bytes(prec);
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

int conv_wgrad_splits_shape(int prec, const ConvWgrad& g, int* pix_per_split) {
  if (use_wgrad_halo(prec, g)) {
    *pix_per_split = 0;
    return wgrad_halo_grid(prec, g);
  }
  return conv_wgrad_splits(prec, g.Cout, g.KH * g.KW * g.Cin, (long)g.N * g.Ho * g.Wo, pix_per_split);
}

const char* conv_wgrad_kernel_name_shape(int prec, const ConvWgrad& g) {
  if (use_wgrad_halo(prec, g)) return prec == PREC_F16 ? "conv_wgrad_halo_kernel<_Float16>" : "conv_wgrad_halo_kernel<bf16>";
  return conv_wgrad_kernel_name(prec, g.Cout, g.KH * g.KW * g.Cin);
}

int conv_wgrad_launch(int prec, const ConvWgrad& g, hipStream_t s) {
  if (use_wgrad_halo(prec, g))
    return with_prec(prec, [&](auto tag) {
      using T = decltype(tag);
      if constexpr (sizeof(T) == 2) return launch_wgrad_halo<T>(g, s);
      return -1;
    });
  // the pipelined kernels address both operands with 31-bit byte offsets
  const long es = prec_bytes(prec);
  if ((long)g.Mpix * g.Cout * es >= (1l << 31) || (long)g.N * g.H * g.W * g.Cin * es >= (1l << 31)) return -1;
  return with_prec(prec, [&](auto tag) { return wgrad_dispatch<decltype(tag)>(g, s); });
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
