// Host-side launchers of the gfx950 kernels (defined in the .hip files).
#pragma once
#include "common.h"

namespace rn18 {

// ---------------------------------------------------------------------------
// Implicit-GEMM convolution "gather" form, used for the forward pass and the
// data gradient: C[m][col] = sum_{tap,ci} A[pixel(m,tap)][ci] * B[col][wtap][ci]
// ---------------------------------------------------------------------------
struct ConvGather {
  const void* A;   // NHWC activations [N][Hin][Win][Cin]
  const void* B;   // weights [Cols][KHW][Cin]
  void* C;         // NHWC output [N][Hout][Wout][Cols]
  const void* R;   // epilogue: residual gradient (mode 2)
  const void* Rm;  // epilogue: ReLU mask bytes of the residual (mode 2; bn_apply_launch's layout)
  int N, Hin, Win, Cin;
  int Hm, Wm, M;             // GEMM row grid per image; M = N*Hm*Wm
  int Hout, Wout, Cols;
  int os, oph, opw;          // output pixel (i*os+oph, j*os+opw)
  int is, ip;                // input base (i*is-ip, j*is-ip)
  int nth, ntw;              // taps along h and w
  int dh0, dhs, dw0, dws;    // input offset of tap (th,tw): (dh0+th*dhs, dw0+tw*dws)
  int wkh0, wkhs, wkw0, wkws, KW, KHW;  // weight tap (wkh0+th*wkhs)*KW + wkw0+tw*wkws
  int K;                     // nth*ntw*Cin
  int mode;                  // 0 store, 1 C += acc, 2 C = acc + (mask ? R : 0)
  FastDiv fd_hw, fd_w;       // division by Hm*Wm and by Wm (set by the launcher)
  float* stats;              // optional BN partials (rows, shift, sum, sum sq) [tiles_m][Cols][4] of the stored output
  const void* zero;          // 16-byte zero page (set by the launcher)
  // Optional second K segment, summed into the same accumulators before the
  // epilogue: C[m][col] += sum_ci A2[pixel(hb, wb)][ci] * B2[col][ci], where
  // (hb, wb) = (i*is-ip, j*is-ip) is the row's input base itself (tap offset
  // 0). A2 is shaped like A ([N][Hin][Win][Cin]) and B2 is [Cols][Cin];
  // K2 = Cin, or 0 for none. Only the persistent multi-phase kernel takes
  // it (the projection shortcut's data gradient fused into parity phase
  // (0,0) of the block's stride-2 data gradient).
  const void* A2;
  const void* B2;
  int K2;
  // Optional split-K scratch of the caller (nullptr: never split). A launch
  // with too few tiles to fill the chip may cut its K stages into ksplit
  // contiguous ranges: block (tile, range) writes its fp32 tile to
  // part[range][M][Cols], and a reduce pass sums the ranges in a fixed order
  // and applies the epilogue (mode, storage rounding, BN partials). ksplit
  // and part are set by the launcher.
  void* ws;
  size_t ws_bytes;
  int ksplit;
  float* part;
  // Optional BN backward partials of the stored output (the output is the
  // gradient entering the backward pass of a BN whose forward output by has
  // the shape of C): per tile of rows and channel, sum g and sum g * xhat,
  // g = the stored value where that BN's ReLU passed, xhat = (by - bmean) *
  // brstd. The ReLU mask is bit e of the chunk's byte in bmask, or, with
  // bmask null, relu(by * bsc + bsf) > 0 as stored. Written as float2
  // entries bstats[entry][Cols]; conv_gather_bwd_entries gives the count.
  float* bstats;
  const void* by;
  const uint8_t* bmask;
  const float* bmean;
  const float* brstd;
  const float* bsc;
  const float* bsf;
};
int conv_gather_launch(int prec, const ConvGather& g, hipStream_t s);
// Up to four sub-problems of one operation (the parity phases of a stride-2
// data gradient) with one configuration; persistent configurations run them
// in a single grid.
int conv_gather_launch_multi(int prec, const ConvGather* g, int np, hipStream_t s);
// Tile configuration (BM*1000 + BN) the dispatcher picks for a launch.
int conv_gather_tile(int prec, const ConvGather& g);
// Number of BN partial-statistics entries a forward launch with g.stats set
// writes (at most one per 32 GEMM rows).
int conv_gather_stat_entries(int prec, const ConvGather& g);
// Force one kernel configuration for every gather launch (0 = automatic choice).
int conv_gather_override(int id);
// Split-K: number of K ranges a launch of g runs with its scratch (1 = none).
int conv_gather_split_count(int prec, const ConvGather& g);
// BN backward partials in the epilogue (g.bstats): whether the kernel a
// launch of g runs computes them, and how many entries it writes.
bool conv_gather_bwd_ok(int prec, const ConvGather& g);
int conv_gather_bwd_entries(int prec, const ConvGather& g);
bool conv_gather_bwd_ok_multi(int prec, const ConvGather* g, int np);
int conv_gather_bwd_entries_multi(int prec, const ConvGather* g, int np);
// Force the split count of every gather launch that has scratch for it
// (0 = automatic choice, 1 = never split; at most the launch's K stages).
int conv_gather_split_override(int k);

// Weight gradient: P[split][co][tap*Cin+ci] = sum_pixels dY[p][co] * Xcol[p][tap,ci]
struct ConvWgrad {
  const void* DY;  // [N][Ho][Wo][Cout]
  const void* X;   // [N][H][W][Cin]
  float* P;        // split partials [splits][Cout][KHW*Cin]
  int N, H, W, Cin, Ho, Wo, Cout, KH, KW, stride, pad;
  int Mpix, Kcols, pix_per_split, splits;
};
int conv_wgrad_launch(int prec, const ConvWgrad& g, hipStream_t s);
int conv_wgrad_tile(int prec, int Cout, int Kcols);
// Names of the kernel instance a launch would use, in the form a profiler's
// demangler prints them (namespace dropped, uint16_t storage shown as bf16);
// kernel_instance_name(base, prec) is base<bf16> or base<float>.
const char* conv_gather_kernel_name(int prec, const ConvGather& g);
const char* conv_gather_kernel_name_multi(int prec, const ConvGather* g, int np);
int conv_gather_tile_multi(int prec, const ConvGather* g, int np);
const char* conv_wgrad_kernel_name(int prec, int Cout, int Kcols);
const char* kernel_instance_name(const char* base, int prec);
// Force one weight-gradient configuration (0 = automatic choice).
int conv_wgrad_override(int id);
// Choose the split count for a weight-gradient GEMM (deterministic function of the shape).
int conv_wgrad_splits(int prec, int Cout, int Kcols, long Mpix, int* pix_per_split);
// Split count (and pixels per split) for a weight-gradient launch of this
// shape (N, H, W, Cin, Ho, Wo, Cout, KH, KW, stride, pad set in g): the
// 64-channel 3x3 stride-1 shape runs the halo kernel, one split per block.
int conv_wgrad_splits_shape(int prec, const ConvWgrad& g, int* pix_per_split);
const char* conv_wgrad_kernel_name_shape(int prec, const ConvWgrad& g);
// Sum partials in split order; write OIHW gradient (Cin_real of Cin channels kept).
// Fixed-order sum of the split partials [splits][Cout][KHW][Cin] into OIHW
// [Cout][Cin_real][KHW]; s2d = 1 maps the space-to-depth stem partials
// [Cout][4x4][16] back to the 7x7 stem [Cout][3][7][7].
int wgrad_reduce_launch(const float* P, int splits, int Cout, int KHW, int Cin, int Cin_real,
                        float* out_oihw, int s2d, hipStream_t s);

// ---------------------------------------------------------------------------
// Batch norm (per-channel over M = N*H*W rows of an [M][C] tensor)
// ---------------------------------------------------------------------------
// partial sums of (y - pivot) and (y - pivot)^2 per block; pivot = y[0][c]
// Batch statistics from the forward conv epilogue's per-tile partials
// (rows, shift, sum of v - shift, sum of (v - shift)^2) [ntiles][C][4].
// scratch: bn_stats_tiles_chunks(ntiles) * C * 3 doubles
int bn_stats_tiles_chunks(int ntiles);
int bn_stats_tiles_final_launch(const float* tile_stats, int ntiles, int C, double* scratch, const float* gamma,
                                const float* beta, float eps, float momentum, float* run_mean, float* run_var,
                                float* mean, float* rstd, float* scale, float* shift, hipStream_t s);
// z = act(y*scale+shift [+ r] [+ (yd*scale2+shift2)])
//  res_mode: 0 none, 1 identity residual r, 2 projected residual (yd, scale2, shift2)
// ReLU mask bytes (mbits, optional, M*C/VW bytes): one byte per 16-byte
// storage chunk of z (VW = 8 bf16 or 4 fp32 elements), bit e set iff element
// e of the chunk as stored is > 0.
int bn_apply_launch(int prec, const void* y, const float* scale, const float* shift, int relu,
                    int res_mode, const void* r, const float* scale2, const float* shift2,
                    void* z, long M, int C, hipStream_t s, uint8_t* mbits = nullptr);
// eval-mode BN coefficients from running statistics
int bn_eval_coef_launch(const float* gamma, const float* beta, const float* rm, const float* rv,
                        float eps, int C, float* scale, float* shift, hipStream_t s);
// backward partials of g = dz*mask (or dz): sum g, sum g*(y-mean)*rstd
// The ReLU mask comes from mask bytes mb (the layout bn_apply_launch writes)
// when given; with mb = NULL and mscale set it is recomputed as
// relu(y * mscale + mshift) > 0 of the stored value (the first BN of a
// block, whose ReLU output feeds only the next conv); with neither, there is
// no mask.
int bn_bwd_partial_launch(int prec, const void* dz, const uint8_t* mb, const void* y, const float* mean,
                          const float* rstd, long M, int C, float* part, int* nblk, hipStream_t s,
                          const float* mscale = nullptr, const float* mshift = nullptr);
// blocks (= partial entries of 2 floats per channel) that the two backward
// partial launches use for a shape; `part` must hold blocks * C * 2 floats
int bn_bwd_partial_blocks(int prec, long M, int C);
int bn_bwd_partial_pool_blocks(int prec, int N, int H, int W, int C);
// dgamma, dbeta into grad; coefficients for the apply
// ImageNet stem fused with its max pool (y = stem conv output [N][H][W][C],
// pool / arg = pool output and argmax [N][Ho][Wo][C]): forward BN-apply +
// ReLU + pool; backward BN reduce / apply reading the pooled gradient.
int bn_apply_pool_launch(int prec, const void* y, const float* scale, const float* shift, void* pool, uint8_t* arg,
                         int N, int H, int W, int C, int Ho, int Wo, hipStream_t s);
int bn_bwd_partial_pool_launch(int prec, const void* dpool, const uint8_t* arg, const void* y, const float* scale,
                               const float* shift, const float* mean, const float* rstd, int N, int H, int W, int C,
                               int Ho, int Wo, float* part, int* nblk, hipStream_t s);
int bn_bwd_apply_pool_launch(int prec, const void* dpool, const uint8_t* arg, const void* y, const float* scale,
                             const float* shift, const float* mean, const float* coef, void* dy, int N, int H, int W,
                             int C, int Ho, int Wo, hipStream_t s);
int bn_bwd_final_launch(const float* part, int nblk, long M, int C, const float* gamma, const float* rstd,
                        float* dgamma, float* dbeta, float* coef, hipStream_t s);
// dy = k1*g + k2*(y-mean) + k3; done (optional) is recorded by the kernel
// launch itself, completing when the kernel does
int bn_bwd_apply_launch(int prec, const void* dz, const uint8_t* mb, const void* y, const float* mean,
                        const float* coef, void* dy, long M, int C, hipStream_t s, const float* mscale = nullptr,
                        const float* mshift = nullptr, hipEvent_t done = nullptr);

// ---------------------------------------------------------------------------
// Misc streams
// ---------------------------------------------------------------------------
// A non-finite image value sets DEVERR_NONFINITE in *err.
int ingest_launch(int prec, const float* img, void* x, int N, int H, int W, int Cp, unsigned* err, hipStream_t s);
// NCHW fp32 images (3 channels, H and W even) -> 2x2 space-to-depth NHWC
// [N][H/2][W/2][16]: channel (2*dy + dx)*3 + c holds pixel (2i+dy, 2j+dx) of
// channel c; channels 12..15 are zero.
int ingest_s2d_launch(int prec, const float* img, void* x, int N, int H, int W, unsigned* err, hipStream_t s);
// mode 0: OIHW -> [Cout][KHW][Cin_p] (+ [Cin_p][KHW][Cout] when dst_d >= 0);
// mode 1: the 7x7 stride-2 stem (Cin 3) as a 4x4 conv over its 2x2
// space-to-depth input: [Cout][4x4][16], channel (2*dy + dx)*3 + c.
struct RepackEntry { long src; long dst_f; long dst_d; int Cout, Cin, Cin_p, KHW; long n; long nprefix; int mode, pad_; };
// y = bf16(x), round to nearest even, as every kernel stores bf16 (n multiple of 8)
int round_bf16_launch(const float* x, uint16_t* y, long n, hipStream_t s);
// Weight shadows from the fp32 state: entries repacked element by element
// (total elements over them), and entries of kernels with at most 9 taps
// through an LDS-tiled transpose (n = tiles, nprefix = tile prefix; ntiles
// blocks in all).
int repack_launch(int prec, const float* state, void* wf, void* wd, const RepackEntry* table_dev,
                  int nentries, long total, hipStream_t s);
int repack_tiled_launch(int prec, const float* state, void* wf, void* wd, const RepackEntry* table_dev,
                        int nentries, int ntiles, hipStream_t s);
bool repack_tiled_fits(int khw);
int repack_tiles(int cout, int cin_p);
int maxpool_fwd_launch(int prec, const void* x, void* y, uint8_t* arg, int N, int H, int W, int C,
                       int Ho, int Wo, hipStream_t s);
int maxpool_bwd_launch(int prec, const void* dy, const uint8_t* arg, void* dx, int N, int H, int W, int C,
                       int Ho, int Wo, hipStream_t s);
int avgpool_fwd_launch(int prec, const void* x, float* f, int N, int HW, int C, hipStream_t s);
int avgpool_bwd_launch(int prec, const float* df, void* dx, int N, int HW, int C, hipStream_t s);
// C[m][n] = sum_k A(m,k) B(k,n) (+ bias[n]); A(m,k) = A[m*sam + k*sak], B(k,n) = B[k*sbk + n*sbn]
// Classifier GEMM; `part` (gemm_f32_workspace bytes, may be NULL for one
// split) holds split-K partial products.
int gemm_f32_splits(int M, int N, int K);
size_t gemm_f32_workspace(int M, int N, int K);
int gemm_f32_launch(const float* A, long sam, long sak, const float* B, long sbk, long sbn, const float* bias,
                    float* C, int M, int N, int K, float* part, hipStream_t s);
int colsum_launch(const float* A, int M, int N, float* out, hipStream_t s);
// Dynamic loss scaling of the fp16 precision (device state of a context).
struct LossScale {
  float scale;        // current scale, a power of two in [1, 2^24]
  float inv_scale;    // 1 / scale
  unsigned overflow;  // set by the finiteness check of this step's gradient
  unsigned good;      // steps in a row without an overflow
  unsigned interval;  // growth interval: the scale doubles after this many
  unsigned skipped;   // steps skipped because of an overflow
};
// ls != NULL: dz is multiplied by ls->scale.
int softmax_ce_launch(const float* z, const int32_t* labels, int N, int C, float* dz, float* row_loss,
                      float* loss, unsigned* err, hipStream_t s, const LossScale* ls = nullptr);
// In-place dropout of n (a multiple of 4) fp32 values with the Philox4x32-10
// mask of (seed, step) and keep threshold thresh (top 24 bits of a word),
// kept values multiplied by scale.
int dropout_launch(float* x, long n, uint64_t seed, uint64_t step, uint32_t thresh, float scale, hipStream_t s);
// ls != NULL: g holds scale x gradient; the update is skipped after an
// overflow, else g is multiplied by 1/scale.
int sgd_launch(float* w, const float* g, float* v, long n, float lr, float mom, float wd, hipStream_t s,
               const LossScale* ls = nullptr);
int grad_check_launch(const float* g, long n, LossScale* ls, hipStream_t s);
int loss_scale_update_launch(LossScale* ls, hipStream_t s);
int merge_launch(float* p, const float* ds, const float* dl, long n, float f, hipStream_t s);
int delta_launch(const float* pulled, const float* local, float* delta, long n, hipStream_t s);
int fill_zero_launch(void* p, size_t bytes, hipStream_t s);

}  // namespace rn18
