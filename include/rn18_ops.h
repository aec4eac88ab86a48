/* rn18_ops.h - single-operator entry points of the gfx950 ResNet-18 library.
 *
 * These expose the kernels the training step is built from, on the library's
 * internal layouts, so each can be checked against a reference on its own.
 * The operators are those of the ResNet-18 training step (the unit of work of
 * the paper's Sec. 3 and 4 schemes); the paper itself gives no operator
 * formulas, so each follows the textbook definition stated below.
 *
 * Common rules: device pointers, caller-owned, 16-byte aligned; `prec` is
 * RN18_FP32 (float elements) or RN18_BF16 (bf16 elements as uint16 bit
 * patterns); activations are NHWC; channel counts of activation tensors must
 * be multiples of 4 (fp32) or 8 (bf16). Work is enqueued on `hip_stream`.
 * Invalid arguments return RN18_EINVAL before any launch, among them any
 * tensor of more than 2^31 - 2^24 bytes (32-bit byte offsets in the kernels).
 */
#ifndef RN18_OPS_H
#define RN18_OPS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Convolution, no bias, zero padding, square kernel k, stride s, pad p:
 *   y[n,i,j,o] = sum_{c,kh,kw} w[o,kh,kw,c] * x[n, i*s-p+kh, j*s-p+kw, c]
 * x [N][H][W][Cin], w [Cout][k][k][Cin] (OHWI), y [N][Ho][Wo][Cout] with
 * Ho = (H+2p-k)/s + 1. Implicit GEMM on MFMA, fp32 accumulation. */
int rn18op_conv2d_fwd(int prec, const void* x, const void* w_ohwi, void* y, int N, int H, int W, int Cin, int Cout,
                      int k, int s, int p, void* hip_stream);

/* Data gradient (adjoint of the above in x):
 *   dx[n,h,w,c] = sum over (i,j,kh,kw) with i*s-p+kh = h, j*s-p+kw = w of
 *                 w[o,kh,kw,c] * dy[n,i,j,o]
 * dy [N][Ho][Wo][Cout], w_ihwo [Cin][k][k][Cout] (the forward weights with
 * the channel axes exchanged), dx [N][H][W][Cin]. Stride 2 runs as four
 * parity-phase sub-convolutions (no multiplications by inserted zeros). */
int rn18op_conv2d_dgrad(int prec, const void* dy, const void* w_ihwo, void* dx, int N, int H, int W, int Cin,
                        int Cout, int k, int s, int p, void* hip_stream);

/* Weight gradient: dw[o,c,kh,kw] = sum_{n,i,j} dy[n,i,j,o] * x[n,i*s-p+kh,j*s-p+kw,c]
 * written fp32 in OIHW order for the first cin_real of the Cin channels.
 * Needs `workspace` of rn18op_conv2d_wgrad_workspace(...) bytes for the
 * deterministic split-K partial sums. */
size_t rn18op_conv2d_wgrad_workspace(int prec, int N, int H, int W, int Cin, int Cout, int k, int s, int p);
int rn18op_conv2d_wgrad(int prec, const void* dy, const void* x, float* dw_oihw, int N, int H, int W, int Cin,
                        int cin_real, int Cout, int k, int s, int p, void* workspace, size_t workspace_bytes,
                        void* hip_stream);

/* Allocation-free variant of rn18op_conv2d_wgrad, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same kernels and the same result,
 * with the split-K partial sums in a static device array of the library
 * (rn18op_conv2d_wgrad_noalloc_limit() bytes, 48 MiB; each GPU the library
 * runs on holds its own copy until the process ends) instead of a caller
 * workspace. Nothing is allocated or freed. A shape whose partials need more
 * than the limit returns RN18_EINVAL before any launch (every ResNet-18
 * layer of the library's split rule fits). Every call on one GPU shares that
 * GPU's array: calls that overlap on one GPU (different streams, or
 * different threads on one stream's queue without ordering) race. */
size_t rn18op_conv2d_wgrad_noalloc_limit(void);
int rn18op_conv2d_wgrad_noalloc(int prec, const void* dy, const void* x, float* dw_oihw, int N, int H, int W,
                                int Cin, int cin_real, int Cout, int k, int s, int p, void* hip_stream);

/* Max pool 3x3, stride 2, padding 1 (padding never wins):
 *   y[n,i,j,c] = max over the window; arg[n,i,j,c] = kh*3+kw of the FIRST
 *   maximum in row-major (kh,kw) order (uint8).
 * Backward: dx[n,h,w,c] = sum of dy over the outputs whose argmax is (h,w). */
int rn18op_maxpool_fwd(int prec, const void* x, void* y, uint8_t* arg, int N, int H, int W, int C,
                       void* hip_stream);
int rn18op_maxpool_bwd(int prec, const void* dy, const uint8_t* arg, void* dx, int N, int H, int W, int C,
                       void* hip_stream);

/* fp32 -> bf16 storage rounding exactly as every bf16 kernel stores values:
 * round to nearest, ties to even (binary32 -> bfloat16; a NaN stays a NaN).
 * x: n fp32, y: n uint16 bf16 bit patterns, n a multiple of 8, 16-byte
 * aligned device pointers. The oracle's rounding points assume this rule. */
int rn18op_round_bf16(const float* x, uint16_t* y, size_t n, void* hip_stream);

/* Debugging aids (not part of the training path).
 * rn18_debug_set(ctx, RN18_DBG_STOP_BLOCKS, k): later train steps end their
 * backward pass after k residual blocks (no stem backward, no SGD update);
 * k = -1 restores full steps.
 * rn18_debug_copy: copy `bytes` of a workspace tensor of the (N,H,W) plan to
 * the device buffer dst, enqueued on the context's stream. `which` selects
 * the tensor (NHWC in the compute type, or fp32 for grad/mean/rstd),
 * `index` the conv layer (forward order) or the residual block. The
 * backward buffers hold what the last step left there: GA / GB the
 * gradients of block outputs (ping-pong), GZ the data gradient of a block's
 * second conv, GY the stem conv's dY, GYD a projection conv's dY. */
enum {
  RN18_DBG_STOP_BLOCKS = 0,
  /* process-wide: force gather-conv kernel configuration `value` (1..45,
   * see conv.hip) for every forward / data-gradient launch; 0 = automatic.
   * ctx may be NULL for this key. For tuning and for testing every
   * configuration. */
  RN18_DBG_GATHER_CONFIG = 1,
  /* process-wide: force weight-gradient kernel configuration `value`
   * (1..10, see conv.hip); 0 = automatic. Plans built afterwards size their
   * split-K scratch for it. ctx may be NULL. */
  RN18_DBG_WGRAD_CONFIG = 2,
  /* per context: launch each convolution of a training step or eval pass
   * over batch chunks of at most `value` images (0 = only where a tensor
   * would exceed the kernels' 32-bit byte offsets). Plans built before are
   * dropped. For testing the chunked path at small sizes. */
  RN18_DBG_CONV_CHUNK = 3,
  /* per context: value != 0 keeps every launch of a training step on the
   * caller's stream (the weight gradients otherwise run on a second stream
   * beside the data-gradient chain). For timing kernels one at a time. */
  RN18_DBG_SERIAL = 4,
  /* process-wide: split count of the K reduction of every forward and
   * stride-1 data-gradient gather launch of a training step or eval pass
   * (at most the launch's K stages, at most 64; 0 = automatic: only
   * launches with fewer output tiles than the chip has compute units
   * split; 1 = never). Plans built afterwards size their split-K scratch
   * for it. ctx may be NULL. For tuning and for testing the split path. */
  RN18_DBG_GATHER_SPLIT = 5
};
enum {
  RN18_DBG_Y = 0, RN18_DBG_Z1 = 1, RN18_DBG_OUT = 2, RN18_DBG_GA = 3, RN18_DBG_GB = 4, RN18_DBG_GZ = 5,
  RN18_DBG_GY = 6, RN18_DBG_GYD = 7, RN18_DBG_GRAD = 8, RN18_DBG_WF = 9, RN18_DBG_WD = 10,
  RN18_DBG_MEAN = 11, RN18_DBG_RSTD = 12, RN18_DBG_ZSTEM = 13, RN18_DBG_PARG = 14
};
/* rn18_debug_capture(ctx, kind, index, dst, bytes): during later train
 * steps, copy a backward-pass tensor to dst as soon as it is produced:
 * RN18_CAP_DY (index = conv layer: the gradient entering its conv),
 * RN18_CAP_DZ1 (block: data gradient of its second conv), RN18_CAP_DX
 * (block: gradient wrt the block input; in a projection block the data
 * gradients of the first conv and of the projection are summed in one GEMM
 * and rounded once), RN18_CAP_DA_AVG (gradient entering
 * the last block from the average pool), RN18_CAP_DA_POOL (max-pool data
 * gradient). dst = NULL clears every capture. */
enum {
  RN18_CAP_DY = 0, RN18_CAP_DZ1 = 1, RN18_CAP_DX = 3, RN18_CAP_DA_AVG = 4, RN18_CAP_DA_POOL = 5
};
int rn18_debug_capture(struct rn18_ctx* ctx, int kind, int index, void* dst, size_t bytes);
int rn18_debug_set(struct rn18_ctx* ctx, int key, long value);
int rn18_debug_copy(struct rn18_ctx* ctx, int N, int H, int W, int which, int index, void* dst, size_t bytes);

#ifdef __cplusplus
}
#endif
#endif
