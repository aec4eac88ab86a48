/* rn18.h - C ABI of the gfx950 (MI355X) ResNet-18 training-step library.
 *
 * The library computes one ResNet-18 training step (forward, data- and
 * weight-gradient convolutions, batch-norm / ReLU / residual, softmax
 * cross-entropy, SGD with momentum) at any batch size and image resolution,
 * the forward pass alone in inference mode, and the parameter-server merge of
 * a small-batch and a large-batch worker's updates with the model-update
 * factor of dual-batch learning.
 *
 * Paper: "Hybrid Dual-Batch and Cyclic Progressive Learning for Efficient
 * Distributed Training" (arXiv 2509.26092). The training step is the unit of
 * work that the dual-batch (Sec. 3) and cyclic-progressive (Sec. 4) schemes
 * schedule at different (batch, resolution) pairs; SGD is Sec. 2.2, Eq. 1;
 * the parameter-server pull/train/push cycle is Sec. 2.3; the model-update
 * factor is Sec. 3.4.
 *
 * Conventions for every call
 *  - Pointers are DEVICE pointers unless stated otherwise. The caller owns
 *    them (typically torch tensors); the library never frees caller memory.
 *  - Every float pointer must be 16-byte aligned.
 *  - All work of a context is enqueued on that context's HIP stream and is
 *    asynchronous; nothing synchronises the host except rn18_init (when it
 *    writes the initial state), rn18_sync_status, rn18_destroy and the
 *    workspace query functions.
 *  - Errors the host can detect are returned at once, before anything is
 *    launched: RN18_EINVAL for null pointers, non-positive sizes, a layer
 *    whose output would be empty, a batch-norm layer with only one value per
 *    channel (N*Ho*Wo == 1), a shape with a tensor of more than
 *    16 * (2^31 - 2^24) bytes (about 34 GB: the kernels index tensors with
 *    32-bit offsets, and a step launches each convolution over batch chunks
 *    whose tensors stay below 2^31 - 2^24 bytes; at 224x224 an ImageNet bf16
 *    step takes up to 21,232 images, more than 288 GB of memory hold; see
 *    rn18_workspace_bytes), or a non-finite factor. rn18_last_error()
 *    returns a thread-local description of the last non-OK return.
 *  - Errors found on the device (a label outside [0, C), a non-finite image
 *    value or a non-finite loss) set a sticky flag of the context; the call
 *    still runs to completion, and rn18_sync_status reports and clears the
 *    flag.
 *  - No C++ exception crosses this interface.
 */
#ifndef RN18_H
#define RN18_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RN18_OK = 0,
  RN18_EINVAL = -1,
  RN18_ELABEL = -2,
  RN18_ENOMEM = -3,
  RN18_EHIP = -4,
  RN18_ENONFINITE = -5
} rn18_status;

/* Network variants (the paper names ResNet-18, Sec. 5.1.1; the variants are
 * the evaluation's CIFAR-100 32x32 and ImageNet shapes plus a one-block net):
 *  RN18_TINY      3x3 s1 stem 3->16, one BasicBlock 16->16, FC 16->C
 *  RN18_CIFAR     3x3 s1 stem 3->64, no max pool, stages 64/128/256/512 x 2
 *  RN18_IMAGENET  7x7 s2 p3 stem 3->64, 3x3 s2 p1 max pool, same stages
 * BasicBlock = conv3x3(s)-BN-ReLU-conv3x3-BN (+ shortcut) -ReLU; stride 2 in
 * the first conv of stages 2-4; 1x1 stride-s conv + BN shortcut when the
 * stride or width changes. Convs have no bias, the FC has one. */
typedef enum { RN18_TINY = 0, RN18_CIFAR = 1, RN18_IMAGENET = 2 } rn18_arch;

/* RN18_FP32: all tensors fp32 (fp32 MFMA for the convolutions).
 * RN18_BF16: images, conv weights and activations (and their gradients) in
 * bf16 with fp32 accumulation; master weights, momentum, BN statistics, the
 * classifier and the loss in fp32. This is the mixed precision of the
 * paper's ImageNet runs (Sec. 5.2.3), taken as bf16 without loss scaling.
 * RN18_FP16: the same tensors in IEEE fp16 (round to nearest even) with
 * dynamic loss scaling, the 16-bit mixed-precision training that Sec. 5.2.3
 * cites: the backward pass starts from scale x loss, so every stored
 * gradient is scaled; the weight update multiplies the gradient by 1/scale,
 * or is skipped when a gradient value is not finite (an fp16 overflow). The
 * scale (a power of two, initially 65536) halves after a skipped step and
 * doubles after 2000 steps in a row without one (rn18_set_loss_scale). BN
 * running statistics are updated in the forward pass of a skipped step too. */
typedef enum { RN18_FP32 = 0, RN18_BF16 = 1, RN18_FP16 = 2 } rn18_prec;

typedef struct {
  int arch;            /* rn18_arch */
  int num_classes;     /* C >= 1 */
  int prec;            /* rn18_prec */
  float momentum;      /* SGD momentum, e.g. 0.9 */
  float weight_decay;  /* L2 coefficient added to every trainable gradient, e.g. 5e-4 */
  float bn_eps;        /* e.g. 1e-5 */
  float bn_momentum;   /* running-stat update weight, e.g. 0.1 */
} rn18_config;

typedef struct rn18_ctx rn18_ctx; /* opaque: plans, momentum buffer, bf16 weight shadow */

/* Flat parameter state, fp32, in this order:
 *   for every conv in forward order (stem, then per block c1, c2, [ds]):
 *       W [Cout][Cin][KH][KW], gamma [Cout], beta [Cout]
 *   FC weight [C][F], FC bias [C]                      (P trainable floats)
 *   for every BN in the same order: running_mean [Cout], running_var [Cout]
 * Returns P+R and, if n_trainable is not NULL, stores P there.
 * Returns 0 for an invalid config. */
size_t rn18_state_floats(const rn18_config* cfg, size_t* n_trainable);

/* Create a context bound to hip_stream (a hipStream_t; NULL = default
 * stream). If state_out is not NULL, write a He-normal (fan-in) initial state
 * drawn from `seed` (gamma 1, beta 0, FC bias 0, running mean 0, running var
 * 1) and wait for the copy. The momentum buffer starts at zero. */
int rn18_init(const rn18_config* cfg, uint64_t seed, void* hip_stream, float* state_out, rn18_ctx** ctx);

/* Device workspace needed by a train step or eval pass of shape (N,H,W), in
 * bytes. Returns 0 if the shape is invalid. */
size_t rn18_workspace_bytes(rn18_ctx* ctx, int N, int H, int W);

/* Hand the library a caller-allocated device workspace (e.g. a torch uint8
 * tensor). Steps whose workspace does not fit return RN18_ENOMEM. Without
 * this call the library allocates and grows its own workspace. */
int rn18_set_workspace(rn18_ctx* ctx, void* dev, size_t bytes);

/* One training step on `state` (in/out, P+R floats): forward with batch
 * statistics, softmax cross-entropy loss averaged over the batch, backward,
 * BN running-stat update, then g' = g + wd*w, v = mu*v + g', w -= lr*v on all
 * P trainable floats.
 *   images  [N][3][H][W] fp32 (NCHW)
 *   labels  [N] int32 in [0, C)   (out-of-range labels set RN18_ELABEL and
 *                                  contribute neither loss nor gradient)
 *   loss    1 fp32 (device), written with the pre-update loss; may be NULL */
int rn18_train_step(rn18_ctx* ctx, float* state, const float* images, const int32_t* labels, int N, int H, int W,
                    float lr, float* loss);

/* Forward pass in inference mode (BN with the running statistics in
 * `state`); writes logits [N][C] fp32. */
int rn18_eval_logits(rn18_ctx* ctx, const float* state, const float* images, int N, int H, int W, float* logits);

/* Parameter-server merge of dual-batch learning (Sec. 2.3 pull/train/push,
 * Sec. 3.4 model-update factor). g_small and g_large are the update vectors
 * the two workers push, Delta = p_pulled - p_after_local_step (see
 * ps_worker_delta); the server applies
 *     state[i] <- state[i] - (g_large[i] + factor * g_small[i]),  i < n,
 * with factor = d_S/d_L for the paper's scheme (1 for the large worker is
 * implicit). n is normally P+R (the BN running statistics merge by the same
 * rule). g_small/g_large may alias each other but not `state`.
 * RN18_EINVAL if a pointer is NULL or misaligned or factor is not finite. */
int ps_dual_merge(float* state, const float* g_small, const float* g_large, size_t n, float factor, void* hip_stream);

/* delta[i] = pulled[i] - local[i], i < n: the update vector a worker pushes
 * after training on its pulled copy of the global model (Sec. 2.3). */
int ps_worker_delta(const float* pulled, const float* local, float* delta, size_t n, void* hip_stream);

/* Wait for the context's stream; return and clear the sticky device error
 * (RN18_ELABEL, RN18_ENONFINITE) or RN18_OK. */
int rn18_sync_status(rn18_ctx* ctx);

/* Copy the momentum buffer (P floats, device) out / in, for checkpoint and
 * resume of a worker. */
int rn18_get_momentum(rn18_ctx* ctx, float* dst);
int rn18_set_momentum(rn18_ctx* ctx, const float* src);

/* Dropout on the classifier input during training steps (the adaptive
 * regularisation of Sec. 4.1, whose rates 0.1-0.3 rise with the resolution;
 * the paper does not place the dropout, this library puts it before the
 * fully connected layer). p in [0, 1); p = 0 (the default) turns it off.
 * Feature j of sample n is kept in a training step with counter t iff
 *   (x >> 8) >= floor(p * 2^24),  x = word (nF + j) mod 4 of
 *   Philox4x32-10 (Salmon et al., SC'11) with key (seed mod 2^32,
 *   seed div 2^32) and counter (q mod 2^32, q div 2^32, t mod 2^32,
 *   t div 2^32), q = (nF + j) div 4, F the feature width;
 * kept features are multiplied by (float)(1 / (1 - p)) and the backward pass
 * applies the same mask. t starts at `step` and advances by one with every
 * successful rn18_train_step (whether or not dropout is on); evaluation never
 * drops. RN18_EINVAL for a NULL ctx or p outside [0, 1). */
int rn18_set_dropout(rn18_ctx* ctx, float p, uint64_t seed, uint64_t step);

/* Loss scaling of an RN18_FP16 context (RN18_EINVAL for other precisions).
 * rn18_set_loss_scale waits for the context's stream, then sets the scale
 * (a power of two in [1, 2^24]) and the growth interval (steps without an
 * overflow before the scale doubles, >= 1) and clears the counters.
 * rn18_get_loss_scale waits for the stream and reads the current scale and
 * the number of steps skipped because of a non-finite gradient (either
 * pointer may be NULL). */
int rn18_set_loss_scale(rn18_ctx* ctx, float scale, unsigned growth_interval);
int rn18_get_loss_scale(rn18_ctx* ctx, float* scale, uint64_t* skipped_steps);

/* Synchronise and free everything the context allocated. */
void rn18_destroy(rn18_ctx* ctx);

const char* rn18_last_error(void);

/* Measurement. With profiling enabled, every kernel launch group of later
 * calls on the context is bracketed by HIP events on the context stream.
 * rn18_profile_read waits for the stream, returns up to `max` records in
 * launch order (count = the number recorded) and clears them. flops and
 * bytes are the algorithmic work of the launch (real channels only, no
 * padding, no re-reads): multiply-adds x 2 for convolutions and the
 * classifier, compulsory HBM bytes for the streaming kernels. */
enum {
  RN18_K_CONV_FWD = 0, RN18_K_CONV_DGRAD = 1, RN18_K_CONV_WGRAD = 2, RN18_K_WGRAD_REDUCE = 3,
  RN18_K_BN_STATS = 4, RN18_K_BN_APPLY = 5, RN18_K_BN_BWD_REDUCE = 6, RN18_K_BN_BWD_APPLY = 7,
  RN18_K_MAXPOOL = 8, RN18_K_AVGPOOL = 9, RN18_K_HEAD = 10, RN18_K_SGD = 11, RN18_K_PREP = 12
};
typedef struct {
  int cls;       /* RN18_K_* */
  int layer;     /* conv layer in forward order, or a sub-index */
  int tile;      /* convolutions: tile shape BM*1000+BN of the kernel instance */
  int pad_;
  double flops;  /* algorithmic floating-point operations */
  double bytes;  /* algorithmic bytes */
  double ms;     /* event-measured duration */
  char kernel[104]; /* NUL-terminated name of the (first) kernel of the group as a
                       profiler demangles it, namespace dropped and the bf16
                       storage type shown as bf16, e.g.
                       "conv_gather2_kernel<bf16, 128, 128, 2, 4, 2, true>" */
} rn18_prof_rec;
int rn18_profile_enable(rn18_ctx* ctx, int on);
int rn18_profile_read(rn18_ctx* ctx, rn18_prof_rec* out, int max, int* count);

#ifdef __cplusplus
}
#endif
#endif
