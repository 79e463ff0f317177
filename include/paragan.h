/*
 * paragan.h -- C ABI of libparagan, the MI355X (gfx950) hot path of ParaGAN's
 * per-replica BigGAN training: spectrally normalised convolutions,
 * class-conditional BatchNorm, ReLU, nearest-upsample / avg-pool, the
 * self-attention block, the hinge loss and the D:G train step.
 *
 * The paper (ParaGAN, SoCC'24) trains BigGAN data-parallel: every replica
 * runs the generator and discriminator forward and backward passes on its
 * share of the batch, then synchronises gradients (Design, "Computation
 * Model").  This library is that per-replica compute on one GPU.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Status: every call returns PARAGAN_OK (0) or a negative PARAGAN_E*
 *   code.  Arguments are validated on the host before anything is enqueued:
 *   on error nothing has been launched and paragan_last_error() names the
 *   problem.  No C++ exception crosses the ABI.
 * - Streams: all device work is enqueued on the hipStream_t given to
 *   paragan_create(), in order; paragan_train_step and paragan_async_step
 *   also use a second stream of the context, and with
 *   paragan_set_overlap_wgrad on the step calls use a third (default
 *   priority, created on first use), ordered by events and idle again when
 *   the call returns, also on error.  Calls are asynchronous unless
 *   stated.
 * - Memory: every device buffer is allocated and owned by the caller and
 *   passed as a plain device pointer.  The library allocates no device
 *   memory; its one device-resident object is the fixed 4 MiB scratch
 *   array of paragan_sn_power_iter_noalloc, part of the loaded code.
 *   Sizes of the "saved" (forward -> backward) and "ws" (scratch) buffers
 *   come from the *_sizes() queries and must be 256-byte aligned.
 * - Activations are NHWC.  Their channel stride is the channel count
 *   rounded up to a multiple of 32 (paragan_cpad()); padded channels hold
 *   zeros on input and are written as zeros.  dtype PARAGAN_BF16 means
 *   bfloat16 activations with fp32 accumulation; PARAGAN_F32 means fp32
 *   throughout.
 * - Parameters of a module (block or network) live in ONE flat fp32 buffer
 *   in the order given by paragan_*_layout(); gradients and the Adam moments
 *   use the same layout.  Convolution weights are [Cout][kh][kw][Cin],
 *   linear weights [out][in], embeddings [classes][dim].  Spectral
 *   normalisation keeps one persistent fp32 vector u (length = the weight's
 *   row count, Cout) per SN weight in a separate flat "u" buffer, in
 *   layout order; training-mode forwards update it in place.
 * - Threading: a context is used by one host thread at a time.
 */
#ifndef PARAGAN_H
#define PARAGAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  PARAGAN_OK = 0,
  PARAGAN_EINVAL = -1,        /* bad argument: null pointer, bad shape, ... */
  PARAGAN_EUNSUPPORTED = -2,  /* valid request this build does not handle */
  PARAGAN_EWORKSPACE = -3,    /* a buffer is smaller than the query said */
  PARAGAN_EHIP = -4,          /* a HIP runtime call failed */
  PARAGAN_ENONFINITE = -5,    /* train step produced a NaN/Inf loss */
  PARAGAN_ETIMEOUT = -6       /* a bounded wait ended without its event */
};

enum { PARAGAN_F32 = 0, PARAGAN_BF16 = 1 };

typedef struct paragan_ctx paragan_ctx;

/* Create a context bound to `hip_stream` (a hipStream_t; NULL = the null
 * stream) on the current device.  Checks that the device is gfx950. */
int paragan_create(paragan_ctx** out, void* hip_stream);
void paragan_destroy(paragan_ctx* ctx);
/* Message of the last failed call on this context (or of the last failed
 * paragan_create when ctx is NULL).  Valid until the next call. */
const char* paragan_last_error(const paragan_ctx* ctx);
/* Block until all work enqueued by this context has finished. */
int paragan_sync(paragan_ctx* ctx);
/* Off (0, the default) or on (1): whether the step calls (paragan_g_sample,
 * paragan_d_step, paragan_g_step, paragan_train_step) run the weight
 * gradients of each block backward -- with their bias column sums -- on a
 * further stream of the context (default priority), beside the block's
 * data gradients on the context's stream, ordered by events and joined
 * before the block's SN backward; every call returns with both streams
 * joined (also on error).  Results are bit-identical either way.  On, the
 * data- and weight-gradient kernels share the CUs, so a step finishes
 * sooner while each kernel's own launch takes longer: per-kernel rates
 * measured with it on count the shared time.  Returns PARAGAN_EINVAL for
 * other values. */
int paragan_set_overlap_wgrad(paragan_ctx* ctx, int on);

/* Channel stride of an activation tensor with c channels. */
int64_t paragan_cpad(int64_t c);

/* One entry of a parameter layout. */
typedef struct {
  char name[48];       /* e.g. "g0.conv1.w" */
  int32_t ndim;
  int64_t shape[4];
  int64_t offset;      /* in floats, into the flat parameter buffer */
  int64_t u_offset;    /* in floats, into the flat u buffer; -1 if no SN */
} paragan_tensor_info;

/* ---------------------------------------------------------------------
 * Spectral normalisation (BigGAN's SN, as cited in Related Work): one
 * power iteration per training forward,
 *     v <- N(W^T u),  u <- N(W v),  sigma = u^T W v,   N(t) = t / max(|t|, eps),
 * repeated n_iter times.  W: device fp32, row-major rows x cols (the
 * weight viewed as (Cout, kh*kw*Cin)).  u: device fp32 [rows], read and
 * overwritten.  v: device fp32 [cols], written.  sigma: device fp32 scalar,
 * written.  rows, cols >= 1; n_iter >= 1.  ws: device scratch of
 * paragan_sn_ws_size() bytes, 256-byte aligned.
 * ------------------------------------------------------------------- */
int paragan_sn_ws_size(int64_t rows, int64_t cols, size_t* ws_bytes);
/* Validation only (no device work): the checks paragan_sn_power_iter makes
 * of its sizes and scalars. */
int paragan_sn_check(int64_t rows, int64_t cols, int n_iter, float eps);
int paragan_sn_power_iter(paragan_ctx* ctx, const float* W, int64_t rows,
                          int64_t cols, float* u, float* v, float* sigma,
                          int n_iter, float eps, void* ws);
/* For callers that cannot allocate device memory (code under stream
 * capture, serving loops, harnesses that forbid hipMalloc): the same
 * computation, with the same kernels and results, as paragan_sn_power_iter,
 * but its scratch is a 4 MiB array the library holds on each device until
 * the process ends (its address taken in paragan_create), so the caller
 * passes no workspace and the call allocates nothing.  Every BigGAN-128 and
 * BigGAN-512 SN weight fits (the largest needs about 1 MiB); a weight whose
 * paragan_sn_ws_size() exceeds 4 MiB is rejected with PARAGAN_EINVAL before
 * any work.  All calls on one device share that one array: calls that
 * overlap on a device (two streams, two threads, two contexts) race and
 * must be ordered by the caller.  The kernels write all scratch they read,
 * so nothing has to be cleared between calls. */
int paragan_sn_power_iter_noalloc(paragan_ctx* ctx, const float* W,
                                  int64_t rows, int64_t cols, float* u,
                                  float* v, float* sigma, int n_iter,
                                  float eps);

/* ---------------------------------------------------------------------
 * BigGAN generator residual block (spec block of the benchmark
 * model, Evaluation "Experiment Setup"):
 *   y = conv3x3(ReLU(cBN2(h1))) + b2 + conv1x1(up2(x)) + bsc,
 *   h1 = conv3x3(up2(ReLU(cBN1(x)))) + b1,
 *   cBN_k(t) = (1 + cond Wg_k^T) * BN(t) + cond Wb_k^T  (batch statistics),
 * every weight spectrally normalised.  x: [B][H][W][cpad(cin)], y:
 * [B][2H][2W][cpad(cout)], cond: fp32 [B][dc].  Parameter order from
 * paragan_gblock_layout(): bn1.gain bn1.bias conv1.w conv1.b bn2.gain
 * bn2.bias conv2.w conv2.b sc.w sc.b.
 * ------------------------------------------------------------------- */
typedef struct {
  int32_t B, H, W;       /* input batch and spatial size (H, W >= 1) */
  int32_t cin, cout, dc; /* channels in/out, width of cond */
  int32_t dtype;         /* PARAGAN_BF16 or PARAGAN_F32 */
  int32_t n_power_iter;  /* >= 1 */
  float bn_eps, sn_eps;
} paragan_gblock_desc;

int paragan_gblock_layout(const paragan_gblock_desc* d,
                          paragan_tensor_info* out, int32_t cap,
                          int32_t* count, int64_t* n_params, int64_t* n_u);
int paragan_gblock_sizes(const paragan_gblock_desc* d, size_t* saved_bytes,
                         size_t* ws_bytes);
int paragan_gblock_check(const paragan_gblock_desc* d);
/* Training forward: updates u, writes y and `saved` (read by bwd). */
int paragan_gblock_fwd(paragan_ctx* ctx, const paragan_gblock_desc* d,
                       const float* params, float* u, const void* x,
                       const float* cond, void* y, void* saved, void* ws);
/* Backward from dy ([B][2H][2W][cpad(cout)]): writes dx (x's shape),
 * dcond (fp32 [B][dc]) and grads (flat, parameter layout; overwritten). */
int paragan_gblock_bwd(paragan_ctx* ctx, const paragan_gblock_desc* d,
                       const float* params, const void* x, const float* cond,
                       const void* saved, const void* dy, void* dx,
                       float* dcond, float* grads, void* ws);

/* ---------------------------------------------------------------------
 * BigGAN discriminator residual block (the benchmark model's
 * discriminator, Evaluation "Experiment Setup"; its size pinned by Table
 * tab:GAN's 158.42M parameters):
 *   h = conv3x3([ReLU](x)) + b1,  main = [avgpool2](conv3x3(ReLU(h)) + b2),
 *   y = main + skip,  skip = conv1x1([avgpool2](x)) + bsc (learnable) or x.
 * x: [B][H][W][cpad(cin)] (bf16, or fp32 images when cin <= 4 and
 * x_f32), y: [B][H'][W'][cpad(cout)].  Parameters: conv1.w conv1.b
 * conv2.w conv2.b [sc.w sc.b].
 * ------------------------------------------------------------------- */
typedef struct {
  int32_t B, H, W, cin, cout;
  int32_t preact;        /* ReLU on the input of conv1 */
  int32_t downsample;    /* 2x2 avg-pool (H, W even) */
  int32_t learnable_sc;  /* 1x1 conv skip; required if cin != cout or pooled */
  int32_t dtype;
  int32_t n_power_iter;
  float sn_eps;
} paragan_dblock_desc;

int paragan_dblock_layout(const paragan_dblock_desc* d,
                          paragan_tensor_info* out, int32_t cap,
                          int32_t* count, int64_t* n_params, int64_t* n_u);
int paragan_dblock_sizes(const paragan_dblock_desc* d, size_t* saved_bytes,
                         size_t* ws_bytes);
int paragan_dblock_check(const paragan_dblock_desc* d);
int paragan_dblock_fwd(paragan_ctx* ctx, const paragan_dblock_desc* d,
                       const float* params, float* u, const void* x, void* y,
                       void* saved, void* ws);
/* dx may be NULL (input gradient not wanted). */
int paragan_dblock_bwd(paragan_ctx* ctx, const paragan_dblock_desc* d,
                       const float* params, const void* x, const void* saved,
                       const void* dy, void* dx, float* grads, void* ws);

/* ---------------------------------------------------------------------
 * Self-attention block of the benchmark BigGAN (Evaluation, "Experiment
 * Setup"; one per network at 64x64, counted in Table tab:GAN's 158.42M),
 * bf16 only:
 *   theta = x Wt^T (C/8), phi = maxpool2(x Wp^T) (C/8), g = maxpool2(x Wg^T)
 *   (C/2), P = softmax over keys of theta phi^T (no scaling),
 *   y = x + gamma * (P g) Wo^T.  SN on Wt Wp Wg Wo; gamma has none.
 * x, y: [B][H][W][cpad(C)], H and W even, C a multiple of 8.
 * Parameters: theta phi g o gamma.
 * ------------------------------------------------------------------- */
typedef struct {
  int32_t B, H, W, C;
  int32_t n_power_iter;
  float sn_eps;
} paragan_attn_desc;

int paragan_attn_layout(const paragan_attn_desc* d, paragan_tensor_info* out,
                        int32_t cap, int32_t* count, int64_t* n_params,
                        int64_t* n_u);
int paragan_attn_sizes(const paragan_attn_desc* d, size_t* saved_bytes,
                       size_t* ws_bytes);
int paragan_attn_check(const paragan_attn_desc* d);
int paragan_attn_fwd(paragan_ctx* ctx, const paragan_attn_desc* d,
                     const float* params, float* u, const void* x, void* y,
                     void* saved, void* ws);
int paragan_attn_bwd(paragan_ctx* ctx, const paragan_attn_desc* d,
                     const float* params, const void* x, const void* saved,
                     const void* dy, void* dx, float* grads, void* ws);

/* ---------------------------------------------------------------------
 * Generator output layer (the last generator layer of the model,
 * Evaluation "Experiment Setup"; kept in fp32 arithmetic by the paper's
 * mixed-precision placement, Design "System Optimizations"):
 *   a = ReLU(gain * BN(x) + bias)   (batch statistics over B, H, W),
 *   img = tanh(conv3x3(a, W / sigma(W)) + b)   (3 output channels),
 * with SN on W.  x: bf16 [B][H][W][cpad(C)]; img: fp32 [B][H][W][3].
 * Shapes: cpad(C) <= 128 and W a multiple of 4 (paragan_gout_check says
 * whether W also fits the weight-gradient tile; every W up to 704 does).
 * Parameters: out_bn.gain out_bn.bias out_conv.w out_conv.b.
 * ------------------------------------------------------------------- */
typedef struct {
  int32_t B, H, W, C;
  int32_t n_power_iter;
  float bn_eps, sn_eps;
} paragan_gout_desc;

int paragan_gout_layout(const paragan_gout_desc* d, paragan_tensor_info* out,
                        int32_t cap, int32_t* count, int64_t* n_params,
                        int64_t* n_u);
int paragan_gout_sizes(const paragan_gout_desc* d, size_t* saved_bytes,
                       size_t* ws_bytes);
int paragan_gout_check(const paragan_gout_desc* d);
/* Training forward: updates u, writes img and `saved` (read by bwd). */
int paragan_gout_fwd(paragan_ctx* ctx, const paragan_gout_desc* d,
                     const float* params, float* u, const void* x, float* img,
                     void* saved, void* ws);
/* Backward from dimg (fp32 [B][H][W][3]); img is this layer's forward
 * output.  Writes dx (bf16, x's shape) and grads (flat, parameter layout;
 * overwritten). */
int paragan_gout_bwd(paragan_ctx* ctx, const paragan_gout_desc* d,
                     const float* params, const void* x, const float* img,
                     const void* saved, const float* dimg, void* dx,
                     float* grads, void* ws);

/* ---------------------------------------------------------------------
 * Optimisers.  The paper trains the two networks with different optimisers
 * (Numerical Optimizations, "Asymmetric Optimization Policy": AdaBelief for
 * the generator and Adam for the discriminator converge to the better
 * equilibrium).  Each network carries its own optimiser, on fp32 master
 * weights, with bias correction and no weight decay; t counts the steps
 * taken (the update computes step t + 1):
 *   Adam:       m = b1 m + (1 - b1) g,  v = b2 v + (1 - b2) g^2,
 *               p -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)
 *   AdaBelief (Zhuang et al., NeurIPS 2020, the method the paper cites):
 *               m = b1 m + (1 - b1) g,  s = b2 s + (1 - b2) (g - m)^2 + eps,
 *               p -= lr (m / (1 - b1^t)) / (sqrt(s / (1 - b2^t)) + eps)
 * ------------------------------------------------------------------- */
enum { PARAGAN_ADAM = 0, PARAGAN_ADABELIEF = 1 };

typedef struct {
  int32_t kind;         /* PARAGAN_ADAM or PARAGAN_ADABELIEF */
  float lr, beta1, beta2, eps;   /* lr >= 0, 0 <= beta < 1, eps > 0 */
} paragan_optim;

/* ---------------------------------------------------------------------
 * Full BigGAN networks and the G+D training iteration.  The architecture
 * is given by channel multipliers (BigGAN-128: ch 96, G 16,16,8,4,2,1, D
 * 1,2,4,8,16,16 with the last D block not pooling, attention at 64x64, 1000
 * classes, z 120 split into 6 chunks of 20, shared class embedding 128;
 * Evaluation, "Experiment Setup").  Hinge loss:
 *   L_D = mean relu(1 - D(x_real, y_real)) + mean relu(1 + D(x_fake, y_fake)),
 *   L_G = -mean D(G(z, y), y).
 * ------------------------------------------------------------------- */
typedef struct {
  int32_t img;          /* output resolution */
  int32_t ch;           /* base width */
  int32_t n_g;          /* generator blocks */
  int32_t g_mult[10];   /* n_g + 1 entries: C0 mult, then each block's out */
  int32_t n_d;          /* discriminator blocks */
  int32_t d_mult[10];   /* n_d entries */
  int32_t d_down[10];   /* n_d entries, 0/1 */
  int32_t attn_res;     /* 0: none */
  int32_t n_classes, dz, shared_dim;
  int32_t B;            /* per-GPU batch (D steps see 2B images) */
  int32_t n_power_iter;
  float bn_eps, sn_eps;
  paragan_optim opt_g, opt_d;   /* the generator's and the discriminator's */
} paragan_biggan_desc;

/* which = 0: generator, 1: discriminator. */
int paragan_net_layout(const paragan_biggan_desc* d, int32_t which,
                       paragan_tensor_info* out, int32_t cap, int32_t* count,
                       int64_t* n_params, int64_t* n_u);
int paragan_biggan_check(const paragan_biggan_desc* d);
/* Workspace of every step call below (one size serves them all). */
int paragan_train_step_ws_size(const paragan_biggan_desc* d, size_t* ws_bytes);

typedef struct {
  float* params;   /* flat fp32 master weights (updated by the optimiser) */
  float* u;        /* flat SN vectors (updated by every forward) */
  float* grads;    /* flat fp32: the last gradient computed (overwritten) */
  float* opt_m;    /* flat fp32 first moments */
  float* opt_v;    /* flat fp32 second moments (Adam's v, AdaBelief's s) */
  int64_t opt_t;   /* optimiser steps taken so far (host; incremented) */
} paragan_net_state;

/* Generator forward in training mode (batch statistics, SN u updated):
 * img (fp32 [B][img][img][3], in [-1, 1]) = G(z, y); z fp32 [B][dz], y [B].
 * No parameter changes other than u. */
int paragan_g_sample(paragan_ctx* ctx, const paragan_biggan_desc* d,
                     paragan_net_state* G, const float* z, const int32_t* y,
                     float* img, void* ws);

/* One discriminator step on supplied images: D forward, hinge, backward on
 * the batch concat(x_real, x_fake) with labels concat(y_real, y_fake)
 * (inputs sharing a weight are batched, Implementation "Hardware-Aware
 * Layout Transformation"), then D's optimiser.  x_real, x_fake: fp32
 * [B][img][img][3].  Writes D's gradients and L_D (loss_host, one float);
 * synchronises the stream at the end.  Returns PARAGAN_ENONFINITE (after
 * finishing the step) if L_D is not finite. */
int paragan_d_step(paragan_ctx* ctx, const paragan_biggan_desc* d,
                   paragan_net_state* D, const float* x_real,
                   const int32_t* y_real, const float* x_fake,
                   const int32_t* y_fake, void* ws, float* loss_host);

/* One generator step: G forward on (z, y), D forward (D's u updated, its
 * weights and optimiser state untouched), hinge L_G, D backward for the
 * input gradient only, G backward, G's optimiser.  Writes G's gradients and
 * L_G (loss_host); synchronises at the end; PARAGAN_ENONFINITE as above. */
int paragan_g_step(paragan_ctx* ctx, const paragan_biggan_desc* d,
                   paragan_net_state* G, paragan_net_state* D, const float* z,
                   const int32_t* y, void* ws, float* loss_host);

typedef struct {
  /* n_D entries each: */
  const float* const* x_real;   /* fp32 [B][img][img][3] images in [-1,1] */
  const int32_t* const* y_real; /* [B] */
  const float* const* z_fake;   /* fp32 [B][dz] */
  const int32_t* const* y_fake; /* [B] */
  const float* z_g;             /* fp32 [B][dz] for the generator step */
  const int32_t* y_g;           /* [B] */
} paragan_step_inputs;

/* One training iteration: n_D discriminator steps, each on
 * concat(real_k, G(z_k, y_k)) with labels concat(y_real_k, y_fake_k) -- the
 * same as paragan_g_sample followed by paragan_d_step -- then one generator
 * step on (z_g, y_g) as paragan_g_step; the D:G ratio n_D (1..63) is the
 * caller's (Numerical Optimizations, "Asynchronous Update Scheme": the
 * ratio is adjustable).  The results equal that sequence of calls bit for
 * bit.  Besides the context's stream the call uses a second stream of the
 * context (default priority), ordered by events, for the forwards' SN power
 * iterations and weight packing, which read only parameters; both streams
 * are idle when the call returns, also on error.  losses_host: n_D + 1
 * floats (L_D per D step, then L_G).  Returns PARAGAN_ENONFINITE (after
 * finishing the step) if a loss is not finite. */
int paragan_train_step(paragan_ctx* ctx, const paragan_biggan_desc* d,
                       paragan_net_state* G, paragan_net_state* D,
                       const paragan_step_inputs* in, int32_t n_D, void* ws,
                       float* losses_host);

/* ---------------------------------------------------------------------
 * The asynchronous update scheme (Numerical Optimizations, "Asynchronous
 * Update Scheme"), on one GPU.  One call is one iteration:
 *   1. the discriminator's parameters and SN vectors are copied to a
 *      snapshot held in the workspace;
 *   2. on the context's second stream: a generator step of batch n_D * B on
 *      (z, y) against the snapshot, as paragan_g_step (the snapshot's SN
 *      vectors advance and are discarded with it); its samples G(z, y),
 *      their labels and the snapshot's predictions D_snap(G(z, y)) are kept;
 *   3. concurrently on the context's stream: n_D discriminator steps, step k
 *      as paragan_d_step on x_real[k], y_real[k] and the k-th B samples and
 *      labels of img_buff / lab_buff -- the previous iteration's samples, so
 *      the discriminator sees fakes one generator update stale;
 *   4. after both: img_buff, lab_buff and pred_buff are replaced with this
 *      iteration's samples, labels and predictions.
 * The caller fills img_buff / lab_buff before the first iteration (e.g.
 * with paragan_g_sample).  Together the two sides need about the memory of
 * two generator steps and one discriminator step.
 *   x_real, y_real: n_D device pointers each (fp32 [B][img][img][3], [B]);
 *   z, y:           fp32 [n_D B][dz] and [n_D B] (the generator's batch);
 *   img_buff:       fp32 [n_D B][img][img][3], read then replaced;
 *   lab_buff:       [n_D B], read then replaced;
 *   pred_buff:      fp32 [n_D B], written.
 * losses_host: n_D + 1 floats (L_D per D step, then L_G against the
 * snapshot).  Both streams are idle when the call returns, also on error;
 * PARAGAN_ENONFINITE (after finishing the iteration) if a loss is not
 * finite.  ws: paragan_async_ws_size() bytes, 256-byte aligned.
 * ------------------------------------------------------------------- */
typedef struct {
  const float* const* x_real;
  const int32_t* const* y_real;
  const float* z;
  const int32_t* y;
  float* img_buff;
  int32_t* lab_buff;
  float* pred_buff;
} paragan_async_inputs;

int paragan_async_ws_size(const paragan_biggan_desc* d, int32_t n_D, size_t* ws_bytes);
int paragan_async_step(paragan_ctx* ctx, const paragan_biggan_desc* d,
                       paragan_net_state* G, paragan_net_state* D,
                       const paragan_async_inputs* in, int32_t n_D, void* ws,
                       float* losses_host);

/* ---------------------------------------------------------------------
 * Congestion-aware host data pipeline (Implementation, "Congestion-Aware
 * Data Pipelining").  Host threads fetch batches (by calling `fetch`) into
 * caller-provided host slots ahead of the consumer.  A sliding window holds
 * the latency of the last `window` fetches; once `window` fetches have
 * completed since the last change, a window mean above threshold_ms adds
 * one fetch thread and one batch of prefetch depth (up to the maxima), and a
 * mean at or below it releases one of each (down to the minima).  Depth
 * counts every batch a thread has claimed and the consumer has not yet
 * released.  Batches are delivered in sequence order 0, 1, 2, ..., each
 * exactly once, whatever the number of threads.  Host code only (no device
 * work, usable without a GPU); the caller copies a delivered slot to the
 * device (from pinned memory for an asynchronous copy) and then releases it.
 * Thread-safety: one consumer thread calls next, release and get_stats.
 * ------------------------------------------------------------------- */
/* Fill `slot` (slot_bytes bytes) with batch `seq`; return 0 on success.
 * Called from pipeline threads, concurrently for different seq. */
typedef int (*paragan_fetch_fn)(void* user, int64_t seq, void* slot, size_t slot_bytes);

typedef struct {
  int32_t min_threads, max_threads;   /* 1 <= min <= max <= 64 */
  int32_t min_depth, max_depth;       /* 1 <= min <= max <= n_slots */
  int32_t window;                     /* latency samples, 1 .. 100000 */
  double threshold_ms;                /* > 0 */
} paragan_pipeline_cfg;

typedef struct {
  int32_t threads, depth;             /* the controller's current targets */
  double window_mean_ms;              /* mean latency over the window */
  int64_t fetched, delivered;
  int64_t grows, shrinks;             /* controller adjustments so far */
  double consumer_wait_ms;            /* total time next() has waited */
} paragan_pipeline_stats;

typedef struct paragan_pipeline paragan_pipeline;

/* slots: n_slots host pointers of slot_bytes each, owned by the caller and
 * valid until paragan_pipeline_destroy returns.  Starts min_threads threads. */
int paragan_pipeline_create(paragan_pipeline** out, const paragan_pipeline_cfg* cfg,
                            paragan_fetch_fn fetch, void* user, void* const* slots,
                            int32_t n_slots, size_t slot_bytes);
/* Wait for the next batch in sequence order (timeout_ms < 0: no limit):
 * *seq, *slot.  The slot belongs to the consumer until released.
 * PARAGAN_ETIMEOUT if nothing came in time; PARAGAN_EINVAL when the batch
 * due is one whose fetch failed (the batches before it are delivered first;
 * nothing after it is fetched; the message names the batch). */
int paragan_pipeline_next(paragan_pipeline* p, int64_t* seq, int32_t* slot, int32_t timeout_ms);
int paragan_pipeline_release(paragan_pipeline* p, int32_t slot);
int paragan_pipeline_get_stats(paragan_pipeline* p, paragan_pipeline_stats* out);
/* Message of the last failed call on p (p = NULL: of the last failed
 * paragan_pipeline_create). */
const char* paragan_pipeline_error(const paragan_pipeline* p);
/* Stops the threads (a fetch in progress finishes first) and frees p. */
void paragan_pipeline_destroy(paragan_pipeline* p);

/* Seeded synthetic batches standing in for the image dataset: B images of
 * img x img x 3 floats then B int32 labels per slot.  Value i of batch seq
 * is 2u - 1 with u the top 24 bits of SplitMix64(seed + 2^40 seq + i) over
 * 2^24 (Steele, Lea and Flood, OOPSLA 2014: add 0x9E3779B97F4A7C15, then
 * the finaliser); label b is SplitMix64(seed + 2^40 seq + 2^39 + b) mod
 * n_classes.  latency_ms (host, n_latency entries, may be NULL) injects a
 * delay: fetching batch seq takes at least latency_ms[seq % n_latency]. */
typedef struct {
  uint64_t seed;
  int32_t B, img, n_classes;
  const float* latency_ms;
  int64_t n_latency;
} paragan_synth_source;

size_t paragan_synth_batch_bytes(const paragan_synth_source* s);
/* A paragan_fetch_fn with user = a paragan_synth_source*. */
int paragan_synth_fetch(void* user, int64_t seq, void* slot, size_t slot_bytes);

/* ---------------------------------------------------------------------
 * Launch profiler (instrumentation for the roofline report).  When enabled,
 * every convolution, weight-gradient and attention launch is bracketed by a
 * HIP event pair on the stream it runs on and tagged with its kernel
 * template instance and algorithmic FLOPs (real, unpadded channels); the
 * bandwidth-bound launches (SN power iteration and backward, weight packing,
 * BN statistics / apply / backward, column sums, pooling, the optimisers)
 * are tagged with their algorithmic HBM bytes instead.  Launches on the
 * context's second stream overlap the first, so their times include waiting
 * for CUs the other stream holds.
 * paragan_profile_read synchronises the stream, aggregates the records by
 * kernel name into `out` (up to `cap` entries; *count = number of kernels)
 * and clears them.  Off by default; costs two event records per launch.
 * enable = 1 turns it on; enable = 2 also appends each convolution and
 * weight-gradient launch's GEMM shape "[M,N,K]" to its name (rows =
 * pixels, N = padded output channels, K = padded taps x input channels),
 * so launches of one template instance aggregate per shape; 0 turns it off.
 * ------------------------------------------------------------------- */
typedef struct {
  char name[64];
  int64_t launches;
  double total_ms;
  double flops;
  double bytes;     /* algorithmic HBM bytes of the bandwidth-bound launches
                       (SN, packing, BN, column sums, pooling, optimiser) */
} paragan_kernel_stat;

int paragan_profile(paragan_ctx* ctx, int enable);
int paragan_profile_read(paragan_ctx* ctx, paragan_kernel_stat* out,
                         int32_t cap, int32_t* count);

#ifdef __cplusplus
}
#endif
#endif /* PARAGAN_H */
