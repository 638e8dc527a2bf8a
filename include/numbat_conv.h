/*
 * numbat_conv.h -- C ABI of the Conv2d + BatchNorm(train) + SiLU hot path for
 * AMD Instinct MI355X (gfx950).
 *
 * The operations are those of the Conv -> BN -> SiLU block that makes up the
 * YOLOv8m-class detector of the paper's case study (Sec. 6.1), trained with
 * mixed precision as in Sec. 3.2 and Table 1 (precision row): convolutions in
 * 16-bit floating point (here bf16) with fp32 accumulation, batch
 * normalisation and its statistics in fp32, fp32 weight gradients (master
 * weights are fp32).  Operator semantics follow the reference defaults of
 * Sec. 3 (iv): the convolution is a cross-correlation with zero padding and no
 * bias, BN uses the biased batch variance to normalise and the unbiased one
 * for running statistics, SiLU(z) = z * sigmoid(z).
 *
 * Boundary conventions (Sec. 4, the C ABI layer): plain pointers and sizes,
 * runtime-checked problem descriptors carrying their own struct_size (the ABI
 * is versioned and only ever grows), status codes with thread-local detail
 * text, caller-owned memory.  The library allocates no device memory: every
 * buffer, including scratch workspace, is passed in by the caller.  Interfaces
 * refuse before touching data (Sec. 5): every check completes before anything
 * is enqueued, so a call that returns an error has launched nothing.
 *
 * Memory layouts
 *   activations  NHWC bf16.  A tensor is N*H*W "pixels"; pixel i starts at
 *                element i * pixel_stride, its channels are contiguous.  A
 *                pixel stride larger than the channel count describes a
 *                channel slice of a wider tensor (split / concat views).
 *   conv weights OHWI bf16 [c_out][kh][kw][c_in], dense.
 *   weight grads OHWI fp32 [c_out][kh][kw][c_in], dense.
 *   BN vectors   fp32 [c].
 * Alignment: every bf16 tensor pointer and pixel stride must allow 16-byte
 * vector access: pointers 16-byte aligned, pixel strides and channel counts
 * multiples of 8 (the one exception is a 3-channel image input to the
 * convolution, for which x may be 2-byte aligned with pixel stride >= 3).
 *
 * Streams: `stream` is a hipStream_t passed as void* (NULL = default stream).
 * All work is enqueued on it, nothing synchronises; results are valid once the
 * stream reaches the enqueued work.  Device-side faults surface at the
 * caller's next synchronisation.
 *
 * Determinism: for the same inputs, problem and device model every output is
 * bitwise identical from run to run (all reductions use a fixed order; no
 * floating-point atomics), in the spirit of the paper's bitwise-reproducible
 * gradient reduction (Sec. 3.2, DDP).
 */
#ifndef NUMBAT_CONV_H
#define NUMBAT_CONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define NUMBAT_ABI_VERSION 1u

typedef enum {
  NUMBAT_OK = 0,
  NUMBAT_ERR_NULL = 1,        /* a required pointer is NULL */
  NUMBAT_ERR_BAD_DESC = 2,    /* a descriptor field is out of range or inconsistent */
  NUMBAT_ERR_UNSUPPORTED = 3, /* well-formed but not provided (e.g. channels not a multiple of 8) */
  NUMBAT_ERR_ALIGN = 4,       /* pointer or pixel stride breaks the alignment rules above */
  NUMBAT_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than numbat_workspace_size() */
  NUMBAT_ERR_DEVICE = 6,      /* a HIP runtime call failed; detail holds the HIP error text */
  NUMBAT_ERR_VERSION = 7      /* struct_size does not match this library's descriptor */
} numbat_status;

typedef enum {
  NUMBAT_OP_CONV_FWD = 0,
  NUMBAT_OP_CONV_BWD_DATA = 1,
  NUMBAT_OP_CONV_BWD_WEIGHT = 2,
  NUMBAT_OP_BN_SILU_FWD = 3,
  NUMBAT_OP_BN_SILU_BWD = 4,
  NUMBAT_OP_CLIP_SGD_NESTEROV = 5, /* problem ignored (may be NULL) */
  NUMBAT_OP_CONV_BWD_DATA_BN_SILU = 6 /* numbat_conv_bwd_data_bn_silu_prologue: 0 bytes, or
                                         NUMBAT_ERR_UNSUPPORTED for a problem it does not take */
} numbat_op;

/* One 2-D convolution (dilation 1, one group).  Output size
 * ho = (h + 2*pad_h - kh) / stride_h + 1, wo likewise.  Provided: kernel sides kh, kw <= 5,
 * strides <= 4, padding smaller than the kernel, c_out a multiple of 8, c_in a multiple of
 * 8 or below 8; anything else returns NUMBAT_ERR_UNSUPPORTED. */
typedef struct {
  uint32_t struct_size;   /* = sizeof(numbat_conv_problem) */
  int32_t n, h, w;        /* batch and input spatial size */
  int32_t c_in, c_out;
  int32_t kh, kw;
  int32_t stride_h, stride_w;
  int32_t pad_h, pad_w;
  int64_t x_pixel_stride; /* elements between pixels of x and dx; 0 means c_in */
  int64_t y_pixel_stride; /* elements between pixels of y and dy; 0 means c_out */
} numbat_conv_problem;

/* Batch normalisation over m rows (pixels) of c channels, followed by SiLU. */
typedef struct {
  uint32_t struct_size;    /* = sizeof(numbat_bn_problem) */
  int32_t c;               /* channels */
  int64_t m;               /* rows = N*H*W, at least 2 */
  float eps;               /* added to the variance inside the square root */
  float momentum;          /* running-statistics factor; used only when running_* != NULL */
  int64_t y_pixel_stride;  /* pixels of y (the BN input); 0 means c */
  int64_t a_pixel_stride;  /* pixels of out (forward) and g (backward); 0 means c */
  int64_t r_pixel_stride;  /* pixels of residual (forward) and residual_grad (backward); 0 means c */
  int64_t dy_pixel_stride; /* pixels of dy (backward); 0 means c */
} numbat_bn_problem;

/* NUMBAT_ABI_VERSION of the loaded library. */
uint32_t numbat_abi_version(void);

/* Detail text of the last failing call on this thread ("" after success). Owned by
 * the library; valid until the next call on the same thread. */
const char* numbat_last_error(void);

/* Short name of a status code; never NULL. */
const char* numbat_status_string(numbat_status status);

/* Output spatial size of a convolution problem.  Fails like the entry points on a
 * malformed descriptor. */
numbat_status numbat_conv_output_shape(const numbat_conv_problem* p, int32_t* ho, int32_t* wo);

/* Workspace bytes that entry point `op` needs for `problem` (a numbat_conv_problem* for
 * the three convolution ops, a numbat_bn_problem* for the two BN ops).  Depends only on
 * the problem, never on the device.  May be 0; then ws may be NULL.
 * Every non-empty workspace begins with a 256-byte header of counters that some kernels use
 * to coordinate their blocks: it must hold zeros when a workspace is first used (fill it
 * with zeros once after allocating it), and every call leaves it zero again.  One
 * workspace may serve any number of calls that run one after another; calls that may
 * overlap in time need workspaces of their own. */
numbat_status numbat_workspace_size(numbat_op op, const void* problem, size_t* bytes);

/* Forward convolution, the defining sum of a cross-correlation (Sec. 6.1 conv block):
 *   y[n,p,q,o] = sum_{r,s,c} w[o,r,s,c] * x[n, p*stride_h - pad_h + r, q*stride_w - pad_w + s, c]
 * with x = 0 outside the image.  x: bf16 NHWC (pixel stride x_pixel_stride); w: bf16 OHWI;
 * y: bf16 NHWC (pixel stride y_pixel_stride), fp32 accumulation rounded to nearest even.
 * batch_stats: NULL, or fp32 [2*c_out] receiving the batch mean (first c_out entries) and
 * biased batch variance (next c_out) of every output channel over the n*ho*wo rows, taken
 * from the fp32 accumulators before rounding (BN statistics in fp32, Sec. 3.2).
 * ws: numbat_workspace_size(NUMBAT_OP_CONV_FWD) bytes (per-tile statistics partials); it
 * may be NULL when batch_stats is NULL. */
numbat_status numbat_conv_fwd(const numbat_conv_problem* p, const void* x, const void* w, void* y,
                              float* batch_stats, void* ws, size_t ws_bytes, void* stream);

/* Prologue-fused forward: the previous layer's BN + SiLU applied inside this convolution's
 * operand staging (Sec. 3.1: fused element-wise work around the kernels of a block chain),
 *   y = conv(SiLU(BN(y_prev)), w),  BN(v)[c] = gamma[c] (v - mean[c]) / sqrt(var[c] + eps) + beta[c],
 * with the previous layer's batch statistics prev_stats ([mean][variance], c_in entries
 * each, as numbat_conv_fwd's batch_stats), so its activation is never written to memory.
 * y_prev: bf16 NHWC [n,h,w,c_in] (x_pixel_stride); gamma, beta: fp32 [c_in]; w, y,
 * batch_stats, ws as numbat_conv_fwd (ws sized by numbat_workspace_size(NUMBAT_OP_CONV_FWD)).
 * The activations are formed with the same fp32 arithmetic and rounding as
 * numbat_bn_silu_fwd, so y and batch_stats equal numbat_bn_silu_fwd (no residual) followed
 * by numbat_conv_fwd bit for bit wherever that forward runs the same kernel (3x3 problems
 * whose grid has at least 256 tiles).  Supported: 3x3, stride 1, pad 1, c_in a multiple of
 * 16 in 32 .. 1024, images the 3x3 stride-1 kernel takes (up to 95 wide, or a multiple of
 * 32 wide and 8 high); otherwise NUMBAT_ERR_UNSUPPORTED before any launch. */
numbat_status numbat_conv_fwd_bn_silu_prologue(const numbat_conv_problem* p, const void* y_prev,
                                               const float* prev_stats, const float* gamma, const float* beta,
                                               float eps, const void* w, void* y, float* batch_stats, void* ws,
                                               size_t ws_bytes, void* stream);

/* Forward convolution plus a per-channel bias, y = conv(x, w) + bias[o]: the detect head's
 * 1x1 prediction convolutions, which carry a bias and no BN (Sec. 6.1 decoupled head).  Same
 * layouts and checks as numbat_conv_fwd; bias: fp32 [c_out]; no statistics, no workspace. */
numbat_status numbat_conv_fwd_bias(const numbat_conv_problem* p, const void* x, const void* w, const float* bias,
                                   void* y, void* stream);

/* Inference-mode Conv -> BN -> SiLU in one pass: BN with running statistics (evaluation
 * mode, Table 2 #9), folded into the convolution's output stage:
 *   y = SiLU(gamma * (conv(x, w) - running_mean) / sqrt(running_var + eps) + beta)
 * computed from the fp32 accumulators, rounded once to bf16.  Same layouts and checks as
 * numbat_conv_fwd; gamma, beta, running_mean, running_var: fp32 [c_out]; no workspace. */
numbat_status numbat_conv_bn_silu_infer(const numbat_conv_problem* p, const void* x, const void* w,
                                        const float* gamma, const float* beta, const float* running_mean,
                                        const float* running_var, float eps, void* y, void* stream);

/* numbat_conv_fwd without a workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).
 * Same arguments, results and checks as numbat_conv_fwd; the per-tile statistics partials
 * go to a static scratch array of 8 MiB that the library holds on every GPU it runs on
 * until the process ends (the same kernels run, so results equal numbat_conv_fwd's bit
 * for bit).  Calls no allocating routine.  A problem whose partials exceed 8 MiB returns
 * NUMBAT_ERR_WORKSPACE before any launch (the detector's layers need at most 4.7 MiB at
 * batch 32).  Uses the scratch of the current device; the stream must belong to it.  All
 * calls on one GPU share that scratch: calls that may overlap in time on one GPU (several
 * streams, several host threads) race and must be ordered by the caller. */
numbat_status numbat_conv_fwd_noalloc(const numbat_conv_problem* p, const void* x, const void* w, void* y,
                                      float* batch_stats, void* stream);

/* Data gradient of the forward convolution (its adjoint in x): the backward of the
 * detector's conv block (Sec. 6.1), whose training step runs a backward stage over every
 * layer (Sec. 8.2 stage timings); the operator-level check of Sec. 6.3 compares this
 * operator's CPU and GPU backward.  The sum is the transpose of the forward's:
 *   dx[n,h,w,c] = sum over (p,q,r,s,o) with p*stride_h - pad_h + r = h and
 *                 q*stride_w - pad_w + s = w of  w[o,r,s,c] * dy[n,p,q,o].
 * dy: bf16 NHWC [n,ho,wo,c_out] (y_pixel_stride); dx: bf16 NHWC [n,h,w,c_in] (x_pixel_stride).
 * accumulate != 0: dx += result (sum formed in fp32, rounded once), else dx = result.
 * ws: numbat_workspace_size(NUMBAT_OP_CONV_BWD_DATA) bytes: the weights re-laid out per
 * stride phase when the problem is not one the direct-to-LDS kernel reads them in place
 * for (c_out not a multiple of 16 or below 32, or offsets beyond 31 bits), fp32 weights
 * for c_in < 8; otherwise unused.  It may not be NULL. */
numbat_status numbat_conv_bwd_data(const numbat_conv_problem* p, const void* dy, const void* w, void* dx,
                                   int accumulate, void* ws, size_t ws_bytes, void* stream);

/* The data gradient with this layer's BN + SiLU backward applied inside its operand
 * staging: the backward half of fusing the element-wise work around a kernel into it
 * (Sec. 3.1, the fusion templates' pre/post element-wise stages).  For a 3x3 stride-1 pad-1
 * convolution whose output y went through numbat_bn_silu_fwd, given g = dL/d(out) and the
 * dgamma, dbeta that numbat_bn_silu_bwd formed (it may be called with dy = NULL for that):
 *   dy = gamma * save_rstd * (dz - dbeta / m - xhat * dgamma / m)   (numbat_bn_silu_bwd's dy)
 *   dx = the data gradient of dy                                       (numbat_conv_bwd_data's)
 * with m = n * ho * wo.  dy is formed once per element from g and y as the kernel stages
 * its input halo and is also written out (bf16), for the weight gradient; dx and dy equal
 * numbat_bn_silu_bwd followed by numbat_conv_bwd_data bit for bit.
 * g: bf16 [n,ho,wo,c_out] with g_pixel_stride (0 means c_out); y and dy: bf16 with the
 * problem's y_pixel_stride; dx: bf16 with x_pixel_stride, accumulate as numbat_conv_bwd_data;
 * save_mean, save_rstd, gamma, beta, dgamma, dbeta: fp32 [c_out].  g, y, dy, dx 16-byte
 * aligned with pixel strides multiples of 8.  No workspace.  Returns NUMBAT_ERR_UNSUPPORTED
 * unless the problem is 3x3, stride 1, padding 1, c_out a multiple of 16 in 32 .. 1024,
 * c_in a multiple of 8, on an image the halo kernel takes (numbat_workspace_size with
 * NUMBAT_OP_CONV_BWD_DATA_BN_SILU answers that without a launch). */
numbat_status numbat_conv_bwd_data_bn_silu_prologue(const numbat_conv_problem* p, const void* g,
                                                    int64_t g_pixel_stride, const void* y, const float* save_mean,
                                                    const float* save_rstd, const float* gamma, const float* beta,
                                                    const float* dgamma, const float* dbeta, const void* w, void* dx,
                                                    void* dy, int accumulate, void* stream);

/* Weight gradient of the forward convolution (its adjoint in w), fp32 (gradients of the
 * fp32 master weights, Table 1 precision row):
 *   dw[o,r,s,c] = sum_{n,p,q} dy[n,p,q,o] * x[n, p*stride_h - pad_h + r, q*stride_w - pad_w + s, c].
 * accumulate != 0: dw += result, else dw = result.  The sum over n*ho*wo rows is split into
 * fixed ranges reduced in a fixed order, so the result is bitwise reproducible.
 * ws: numbat_workspace_size(NUMBAT_OP_CONV_BWD_WEIGHT) bytes (split partials; for c_in < 8
 * also the input repacked to 8 channels, except for the RGB image layer's shape -- 3
 * channels, 3x3, stride 2, padding 1, c_out <= 64 and a multiple of 8, output rows a
 * multiple of 4 and columns of 64 -- whose kernel needs only its per-block partials). */
numbat_status numbat_conv_bwd_weight(const numbat_conv_problem* p, const void* x, const void* dy, float* dw,
                                     int accumulate, void* ws, size_t ws_bytes, void* stream);

/* Batch normalisation (training mode) + SiLU, forward (BN after Ioffe and Szegedy in fp32,
 * Sec. 3.2; SiLU, Sec. 6.1):
 *   mean, var  = batch_stats if given, else the batch mean and biased variance of the bf16 y
 *   rstd       = 1 / sqrt(var + eps)
 *   out        = SiLU(gamma * (y - mean) * rstd + beta) [+ residual]      (bf16, RNE)
 * y, residual, out: bf16 [m rows][c] with their pixel strides; residual may be NULL.
 * gamma, beta: fp32 [c].  save_mean, save_rstd: fp32 [c] outputs, required (the backward
 * reads them).  running_mean/running_var: both NULL, or fp32 [c] updated in place as
 * running = (1 - momentum) * running + momentum * batch (variance term unbiased, * m/(m-1)). */
numbat_status numbat_bn_silu_fwd(const numbat_bn_problem* p, const void* y, const float* batch_stats,
                                 const float* gamma, const float* beta, const void* residual, void* out,
                                 float* save_mean, float* save_rstd, float* running_mean, float* running_var,
                                 void* ws, size_t ws_bytes, void* stream);

/* BN (evaluation mode, running statistics; Table 2 #9) + SiLU on a stored conv output:
 *   out = SiLU(gamma * (y - running_mean) / sqrt(running_var + eps) + beta) [+ residual]
 * with eps = p->eps (p->momentum unused); layouts and pixel strides as numbat_bn_silu_fwd;
 * nothing is saved or updated; no workspace. */
numbat_status numbat_bn_silu_infer(const numbat_bn_problem* p, const void* y, const float* running_mean,
                                   const float* running_var, const float* gamma, const float* beta,
                                   const void* residual, void* out, void* stream);

/* Backward of numbat_bn_silu_fwd with batch statistics, given g = dL/d(out): BN is trained
 * in fp32 under mixed precision (Sec. 3.2, Table 1 precision row) with batch statistics in
 * the training step, so its gradient flows through the statistics; SiLU is the detector's
 * activation (Sec. 6.1).  The chain rule through those definitions gives:
 *   z = gamma * xhat + beta,  xhat = (y - save_mean) * save_rstd
 *   dz = g * sigmoid(z) * (1 + z * (1 - sigmoid(z)))
 *   dbeta = sum_rows dz,  dgamma = sum_rows dz * xhat                      (fp32 [c])
 *   dy = gamma * save_rstd * (dz - dbeta / m - xhat * dgamma / m)            (bf16, RNE)
 * residual_grad: NULL, or bf16 [m][c] (r_pixel_stride) that receives += g, the gradient of
 * a residual added in the forward.  g, y, dy: bf16 with their pixel strides.  dy NULL: only
 * dgamma and dbeta are formed (for numbat_conv_bwd_data_bn_silu_prologue, which forms dy
 * itself); residual_grad must then be NULL. */
numbat_status numbat_bn_silu_bwd(const numbat_bn_problem* p, const void* g, const void* y,
                                 const float* save_mean, const float* save_rstd, const float* gamma,
                                 const float* beta, void* dy, float* dgamma, float* dbeta, void* residual_grad,
                                 void* ws, size_t ws_bytes, void* stream);

/* One fp32 parameter tensor of the optimiser step: its values, gradient and momentum
 * buffer (device pointers, n elements each) and its parameter group. */
typedef struct {
  float* w;           /* parameters, updated in place */
  const float* grad;  /* gradient of the loss */
  float* momentum;    /* momentum buffer, updated in place; zeros before the first step */
  int64_t n;          /* elements */
  int32_t group;      /* parameter group, 0 .. ngroups-1 (a tensor outside them is left unchanged) */
  int32_t reserved;   /* 0 */
} numbat_param_tensor;

/* Learning rate and weight decay of one parameter group. */
typedef struct {
  float lr;
  float weight_decay;
} numbat_sgd_group;

/* The optimiser step after the weight gradients (Sec. 3.2 optimisation; Table 1 optimisation
 * row): global-norm gradient clipping as one squared-norm accumulation over every gradient
 * (Table 2 #7: clip at 10.0 every step), then SGD with Nesterov momentum in parameter groups
 * (three in the case study: decayed weights, undecayed normalisation gains, undecayed biases),
 * with the reference-default semantics:
 *   total = sqrt(sum over every tensor and element of grad^2)
 *   c     = min(1, max_norm / (total + 1e-6))
 *   d     = c * grad + weight_decay[group] * w
 *   momentum = momentum_factor * momentum + d            (no dampening)
 *   w     = w - lr[group] * (d + momentum_factor * momentum)
 * tensors: DEVICE array of `count` numbat_param_tensor (1 .. 1024), read by the kernels (the
 * caller keeps it for the life of the call); all pointers in it are device pointers, 16-byte
 * aligned ones take the vector path.  groups: HOST array of ngroups (1 .. 8) entries.
 * total_norm: NULL, or a device float receiving `total`.  No host synchronisation: the norm
 * stays on the device.  The sum is taken in fp64 in a fixed order, so results are bitwise
 * reproducible.  ws: numbat_workspace_size(NUMBAT_OP_CLIP_SGD_NESTEROV) bytes (8 KiB). */
numbat_status numbat_clip_sgd_nesterov(const numbat_param_tensor* tensors, int32_t count,
                                       const numbat_sgd_group* groups, int32_t ngroups, float momentum_factor,
                                       float max_norm, float* total_norm, void* ws, size_t ws_bytes, void* stream);

/* A pooled or upsampled NHWC bf16 tensor: n images of h x w pixels, c channels (a multiple
 * of 8).  For the max pool x / dx and y / dy are all n x h x w; for the upsampling x / dx
 * are n x h x w and y / dy are n x 2h x 2w.  Pixel strides as in the other descriptors
 * (0 means c), so operands can be channel slices of concatenation buffers. */
typedef struct {
  uint32_t struct_size;    /* = sizeof(numbat_pool_problem) */
  int32_t n, h, w, c;
  int64_t x_pixel_stride;  /* pixels of x and dx */
  int64_t y_pixel_stride;  /* pixels of y and dy */
} numbat_pool_problem;

/* The SPPF block's max pool (Sec. 6.1 backbone; applied three times in a row): 5 x 5 window,
 * stride 1, padding 2 that never wins:
 *   y[n,p,q,c] = max over in-image (i, j) with |i - p| <= 2, |j - q| <= 2 of x[n,i,j,c]
 * idx: NULL, or uint8 [n][h][w][c] (dense, 8-byte aligned) receiving the row-major window
 * position r * 5 + s (0 .. 24) of each window's FIRST maximum (a later equal value does not
 * replace it), the position the backward sends the gradient to. */
numbat_status numbat_maxpool5_fwd(const numbat_pool_problem* p, const void* x, void* y, uint8_t* idx, void* stream);

/* Backward of numbat_maxpool5_fwd: dx[n,i,j,c] = sum of dy over the windows whose stored
 * first-maximum position is (i, j) (summed in fp32 in a fixed order, rounded once);
 * accumulate != 0: dx += that sum. */
numbat_status numbat_maxpool5_bwd(const numbat_pool_problem* p, const void* dy, const uint8_t* idx, void* dx,
                                  int accumulate, void* stream);

/* The neck's nearest-neighbour 2x upsampling (Sec. 6.1 PAN-FPN neck):
 *   y[n, 2i + a, 2j + b, c] = x[n, i, j, c]   for a, b in {0, 1}. */
numbat_status numbat_upsample2x_fwd(const numbat_pool_problem* p, const void* x, void* y, void* stream);

/* Backward: dx[n,i,j,c] = sum over a, b of dy[n, 2i + a, 2j + b, c] (fp32, rounded once);
 * accumulate != 0: dx += that sum. */
numbat_status numbat_upsample2x_bwd(const numbat_pool_problem* p, const void* dy, void* dx, int accumulate,
                                    void* stream);

/* Launch timing, for measurement (the paper times its training step phase by phase,
 * Sec. 8): while enabled, every kernel the library launches is bracketed by two HIP
 * events recorded on its launch stream, and numbat_timing_read sums their elapsed times
 * per kernel class.  numbat_timing_enable(1) starts a new record set, (0) stops and
 * clears it.  Not for use while a stream is being captured into a graph.  Events are
 * host-side handles created by the library on first use and reused; no device memory is
 * allocated.  Kernel classes are numbered 0 .. numbat_kernel_class_count() - 1;
 * numbat_kernel_class_name gives a short name ("" for an unknown class). */
int numbat_kernel_class_count(void);
const char* numbat_kernel_class_name(int kernel_class);
numbat_status numbat_timing_enable(int enable);
/* Waits for the recorded events of `kernel_class`, then writes their summed duration (ms)
 * and the number of launches.  NUMBAT_ERR_BAD_DESC for an unknown class. */
numbat_status numbat_timing_read(int kernel_class, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* NUMBAT_CONV_H */
