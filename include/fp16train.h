/*
 * fp16train: the all-FP16 training hot path of arXiv:1911.07384,
 * "Distributed low-precision Training Without Mixed Precision", for AMD
 * MI355X (gfx950).
 *
 * Every tensor that crosses this interface is IEEE binary16 (Section 5.2:
 * activations, weights and gradients are all stored in FP16 and no master
 * copy is kept in higher precision).  Inside a kernel, products are formed
 * exactly and accumulated in float32 (matrix cores) and every result is
 * rounded once to binary16, to nearest with ties to even, at its store
 * (Section 4.2 leaves the rounding method open; this library uses the IEEE
 * default).  Binary16 subnormals are kept (gradual underflow) and overflow
 * rounds to +-infinity.
 *
 * Conventions shared by every entry point:
 *   - Buffers are device pointers owned by the caller.  The library never
 *     allocates or frees device memory and keeps no state between calls.
 *     Any scratch memory a call needs is the caller's workspace, sized by
 *     the matching *_workspace_bytes query -- except fp16_conv_wgrad_noalloc,
 *     whose scratch is a fixed device array of the library (see there).
 *   - Work is enqueued on `stream` (a hipStream_t; NULL is the default
 *     stream) and the call returns without waiting for it.
 *   - Arguments are checked before anything is enqueued: a nonzero status
 *     means nothing was launched.  FP16_ERR_HIP reports a failed launch.
 *     Faults inside kernels surface at the caller's next synchronisation.
 *   - Activation, filter, workspace and parameter pointers must be 16-byte
 *     aligned (FP16_ERR_MISALIGNED otherwise).
 *   - Results are deterministic: the same inputs give the same bits on
 *     every run (no floating-point atomics).
 *   - Layout FP16_NHWC: activations [N][H][W][C], filters [K][R][S][C].
 *     Layout FP16_NCHW: activations [N][C][H][W], filters [K][C][R][S].
 *     NHWC is the native layout; NCHW calls convert through the workspace.
 */
#ifndef FP16TRAIN_H
#define FP16TRAIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t fp16_t;      /* IEEE binary16 bit pattern */
typedef void* fp16_stream_t;  /* hipStream_t */

typedef enum {
  FP16_OK = 0,
  FP16_ERR_NULL = 1,        /* a required pointer is NULL */
  FP16_ERR_SHAPE = 2,       /* a dimension is out of range or inconsistent */
  FP16_ERR_LAYOUT = 3,      /* unknown layout value */
  FP16_ERR_MISALIGNED = 4,  /* a pointer is not 16-byte aligned */
  FP16_ERR_ALIASING = 5,    /* an output overlaps an input it must not */
  FP16_ERR_WORKSPACE = 6,   /* workspace missing or smaller than required */
  FP16_ERR_UNSUPPORTED = 7, /* valid request outside what is implemented */
  FP16_ERR_HIP = 8          /* the HIP runtime reported an error */
} fp16_status;

typedef enum { FP16_NHWC = 0, FP16_NCHW = 1 } fp16_layout;

typedef enum { FP16_PASS_FWD = 0, FP16_PASS_DGRAD = 1, FP16_PASS_WGRAD = 2 } fp16_conv_pass;

/* Convolution problem: input x [N,C,H,W] (logical), filter W [K,C,R,S],
 * output y [N,K,P,Q] with P = (H + 2*pad_h - R)/stride_h + 1 and
 * Q = (W + 2*pad_w - S)/stride_w + 1.  Cross-correlation, zero padding,
 * no dilation, one group.  All dimensions >= 1, pads >= 0, P, Q >= 1. */
typedef struct {
  int32_t n, c, h, w;
  int32_t k, r, s;
  int32_t stride_h, stride_w;
  int32_t pad_h, pad_w;
  int32_t layout; /* fp16_layout */
  int32_t accum;  /* 0: float32 accumulators (default);
                     1: every operation in binary16 -- the strict reading of "all
                        arithmetic in FP16" (Section 5.2), to measure what float32
                        accumulators buy: each output is a binary16 accumulator that
                        starts at +0 and takes its terms one at a time as binary16 fused
                        multiply-adds (one rounding of the exact a*b + acc per term).
                        Reduction orders: forward, taps (r, s) row-major and channels c
                        ascending within a tap; data gradient, the taps (r, s) row-major
                        that reach the position from a point of the P x Q grid, output
                        channels k ascending within a tap; weight gradient, the output
                        pixels (n, p, q) in order.  Taps outside the image (or the grid)
                        are not terms.  NHWC only, plain fwd / dgrad / wgrad only
                        (FP16_ERR_UNSUPPORTED for NCHW, fp16_conv_dgrad_add,
                        fp16_conv_dgrad_wf and fp16_conv_bn_relu_fwd); needs no
                        workspace; runs on the vector ALUs, far slower than the default. */
} fp16_conv_desc;

/* Batch normalisation problem on x [N,C,H,W] (logical). */
typedef struct {
  int32_t n, c, h, w;
  int32_t layout;     /* fp16_layout */
  float eps;          /* added to the variance, held in float32 */
  float post_scale;   /* output multiplier s: 0.25 inside residual blocks, 1 for the stem */
  int32_t relu;       /* 1: apply ReLU to the output; 0: no ReLU */
  int32_t use_stats;  /* 0: compute batch statistics from x and write them to `stats`;
                         1: read mean and rstd from `stats` and only apply */
  int32_t swap;       /* 0: y = relu(s*(gamma*xhat + beta) + r);
                         1: the BN swap of Section 4.1, the shortcut joining before gamma:
                            y = relu(s*(gamma*(xhat + r) + beta)); needs the residual */
} fp16_bn_desc;

/* Output spatial size of a convolution; FP16_ERR_SHAPE if it is empty. */
fp16_status fp16_conv_out_dims(const fp16_conv_desc* desc, int32_t* p, int32_t* q);

/* Bytes of workspace a convolution pass needs (0 when it needs none).
 * Returns 0 for an invalid descriptor as well; the pass call reports it. */
size_t fp16_conv_workspace_bytes(const fp16_conv_desc* desc, int32_t pass);

/* Forward convolution (ResNet-50's convolutions, Section 5.1):
 *   y[n,k,p,q] = sum_{c,r,s} x[n,c, p*stride_h - pad_h + r, q*stride_w - pad_w + s] * W[k,c,r,s]
 * with out-of-image taps reading zero.  Accumulation in float32, one
 * rounding to binary16 per output.  y must not overlap x, w or ws. */
fp16_status fp16_conv_fwd(const fp16_conv_desc* desc, const fp16_t* x, const fp16_t* w, fp16_t* y,
                          void* ws, size_t ws_bytes, fp16_stream_t stream);

/* Data gradient: the gradient with respect to the input of ResNet-50's
 * convolutions (Section 5.1), stored in binary16 like every gradient of the
 * method (Section 5.2); the adjoint of fp16_conv_fwd in x:
 *   dx[n,c,h,w] = sum over (k,r,s) with h + pad_h - r = p*stride_h and
 *                 w + pad_w - s = q*stride_w, (p,q) inside the P x Q grid, of dy[n,k,p,q] * W[k,c,r,s].
 * Every element of dx is written (positions no tap reaches get zero).
 * dx must not overlap dy, w or ws. */
fp16_status fp16_conv_dgrad(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* w,
                            fp16_t* dx, void* ws, size_t ws_bytes, fp16_stream_t stream);

/* Data gradient plus an addend, rounded once:
 *   dx = round_to_binary16(dgrad(dy, W) + addend)
 * with the float32 sum of fp16_conv_dgrad and the binary16 addend added in
 * float32 before the single rounding.  This is the input gradient of a
 * residual block (Section 4.1: the identity shortcut carries its own
 * gradient, which joins the branch gradient at the block input).  addend
 * has dx's shape and layout and may equal dx (accumulate in place); it must
 * not overlap dx otherwise.  dx must not overlap dy, w or ws. */
fp16_status fp16_conv_dgrad_add(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* w,
                                const fp16_t* addend, fp16_t* dx, void* ws, size_t ws_bytes,
                                fp16_stream_t stream);

/* The data gradient in two steps, so that the filter rearrangement (which
 * depends only on W) can run ahead of time, off the critical path, e.g. on
 * a second stream during the forward pass:
 *   fp16_conv_dgrad_filter writes W rearranged for the data gradient into wf
 *   (per stride phase, its taps flipped, rows = input channels, reduction
 *   over (tap, output channel) with the output channels padded to a multiple
 *   of 8; fp16_conv_dgrad_filter_bytes bytes, 16-byte aligned, not
 *   overlapping w);
 *   fp16_conv_dgrad_wf computes fp16_conv_dgrad (addend NULL) or
 *   fp16_conv_dgrad_add (addend given, same rules) from wf instead of w,
 *   with identical results.
 * NHWC only (FP16_ERR_UNSUPPORTED for NCHW).  The workspace is the one
 * fp16_conv_workspace_bytes(desc, FP16_PASS_DGRAD) sizes.  wf must hold the
 * rearrangement of the filter the data gradient is meant for: it is not
 * checked. */
size_t fp16_conv_dgrad_filter_bytes(const fp16_conv_desc* desc);
fp16_status fp16_conv_dgrad_filter(const fp16_conv_desc* desc, const fp16_t* w, fp16_t* wf,
                                   fp16_stream_t stream);
fp16_status fp16_conv_dgrad_wf(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* wf,
                               const fp16_t* addend, fp16_t* dx, void* ws, size_t ws_bytes,
                               fp16_stream_t stream);
/* fp16_conv_dgrad_wf with the addend taken under a ReLU mask:
 *   dx = round_to_binary16(dgrad(dy, W) + (mask ? addend : +0))
 * where the mask bit of element (n, h, w, c) is bit c % 8 of byte
 * ((n*H + h)*W + w)*(C/8) + c/8 of addend_mask (the layout fp16_bn_relu_m
 * keeps, x_elems/8 bytes).  With the addend the gradient a block-last BN
 * received and the mask its forward kept, this is the block input gradient
 * of Section 4.1 (branch gradient + the identity shortcut's gradient, which
 * is the BN's incoming gradient through its ReLU) without that BN's backward
 * writing the shortcut gradient out.  Bit-identical to fp16_conv_dgrad_wf on
 * the masked addend.  NHWC with C % 8 == 0 only (FP16_ERR_UNSUPPORTED
 * otherwise); addend and addend_mask non-null (FP16_ERR_NULL); the mask must
 * not overlap dx or ws (FP16_ERR_ALIASING); other rules as
 * fp16_conv_dgrad_wf. */
fp16_status fp16_conv_dgrad_wf_m(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* wf,
                                 const fp16_t* addend, const uint8_t* addend_mask, fp16_t* dx,
                                 void* ws, size_t ws_bytes, fp16_stream_t stream);
/* fp16_conv_dgrad_wf with the addend's optional parts spelled out:
 *   dx = round_to_binary16(dgrad(dy, W) + a),   a = +0 where addend is NULL;
 * with addend_stride s > 1 the addend holds only the pixels whose row and
 * column are multiples of s, laid out NHWC as [N][ceil(H/s)][ceil(W/s)][C]
 * (every other pixel takes a = +0): the gradient a strided 1x1 shortcut
 * (Section 5.1's downsampling blocks) sends to the block input, computed on
 * its own grid instead of written out with three zeros in four; with
 * addend_mask (over the addend's own layout, as in fp16_conv_dgrad_wf_m) a =
 * +0 where the bit is clear.  s = 1 and no mask is fp16_conv_dgrad_wf.
 * 1 <= addend_stride <= 16 (FP16_ERR_SHAPE); a stride or a mask needs the
 * addend (FP16_ERR_NULL) and NHWC (FP16_ERR_UNSUPPORTED), a mask C % 8 == 0;
 * a strided addend may not be dx or overlap it (FP16_ERR_ALIASING). */
fp16_status fp16_conv_dgrad_wf_ex(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* wf,
                                  const fp16_t* addend, const uint8_t* addend_mask,
                                  int32_t addend_stride, fp16_t* dx, void* ws, size_t ws_bytes,
                                  fp16_stream_t stream);
/* fp16_conv_dgrad_filter for `count` convolutions at once (descs[i], w[i],
 * wf[i]; host arrays, read during the call only): every filter of a network
 * rearranged by one launch (or a few) instead of one launch each, with
 * identical results.  0 <= count <= FP16_DGRAD_FILTERS_MAX (else
 * FP16_ERR_SHAPE); every item is validated as fp16_conv_dgrad_filter does
 * before anything is launched, and no wf[i] may overlap any w[j] or another
 * wf[j] (FP16_ERR_ALIASING). */
#define FP16_DGRAD_FILTERS_MAX 1024
fp16_status fp16_conv_dgrad_filters(int32_t count, const fp16_conv_desc* descs,
                                    const fp16_t* const* w, fp16_t* const* wf,
                                    fp16_stream_t stream);

/* Weight gradient: the gradient with respect to the filter that the
 * momentum-SGD update of Section 5.1 consumes, stored in binary16 with no
 * higher-precision copy (Section 5.2); the adjoint of fp16_conv_fwd in W:
 *   dW[k,c,r,s] = sum_{n,p,q} dy[n,k,p,q] * x[n,c, p*stride_h - pad_h + r, q*stride_w - pad_w + s].
 * Partial sums over pixel ranges stay float32 in the workspace and are
 * added in a fixed order before the single rounding.  dw must not overlap
 * x, dy or ws. */
fp16_status fp16_conv_wgrad(const fp16_conv_desc* desc, const fp16_t* x, const fp16_t* dy,
                            fp16_t* dw, void* ws, size_t ws_bytes, fp16_stream_t stream);
/* fp16_conv_wgrad split over fewer pixel ranges, for a weight gradient that
 * runs beside other work on the device (the data-parallel backward of
 * Section 5.1 overlaps the weight gradients with the data gradients and BN
 * backwards on a second stream): the partial products aim at `workgroups`
 * workgroups in all, 1 <= workgroups <= 512, instead of the default 512 (two
 * per compute unit); 0 is the default, identical to fp16_conv_wgrad.  Fewer
 * ranges mean fewer float32 partial sums written and re-read and more of the
 * device left to the other stream; the partial sums are added in a fixed
 * order as always, so results are deterministic for a given count (and
 * differ from the default's only by float32 summation order).  The workspace
 * fp16_conv_workspace_bytes(desc, FP16_PASS_WGRAD) reports suffices for
 * every count.  FP16_ERR_SHAPE for a count outside [0, 512]; other errors as
 * fp16_conv_wgrad. */
fp16_status fp16_conv_wgrad_ex(const fp16_conv_desc* desc, const fp16_t* x, const fp16_t* dy,
                               fp16_t* dw, void* ws, size_t ws_bytes, int32_t workgroups,
                               fp16_stream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * weight gradient of fp16_conv_wgrad, bit-identical to it, with no workspace
 * argument.  Its scratch (the float32 split-K partial sums, and for the
 * ResNet stem the space-to-depth image) lives in a library-owned device
 * array of fp16_noalloc_scratch_bytes() = 32 MiB on each GPU the library
 * runs on, held from its first use on that GPU until the process ends; the
 * call itself allocates nothing.  A problem whose fp16_conv_workspace_bytes
 * (desc, FP16_PASS_WGRAD) exceeds that size returns FP16_ERR_WORKSPACE (every
 * ResNet-50 layer at batch 128 fits except the stem).  The work goes on
 * `stream`'s device (the current device for the NULL stream).  Calls that
 * overlap in time on one GPU share the array and race: order them on one
 * stream or synchronise between them.  Other arguments and errors as for
 * fp16_conv_wgrad. */
size_t fp16_noalloc_scratch_bytes(void);
fp16_status fp16_conv_wgrad_noalloc(const fp16_conv_desc* desc, const fp16_t* x, const fp16_t* dy,
                                    fp16_t* dw, fp16_stream_t stream);

/* Bytes of workspace the BN forward or backward call needs. */
size_t fp16_bn_workspace_bytes(const fp16_bn_desc* desc);

/* BN forward fused with the output multiplier, the identity shortcut and
 * ReLU (Eq. 1-2 of Section 4.1; the 0.25 multiplier after each BN inside a
 * residual block and the unchanged stem BN of Section 4.2; statistics over
 * this GPU's batch only, Section 5.1):
 *   mean_c, var_c over the M = N*H*W elements of channel c (biased variance);
 *   rstd_c = 1 / sqrt(var_c + eps);
 *   y = relu( s * (gamma_c * (x - mean_c) * rstd_c + beta_c) + r ).
 * With use_stats = 0, mean and rstd (float32) are computed in this call and
 * written to stats[0..C) and stats[C..2C).  With use_stats = 1 they are read
 * from stats.  The apply step is the float32 sequence
 *   a = fl(fl(s*gamma)*rstd); b = fl(s*beta); t = fl(x - mean);
 *   v = fma(t, a, b); v = fl(v + r); y = round_to_binary16(relu(v)),
 * so given statistics determine y bit for bit.  residual may be NULL.
 * y may equal x (in place); y must not overlap gamma, beta, stats or ws. */
fp16_status fp16_bn_relu(const fp16_bn_desc* desc, const fp16_t* x, const fp16_t* gamma,
                         const fp16_t* beta, const fp16_t* residual, fp16_t* y, float* stats,
                         void* ws, size_t ws_bytes, fp16_stream_t stream);

/* With desc->swap = 1 (BN swap) the apply step is instead
 *   sg = fl(s*gamma); a = fl(sg*rstd); b = fl(s*beta); t = fl(x - mean);
 *   w = fma(sg, r, b); v = fma(t, a, w); y = round_to_binary16(relu(v)),
 * and residual must not be NULL (FP16_ERR_NULL). */

/* BN backward through the same fused forward (not one of the paper's named
 * operations, but what training through Eq. 1-2 requires):
 *   mask = [y > 0] (all ones without ReLU);  g = s * dy * mask;
 *   S1_c = sum g;  S2_c = sum g * xhat,  xhat = (x - mean_c) * rstd_c;
 *   dbeta_c = S1_c;  dgamma_c = S2_c;
 *   dx = gamma_c * rstd_c * (g - S1_c/M - xhat * S2_c/M);
 *   dresidual = mask ? dy : 0  (the gradient reaching the identity shortcut).
 * With desc->swap = 1: dgamma_c = S2_c + S3_c with S3_c = sum g * r, dx as
 * above, and dresidual = round_to_binary16(gamma_c * g); residual must not
 * be NULL.
 * stats holds the forward's mean and rstd (float32, 2C values).  y is the
 * forward output; it may be NULL, in which case the mask is recomputed from
 * x, gamma, beta, residual and stats by the forward's float32 apply
 * sequence (bit-identical to what the forward stored).  dresidual may be
 * NULL.  dx may equal dy (in place). */
fp16_status fp16_bn_relu_bwd(const fp16_bn_desc* desc, const fp16_t* x, const fp16_t* y,
                             const fp16_t* dy, const fp16_t* gamma, const fp16_t* beta,
                             const fp16_t* residual, const float* stats, fp16_t* dx,
                             fp16_t* dgamma, fp16_t* dbeta, fp16_t* dresidual, void* ws,
                             size_t ws_bytes, fp16_stream_t stream);

/* ---- the ReLU mask kept from the forward for the backward ----
 * The backward of a BN whose output joins the shortcut before the ReLU (the
 * last BN of each residual block, Section 4.1's bottleneck) needs the ReLU
 * mask, [y > 0].  Recomputing it reads the shortcut again (2 bytes per
 * element); the forward can keep it instead, one bit per element, and the
 * backward read that (1/8 byte per element).  The mask is one byte per 8
 * channels of each pixel, for NHWC with C/8 a power of two up to 256 (C = 8,
 * 16, ..., 2048: every BN of ResNet-50 but the stem's) and ReLU on:
 *   mask[(n*H*W + h*W + w) * (C/8) + j] bit e = [y[n,h,w,8j+e] > 0].
 * fp16_bn_mask_bytes: its size, 0 where it is not offered (NCHW, other C, no
 * ReLU, the BN swap); the _m calls then return
 * FP16_ERR_UNSUPPORTED.  The mask is caller-owned, 16-byte aligned, and must
 * not overlap any other argument.
 * fp16_bn_relu_m / fp16_conv_bn_relu_fwd_m: fp16_bn_relu /
 *   fp16_conv_bn_relu_fwd (bit-identical outputs) that also write the mask of
 *   their BN output.
 * fp16_bn_relu_bwd_m: fp16_bn_relu_bwd with the mask read from `mask`
 *   instead of being taken from y or recomputed from the shortcut (which is
 *   not needed: dresidual = mask ? dy : 0); bit-identical outputs. */
size_t fp16_bn_mask_bytes(const fp16_bn_desc* desc);
fp16_status fp16_bn_relu_m(const fp16_bn_desc* desc, const fp16_t* x, const fp16_t* gamma,
                           const fp16_t* beta, const fp16_t* residual, fp16_t* y, float* stats,
                           uint8_t* mask, void* ws, size_t ws_bytes, fp16_stream_t stream);
fp16_status fp16_bn_relu_bwd_m(const fp16_bn_desc* desc, const fp16_t* x, const uint8_t* mask,
                               const fp16_t* dy, const fp16_t* gamma, const fp16_t* beta,
                               const float* stats, fp16_t* dx, fp16_t* dgamma, fp16_t* dbeta,
                               fp16_t* dresidual, void* ws, size_t ws_bytes,
                               fp16_stream_t stream);

/* Momentum SGD on FP16 weights and an FP16 momentum buffer, with no master
 * copy (Section 5.1 recipe: PyTorch SGD, dampening 0, no Nesterov;
 * Section 5.2), in place over n elements:
 *   d = fma(weight_decay, w, g);  m = round_to_binary16(fma(momentum, m, d));
 *   w = round_to_binary16(fma(-lr, m, w))
 * evaluated in float32 exactly as written, so results are unique bit
 * patterns.  BN parameters take weight_decay = 0 (Section 5.1).  g must not
 * overlap w or m; w and m must not overlap each other.  n = 0 is a no-op. */
fp16_status fp16_sgd_step(fp16_t* w, const fp16_t* g, fp16_t* m, size_t n, float lr,
                          float momentum, float weight_decay, fp16_stream_t stream);

/* The same update with every operation in binary16 arithmetic (the strict
 * reading of "all arithmetic in FP16", Section 5.2), for measuring what the
 * float32 sequence of fp16_sgd_step buys:
 *   d = fma16(wd, w, g);  m = fma16(mu, m, d);  w = fma16(nlr, m, w)
 * where fma16 rounds a*b + c once to binary16 (nearest even) and wd, mu and
 * nlr are the binary16 roundings of the float32 arguments weight_decay,
 * momentum and -lr.  Same aliasing rules and error behaviour as
 * fp16_sgd_step. */
fp16_status fp16_sgd_step_f16(fp16_t* w, const fp16_t* g, fp16_t* m, size_t n, float lr,
                              float momentum, float weight_decay, fp16_stream_t stream);

/* ---- a convolution fused with the statistics of the BN that follows ---- */

/* Workspace bytes of fp16_conv_bn_relu_fwd; 0 for invalid descriptors. */
size_t fp16_conv_bn_workspace_bytes(const fp16_conv_desc* conv, const fp16_bn_desc* bn);

/* Convolution forward followed by its BN (+ multiplier, shortcut, ReLU), the
 * BN statistics taken in the convolution's epilogue instead of a second pass
 * over y (a fusion of the network's conv -> BN pairs, ResNet-50, Section 5.1;
 * Eq. 1-2 of Section 4.1):
 *   y = fp16_conv_fwd(conv, x, w)              (bit-identical to that call)
 *   mean, rstd of y per channel                 (written to stats[0..2C))
 *   z = the BN apply of fp16_bn_relu on y with those statistics.
 * The epilogue keeps, per 128-row tile of y and channel, a shift K (the
 * tile's first value) and float32 sums of (y - K) and (y - K)^2 over its
 * rounded values; the tiles are combined in float64.  (Shapes whose
 * convolution kernel does not take the statistics -- the LDS-staged one,
 * used for channel counts that are not a multiple of 32 and for long
 * reductions over large outputs with fewer than 64-multiple channels -- run
 * the convolution and the BN's own statistics pass instead, with the same
 * results as the two separate calls.)  The statistics may differ from
 * fp16_bn_relu's in the last
 * bits (another summation grouping); z is bit-exact against the declared
 * apply with the statistics written.
 * Requires NHWC, conv->k a multiple of 8, a BN descriptor of y's shape
 * (n = n, c = k, h = p, w = q) with use_stats = 0 (FP16_ERR_UNSUPPORTED /
 * FP16_ERR_SHAPE otherwise).  z may equal y (then only the BN output
 * remains) or the residual; y must not overlap x, w, the residual or any
 * other argument. */
fp16_status fp16_conv_bn_relu_fwd(const fp16_conv_desc* conv, const fp16_bn_desc* bn,
                                  const fp16_t* x, const fp16_t* w, const fp16_t* gamma,
                                  const fp16_t* beta, const fp16_t* residual, fp16_t* y,
                                  fp16_t* z, float* stats, void* ws, size_t ws_bytes,
                                  fp16_stream_t stream);

/* The same with the ReLU mask of z kept (see fp16_bn_mask_bytes). */
fp16_status fp16_conv_bn_relu_fwd_m(const fp16_conv_desc* conv, const fp16_bn_desc* bn,
                                    const fp16_t* x, const fp16_t* w, const fp16_t* gamma,
                                    const fp16_t* beta, const fp16_t* residual, fp16_t* y,
                                    fp16_t* z, float* stats, uint8_t* mask, void* ws,
                                    size_t ws_bytes, fp16_stream_t stream);

/* ---- the rest of ResNet-50 around the residual blocks (Section 5.1) ---- */

/* Pooling problem on x [N,C,H,W] (logical) with an R x S window:
 * output [N,C,P,Q], P = (H + 2*pad_h - R)/stride_h + 1 (likewise Q).
 * Layouts as for activations above. */
typedef struct {
  int32_t n, c, h, w;
  int32_t r, s;
  int32_t stride_h, stride_w;
  int32_t pad_h, pad_w;
  int32_t layout; /* fp16_layout */
} fp16_pool_desc;

/* Output spatial size of a pooling window; FP16_ERR_SHAPE if invalid.
 * Valid: all sizes >= 1, 1 <= r, s <= 15, 1 <= strides <= 16,
 * 0 <= pad_h < r, 0 <= pad_w < s (every window meets the image). */
fp16_status fp16_pool_out_dims(const fp16_pool_desc* desc, int32_t* p, int32_t* q);

/* Max pooling (the 3x3 stride-2 pool after ResNet-50's stem).  Positions in
 * the padding are not candidates.  Each window is scanned in (r, s) order; a
 * later element replaces the running maximum only if it is strictly larger,
 * and the first NaN met is kept.  y[n,c,p,q] is the winning element (no
 * rounding), idx[n,c,p,q] its tap r*S + s (one byte per output, laid out
 * like y).  y and idx must not overlap x or each other; idx is 16-byte
 * aligned like every buffer. */
fp16_status fp16_maxpool_fwd(const fp16_pool_desc* desc, const fp16_t* x, fp16_t* y,
                             uint8_t* idx, fp16_stream_t stream);

/* Max-pooling backward from the forward's idx:
 *   dx[n,c,h,w] = sum of dy[n,c,p,q] over the outputs whose winning position
 *                 is (h, w), added in float64 (exact) and rounded once;
 *                 +0 where no output selects the position.
 * Every element of dx is written.  dx must not overlap dy or idx. */
fp16_status fp16_maxpool_bwd(const fp16_pool_desc* desc, const uint8_t* idx, const fp16_t* dy,
                             fp16_t* dx, fp16_stream_t stream);

/* BN + ReLU whose output only feeds a max pool (ResNet-50's stem BN, Section
 * 5.1, and the 3x3 stride-2 pool after it), in one pass that never writes the
 * BN output: y and idx are bit for bit those of
 *   fp16_bn_relu(bn, x, gamma, beta, NULL, z, stats, ws) then
 *   fp16_maxpool_fwd(pool, z, y, idx)
 * and stats is written (or read, with bn->use_stats) as fp16_bn_relu does.
 * The backward needs only x, stats and idx: fp16_bn_relu_bwd recomputes the
 * ReLU mask from x (y = NULL).  Taken: NHWC, bn->relu = 1, no BN swap, C a
 * multiple of 8 with C/8 a power of two <= 256, a 3x3 pool window
 * (FP16_ERR_UNSUPPORTED otherwise); the pool descriptor's n, c, h, w and
 * layout equal the BN's (FP16_ERR_SHAPE otherwise).  Workspace:
 * fp16_bn_workspace_bytes(bn).  y, idx and the workspace must not overlap x,
 * gamma, beta, stats or each other (FP16_ERR_ALIASING). */
fp16_status fp16_bn_relu_maxpool(const fp16_bn_desc* bn, const fp16_pool_desc* pool,
                                 const fp16_t* x, const fp16_t* gamma, const fp16_t* beta,
                                 float* stats, fp16_t* y, uint8_t* idx, void* ws, size_t ws_bytes,
                                 fp16_stream_t stream);

/* Global average pooling (before ResNet-50's classifier): the window must be
 * the whole image (r = h, s = w, pads 0; FP16_ERR_UNSUPPORTED otherwise).
 *   y[n,c] = (sum over the H x W grid of x[n,c,.,.]) / (H*W)
 * with the sum exact in float64, one float64 division and one rounding.
 * y is [N,C] in both layouts.  y must not overlap x. */
fp16_status fp16_avgpool_fwd(const fp16_pool_desc* desc, const fp16_t* x, fp16_t* y,
                             fp16_stream_t stream);

/* Its adjoint: dx[n,c,h,w] = round_to_binary16(dy[n,c] / (H*W)) (float64
 * division).  dy is [N,C]; dx has x's shape and layout and must not overlap dy. */
fp16_status fp16_avgpool_bwd(const fp16_pool_desc* desc, const fp16_t* dy, fp16_t* dx,
                             fp16_stream_t stream);

/* Classifier bias and softmax cross-entropy averaged over the batch.
 * z [N,K] is the classifier's product (a 1x1 convolution), bias [K],
 * labels [N] int32 in [0, K):
 *   l = round_to_binary16(z + bias)                       (the logits)
 *   loss[n] = log(sum_j exp(l_nj - m_n)) + (m_n - l_n,label),  m_n = max_j l_nj
 *   dz[n,j] = round_to_binary16((softmax(l_n)_j - [j == label_n]) / N)
 *   dbias[j] = round_to_binary16(sum_n dz[n,j])           (exact float64 sum)
 * computed in float64; loss (float32, N values) is per sample, its mean is
 * the batch loss; dz is the gradient of that mean with respect to z and the
 * logits (no loss scaling: entries near 1/(N*K) are binary16 subnormals and
 * are kept).  A label outside [0, K) gives a NaN loss for its row and no
 * one-hot term.  dz may equal z; otherwise no output overlaps an input or
 * another output.  1 <= K <= 65535. */
fp16_status fp16_softmax_ce(int32_t n, int32_t k, const fp16_t* z, const fp16_t* bias,
                            const int32_t* labels, float* loss, fp16_t* dz, fp16_t* dbias,
                            fp16_stream_t stream);

/* Human-readable name of a status code (static string). */
const char* fp16_status_string(fp16_status status);

/* Library version, e.g. "fp16train 0.1". */
const char* fp16_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FP16TRAIN_H */
