/*
 * cosmoflow.h -- C ABI of the MI355X (gfx950) CosmoFlow convolution hot path.
 *
 * The operations are those of the CosmoFlow network (arXiv:1808.04728):
 * 3D convolution forward, backward-data and backward-weights (Section III-C,
 * Algorithm 1 and the paragraphs after it), bias + leaky ReLU (Section III-A:
 * every convolution layer uses leaky ReLU), and 3D average pooling with
 * stride (2,2,2) (Section III-A; Section III-C treats it as a per-channel
 * convolution with constant weights 1/KS^3).
 *
 * Conventions shared by every entry point
 *   - Activations are NDHWC (channels innermost), weights are DHWIO
 *     W[kd][kh][kw][c_in][c_out]; all tensors are dense and contiguous.
 *   - Convolution is a cross-correlation: output o reads input o*stride +
 *     tap - pad_before (no kernel flip).  CF_PAD_SAME_TF uses TensorFlow's
 *     SAME rule (out = ceil(in/stride), the odd padding element after the
 *     data); CF_PAD_VALID has no padding (out = floor((in-k)/stride)+1).
 *   - Every pointer is a DEVICE pointer owned by the caller, except where
 *     stated.  The library never allocates or frees device memory, never
 *     synchronises, and launches on the caller's `stream` (a hipStream_t,
 *     may be NULL for the default stream).  Calls are asynchronous and
 *     stream-ordered.
 *   - CF_BF16 tensors hold IEEE bfloat16; every bf16 store rounds to nearest
 *     even.  Accumulation is fp32 in every dtype.  bias, db and dW are
 *     always fp32.
 *   - Errors: arguments are validated on the host before any launch.  On a
 *     validation error nothing is launched, outputs are untouched, the code
 *     is returned and cf_last_error() describes it.  A batch of 0 (or any
 *     empty extent) is a no-op returning CF_OK.  A failed launch returns
 *     CF_ERR_LAUNCH.  Input and output buffers of a call must not overlap
 *     unless stated (CF_ERR_ALIAS).  Pointers must be 16-byte aligned
 *     (CF_ERR_ALIGNMENT).
 *   - Results are deterministic: no floating-point atomics; every reduction
 *     has a fixed order that depends only on the shapes.
 */
#ifndef COSMOFLOW_H
#define COSMOFLOW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum cf_status {
  CF_OK = 0,
  CF_ERR_INVALID_ARG = 1, /* null pointer, non-positive size, kernel larger than input ... */
  CF_ERR_UNSUPPORTED = 2, /* valid but not implemented (e.g. pooling with k != s) */
  CF_ERR_ALIGNMENT = 3,   /* a pointer is not 16-byte aligned */
  CF_ERR_ALIAS = 4,       /* input and output buffers overlap where that is forbidden */
  CF_ERR_WORKSPACE = 5,   /* workspace missing or smaller than the size query returns */
  CF_ERR_LAUNCH = 6       /* the HIP runtime reported an error */
} cf_status;

typedef enum cf_dtype { CF_F32 = 0, CF_BF16 = 1 } cf_dtype;

typedef enum cf_pad { CF_PAD_SAME_TF = 0, CF_PAD_VALID = 1 } cf_pad;

/* Geometry of one 3D convolution layer.  n, d, h, w: batch and input
 * extent; c_in, c_out: channels; kd, kh, kw: kernel; sd, sh, sw: strides;
 * pad: a cf_pad; dtype: a cf_dtype (type of x, W, z, dz, dx). */
typedef struct cf_conv3d_desc {
  int32_t n, d, h, w;
  int32_t c_in, c_out;
  int32_t kd, kh, kw;
  int32_t sd, sh, sw;
  int32_t pad;
  int32_t dtype;
} cf_conv3d_desc;

/* Library version string (static storage). */
const char *cf_version(void);

/* Message of the last error returned on the calling thread ("" if none). */
const char *cf_last_error(void);

/* Host-only.  Output extent out_dhw[3] of the convolution described by desc
 * (SAME: ceil(in/s); VALID: floor((in-k)/s)+1). */
cf_status cf_conv3d_out_shape(const cf_conv3d_desc *desc, int32_t out_dhw[3]);

/* Forward convolution, Section III-C / Algorithm 1:
 *   z[n,o,co] = sum_{t,ci} x[n, o*s + t - pad_before, ci] * W[t,ci,co]
 * x: [n,d,h,w,c_in], W: [kd,kh,kw,c_in,c_out], z: [n,od,oh,ow,c_out], all in
 * desc->dtype.  z must not overlap x or W. */
cf_status cf_conv3d_fwd(const cf_conv3d_desc *desc, const void *x, const void *w,
                        void *z, void *stream);

/* Backward data, Section III-C (the operator that propagates the output
 * difference signal to the input): the adjoint of cf_conv3d_fwd in x,
 *   dx[n,i,ci] = sum over (o,t) with o*s + t - pad_before = i of
 *                sum_co dz[n,o,co] * W[t,ci,co].
 * dz: [n,od,oh,ow,c_out], W as above, dx: [n,d,h,w,c_in]; every element of
 * dx is written (zero where no output reads it).  dx must not overlap dz/W. */
cf_status cf_conv3d_bwd_data(const cf_conv3d_desc *desc, const void *dz, const void *w,
                             void *dx, void *stream);

/* Bytes of device workspace cf_conv3d_bwd_weight needs for desc (the
 * per-slice fp32 partial sums of the split reduction); 0 on invalid desc. */
size_t cf_conv3d_bwd_weight_workspace_size(const cf_conv3d_desc *desc);

/* Backward weights, Section III-C (a forward-like convolution with a large
 * reduction and a small output; voxel slices accumulate privately and are
 * then combined): the adjoint of cf_conv3d_fwd in W,
 *   dW[t,ci,co] = sum_{n,o} x[n, o*s + t - pad_before, ci] * dz[n,o,co].
 * x and dz in desc->dtype, dW fp32 [kd,kh,kw,c_in,c_out] (overwritten, not
 * accumulated).  ws: caller-owned device workspace of at least
 * cf_conv3d_bwd_weight_workspace_size(desc) bytes (may be NULL if that is 0).
 * The reduction over voxels is split into fixed slices whose partials are
 * summed in slice order, so the result is bitwise reproducible. */
cf_status cf_conv3d_bwd_weight(const cf_conv3d_desc *desc, const void *x, const void *dz,
                               float *dw, void *ws, size_t ws_bytes, void *stream);

/* Backward weights without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc).  Same operation, kernels and result bits
 * as cf_conv3d_bwd_weight; the split reduction's partials go to a scratch
 * region the library owns instead: a file-scope device array of
 * CF_NOALLOC_SCRATCH_BYTES per GPU, held from the first use on that GPU until
 * the process ends.  Nothing is allocated or freed by the call.  A layer whose
 * partials need more than that returns CF_ERR_UNSUPPORTED (use
 * cf_conv3d_bwd_weight with a workspace).  Every call on one GPU shares that
 * GPU's region, and the region keeps the last call's contents (every partial
 * is written before it is summed, so nothing needs clearing): calls that
 * overlap in time on one GPU (different streams, or host threads without
 * ordering) race and give undefined results; calls ordered on one stream do
 * not.  CF_ERR_LAUNCH if the region's device address cannot be resolved. */
#define CF_NOALLOC_SCRATCH_BYTES (16u << 20)
cf_status cf_conv3d_bwd_weight_noalloc(const cf_conv3d_desc *desc, const void *x, const void *dz,
                                       float *dw, void *stream);

/* Bytes of workspace cf_avgpool3d_lrelu_bwd needs (per-block bias partials);
 * d, h, w = the conv-output (pool input) extent. */
size_t cf_avgpool3d_lrelu_bwd_workspace_size(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c);

/* dz of a pooled layer whose forward ran fused (cf_conv3d_fwd_fused with
 * CF_FUSE_POOL2): the adjoints of the 2^3 stride-2 pool and of the leaky ReLU
 * (Section III-C: pooling is a per-channel convolution with constant weights
 * 1/8; Section III-A: leaky ReLU after every convolution) in one pass,
 *   dz[n,i,c] = dp[n,i/2,c] / 8 * (mask(n,i,c) ? 1 : alpha)  (0 where no
 *               complete window covers i),          db[c] = sum dz[.,c],
 * i.e. cf_avgpool3d_bwd then cf_bias_lrelu_bwd with the slope taken from the
 * forward's mask instead of the saved activation.  d,h,w = the conv-output
 * extent; dp [n,d/2,h/2,w/2,c] and dz [n,d,h,w,c] in dtype; mask as in
 * cf_conv3d_mask_bytes (bit per dz element); db fp32 [c] (overwritten; may be
 * NULL, then ws is unused), summed over the unrounded fp32 products in a fixed
 * order.  c must be a power-of-two multiple of 16 bytes of elements (at most
 * 64 of them) and at most 256, else CF_ERR_UNSUPPORTED; alpha finite, >= 0. */
cf_status cf_avgpool3d_lrelu_bwd(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c, int32_t dtype,
                                 const void *dp, const void *mask, float alpha, void *dz, float *db,
                                 void *ws, size_t ws_bytes, void *stream);

/* Bias + leaky ReLU forward (Section III-A):
 *   y[v,c] = u > 0 ? u : alpha*u,  u = z[v,c] + bias[c]   (u in fp32)
 * nvox = number of voxels (n*d*h*w), c = channels; z, y in dtype; bias fp32
 * [c].  y may alias z exactly (in place); partial overlap is CF_ERR_ALIAS.
 * alpha must be finite. */
cf_status cf_bias_lrelu_fwd(int64_t nvox, int32_t c, int32_t dtype, const void *z,
                            const float *bias, float alpha, void *y, void *stream);

/* Bytes of workspace cf_bias_lrelu_bwd needs (per-block bias partials). */
size_t cf_bias_lrelu_bwd_workspace_size(int64_t nvox, int32_t c);

/* Bias + leaky ReLU backward:
 *   dz[v,c] = dy[v,c] * (y[v,c] > 0 ? 1 : alpha),   db[c] = sum_v dz[v,c].
 * The slope is read from the SAVED OUTPUT y (for alpha > 0, y > 0 exactly
 * when the pre-activation is > 0; at a pre-activation of exactly 0 the slope
 * is alpha).  dy, y, dz in dtype; db fp32 [c] (overwritten); the sum runs in
 * fp32 over the unrounded products in a fixed order.  dz may alias dy
 * exactly.  db may be NULL (no bias gradient; ws then unused). */
cf_status cf_bias_lrelu_bwd(int64_t nvox, int32_t c, int32_t dtype, const void *dy,
                            const void *y, float alpha, void *dz, float *db, void *ws,
                            size_t ws_bytes, void *stream);

/* Average pooling forward (Section III-C: per-channel convolution with
 * constant weights 1/k^3; Section III-A: stride (2,2,2)):
 *   p[n,o,c] = (1/k^3) * sum_{a in [0,k)^3} y[n, o*s + a, c]
 * y: [n,d,h,w,c], p: [n,(d-k)/s+1,(h-k)/s+1,(w-k)/s+1,c] (floor), dtype.
 * Only non-overlapping windows (k == s) are implemented; other pairs return
 * CF_ERR_UNSUPPORTED.  The sum is fp32, rounded once on store. */
cf_status cf_avgpool3d_fwd(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c,
                           int32_t k, int32_t s, int32_t dtype, const void *y, void *p,
                           void *stream);

/* Average pooling backward: the adjoint of cf_avgpool3d_fwd,
 *   dy[n,i,c] = dp[n, i/s, c] / k^3 where i is covered by a window, else 0.
 * Dimensions as for the forward call (d,h,w = the forward INPUT extent). */
cf_status cf_avgpool3d_bwd(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c,
                           int32_t k, int32_t s, int32_t dtype, const void *dp, void *dy,
                           void *stream);

/* Both backward products of a layer from one dz (Section III-C: the data
 * and weight gradients read the same dz): dW exactly as cf_conv3d_bwd_weight
 * and dx exactly as cf_conv3d_bwd_data, with their arguments (bitwise the same
 * results).  Where both products run on the fp32 register-streamed kernels
 * one launch holds them side by side; otherwise the two calls run in
 * sequence.  ws: cf_conv3d_bwd_weight_workspace_size bytes; dx must not
 * overlap x, dW or ws (CF_ERR_ALIAS). */
cf_status cf_conv3d_bwd(const cf_conv3d_desc *desc, const void *x, const void *dz, const void *w,
                        float *dw, void *dx, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Fused layer variants.  Same mathematics as the unfused composition
 *   conv -> bias + leaky ReLU -> 2^3 stride-2 average pool     (forward)
 *   pool backward -> leaky-ReLU backward (+ db) -> weight / data gradient
 * but the full-resolution activation and its gradient never reach HBM: the
 * forward epilogue writes the pooled output plus a 1-bit slope mask, and the
 * backward kernels rebuild dz from the pooled-output gradient and the mask.
 * Rounding differs from the unfused composition only in where values are
 * rounded to bf16 (the fused path rounds once, at the pooled output).
 * ------------------------------------------------------------------------ */

/* flags */
#define CF_FUSE_POOL2 1u /* a 2^3 stride-2 average pool follows the activation */
#define CF_FUSE_MASK 2u  /* forward: also write the slope mask (implied by CF_FUSE_POOL2) */

/* Bitmask of the fused entry points of this library that accept (desc, flags):
 * 1 = cf_conv3d_fwd_fused, 2 = cf_conv3d_bwd_weight_fused,
 * 4 = cf_conv3d_bwd_data_fused, 8 = cf_conv3d_bwd_weight_fused_dz.
 * The backward calls take (g, mask) = (pooled-output gradient, slope mask)
 * with CF_FUSE_POOL2, and (dy, y) -- the gradient of the activation and the
 * activation the fused forward wrote -- with flags == 0 (fp32 layers).
 * Host-only; 0 on an invalid desc. */
int32_t cf_conv3d_fused_supported(const cf_conv3d_desc *desc, uint32_t flags);

/* Bytes of the slope mask of a layer: one bit per element of the conv output
 * [n,od,oh,ow,c_out], bit e (NDHWC element index) = bit e%32 of 32-bit word
 * e/32, i.e. ceil(n*od*oh*ow*c_out/32)*4 bytes.  0 on invalid desc. */
size_t cf_conv3d_mask_bytes(const cf_conv3d_desc *desc);

/* Fused forward: u = conv(x, W) + bias (fp32), y = u > 0 ? u : alpha*u.
 * With CF_FUSE_POOL2: out = avgpool 2^3 stride 2 of y, [n,od/2,oh/2,ow/2,c_out]
 * (floor), summed in fp32 and rounded once; mask (required, see
 * cf_conv3d_mask_bytes) records u > 0 for every conv-output element.
 * Without it: out = y [n,od,oh,ow,c_out] in dtype, and mask may be NULL
 * (required with CF_FUSE_MASK).
 * alpha must be finite and >= 0 (then u > 0 <=> y > 0, the slope rule of
 * cf_bias_lrelu_bwd).  Unsupported shapes return CF_ERR_UNSUPPORTED (see
 * cf_conv3d_fused_supported); the unfused calls cover every shape. */
cf_status cf_conv3d_fwd_fused(const cf_conv3d_desc *desc, const void *x, const void *w,
                              const float *bias, float alpha, uint32_t flags, void *out,
                              void *mask, void *stream);

/* Workspace bytes of cf_conv3d_bwd_weight_fused for (desc, flags). */
size_t cf_conv3d_bwd_weight_fused_workspace_size(const cf_conv3d_desc *desc, uint32_t flags);

/* Fused backward-weights.  With CF_FUSE_POOL2, g is the gradient of the
 * pooled output [n,od/2,oh/2,ow/2,c_out] and mask the forward's slope mask:
 *   dz[v,c] = g[pool(v),c] / 8 * (mask(v,c) ? 1 : alpha)  (0 where no window covers v)
 * With flags == 0 (unpooled layer, the "dy + y" form), g is the gradient dy of
 * the activation and mask points to the activation y [n,od,oh,ow,c_out] the
 * fused forward wrote (both in dtype):
 *   dz[v,c] = dy[v,c] * (y[v,c] > 0 ? 1 : alpha)   (the slope rule of cf_bias_lrelu_bwd)
 *   dW[t,ci,co] = sum_{n,o} x[n, o*s + t - pad_before, ci] * dz[n,o,co]   (fp32)
 *   db[c] = sum_v dz[v,c]                                                  (fp32)
 * dz is formed in fp32 (bf16 path: rounded to bf16 before the product, as
 * the unfused path stores it); db sums the unrounded values.  ws: caller
 * workspace of cf_conv3d_bwd_weight_fused_workspace_size bytes.  Partial sums
 * are combined in a fixed order (bitwise reproducible). */
cf_status cf_conv3d_bwd_weight_fused(const cf_conv3d_desc *desc, const void *x, const void *g,
                                     const void *mask, float alpha, uint32_t flags, float *dw,
                                     float *db, void *ws, size_t ws_bytes, void *stream);

/* Fused backward-weights that also stores the rebuilt dz (bit 8 of
 * cf_conv3d_fused_supported; either form of the inputs).  dW, db and ws exactly
 * as cf_conv3d_bwd_weight_fused (bitwise the same results); in addition dz
 * [n,od,oh,ow,c_out] in dtype receives every element of the rebuilt
 * gradient, rounded as described there -- the input a following
 * cf_conv3d_bwd_data call needs, which then returns the same dx bits as
 * cf_conv3d_bwd_data_fused.  The tiles of the weight-gradient pass partition
 * dz, so each element is built and stored once; dz must not overlap any
 * other argument (CF_ERR_ALIAS).  NULL dz is CF_ERR_INVALID_ARG. */
cf_status cf_conv3d_bwd_weight_fused_dz(const cf_conv3d_desc *desc, const void *x, const void *g,
                                        const void *mask, float alpha, uint32_t flags, float *dw,
                                        float *db, void *dz, void *ws, size_t ws_bytes,
                                        void *stream);

/* Fused backward-data: dz is rebuilt from (g, mask) -- the pooled-output
 * gradient and the slope mask with CF_FUSE_POOL2, (dy, y) with flags == 0 --
 * exactly as in cf_conv3d_bwd_weight_fused (rounded to the path dtype), then
 *   dx[n,i,ci] = sum over (o,t) with o*s + t - pad_before = i of sum_co dz[n,o,co] * W[t,ci,co].
 * dx [n,d,h,w,c_in] in dtype; every element is written. */
cf_status cf_conv3d_bwd_data_fused(const cf_conv3d_desc *desc, const void *g, const void *mask,
                                   const void *w, float alpha, uint32_t flags, void *dx,
                                   void *stream);

/* Fused backward of a layer in one call (Section III-A: leaky ReLU follows
 * every convolution; Section III-C: the weight- and data-gradient operators of
 * the same layer read the same dz): dW and db exactly as
 * cf_conv3d_bwd_weight_fused and dx exactly as cf_conv3d_bwd_data_fused, with
 * the same arguments (bitwise the same results).  Where both products are
 * small (the stack's unpooled deep layers in fp32) one launch runs them side
 * by side; otherwise the two calls run in sequence.  ws: the
 * cf_conv3d_bwd_weight_fused_workspace_size bytes; dx must not overlap dW, db
 * or ws (CF_ERR_ALIAS).  Supported wherever both fused calls are (bits 2 and 4
 * of cf_conv3d_fused_supported). */
cf_status cf_conv3d_bwd_fused(const cf_conv3d_desc *desc, const void *x, const void *g,
                              const void *mask, const void *w, float alpha, uint32_t flags,
                              float *dw, float *db, void *dx, void *ws, size_t ws_bytes,
                              void *stream);

/* ------------------------------------------------------------------------
 * Deferred gradient sums.  Every weight- and bias-gradient entry point ends
 * with fixed-order column sums of per-workgroup fp32 partials held in its
 * workspace (dW[c] = sum_r part[r][c], r ascending in a fixed grouping: the
 * bitwise-reproducible reduction).  Nothing in a backward pass reads dW or db,
 * so a training step can run those sums for all layers in one launch: the
 * _deferred variants below do everything their plain counterparts do except
 * these sums, and describe them in `pending` instead.  Passing the collected
 * descriptions to cf_reduce_partials (in stream order, before dW / db are
 * read and before the workspaces are reused) writes exactly the bits the
 * plain call would have written.
 * ------------------------------------------------------------------------ */

/* One pending sum: out[c] = sum over r of part[r * cols + c], c < cols. */
typedef struct cf_reduction {
  const float *part; /* [rows][cols] fp32 partials (device, in a caller workspace) */
  float *out;        /* [cols] fp32 result (device) */
  int32_t rows, cols;
} cf_reduction;

/* Most pending sums one deferred call records. */
#define CF_MAX_PENDING 4

/* Runs n pending sums (any mix of layers) in as few launches as possible;
 * each job's result bits depend only on its partials and (rows, cols).
 * Pointers 4-byte aligned (CF_ERR_ALIGNMENT); out must not overlap its own
 * partials (CF_ERR_ALIAS). */
cf_status cf_reduce_partials(int32_t n, const cf_reduction *jobs, void *stream);

/* cf_conv3d_bwd_weight without the final sums: dW is written by
 * cf_reduce_partials(*npending, pending).  pending: room for CF_MAX_PENDING
 * entries (host memory); *npending receives the count (0 when nothing is
 * pending, e.g. an empty batch, whose dW is written directly). */
cf_status cf_conv3d_bwd_weight_deferred(const cf_conv3d_desc *desc, const void *x, const void *dz,
                                        float *dw, void *ws, size_t ws_bytes,
                                        cf_reduction *pending, int32_t *npending, void *stream);

/* cf_avgpool3d_lrelu_bwd without the final bias-gradient sum (db by
 * cf_reduce_partials).  pending / npending as above. */
cf_status cf_avgpool3d_lrelu_bwd_deferred(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c, int32_t dtype,
                                          const void *dp, const void *mask, float alpha, void *dz, float *db,
                                          void *ws, size_t ws_bytes, cf_reduction *pending,
                                          int32_t *npending, void *stream);

/* cf_bias_lrelu_bwd without the final bias-gradient sum (dz is written by
 * this call; db by cf_reduce_partials).  pending / npending as above. */
cf_status cf_bias_lrelu_bwd_deferred(int64_t nvox, int32_t c, int32_t dtype, const void *dy,
                                     const void *y, float alpha, void *dz, float *db, void *ws,
                                     size_t ws_bytes, cf_reduction *pending, int32_t *npending,
                                     void *stream);

/* cf_conv3d_bwd_weight_fused (dz == NULL) or cf_conv3d_bwd_weight_fused_dz
 * (dz != NULL: dz is written by this call) without the final sums of dW and
 * db.  pending / npending as above. */
cf_status cf_conv3d_bwd_weight_fused_deferred(const cf_conv3d_desc *desc, const void *x,
                                              const void *g, const void *mask, float alpha,
                                              uint32_t flags, float *dw, float *db, void *dz,
                                              void *ws, size_t ws_bytes, cf_reduction *pending,
                                              int32_t *npending, void *stream);

/* cf_conv3d_bwd without the final sums of dW (dx is written by this call).
 * pending / npending as above. */
cf_status cf_conv3d_bwd_deferred(const cf_conv3d_desc *desc, const void *x, const void *dz,
                                 const void *w, float *dw, void *dx, void *ws, size_t ws_bytes,
                                 cf_reduction *pending, int32_t *npending, void *stream);

/* cf_conv3d_bwd_fused without the final sums of dW and db (dx is written by
 * this call).  pending / npending as above. */
cf_status cf_conv3d_bwd_fused_deferred(const cf_conv3d_desc *desc, const void *x, const void *g,
                                       const void *mask, const void *w, float alpha,
                                       uint32_t flags, float *dw, float *db, void *dx, void *ws,
                                       size_t ws_bytes, cf_reduction *pending, int32_t *npending,
                                       void *stream);

/* ------------------------------------------------------------------------
 * Parameter update (Section III-B, "SGD Optimizer").  Per parameter group l
 * (a contiguous range of flat fp32 arrays) at step t:
 *   eta_t  = (eta0 - eta_min) * (1 - min(t, t_decay) / t_decay) + eta_min
 *   vn     = ||v_l||_2,  gn = ||g_l||_2
 *   eta*   = coef * vn / gn if vn != 0 and gn != 0, else fallback
 *   eta+   = min(eta*, clip)
 *   g*     = eta+ * g_l
 *   m      = beta1 m + (1 - beta1) g*,  s = beta2 s + (1 - beta2) g*^2
 *   v_l   -= eta_t sqrt(1 - beta2^(t+1)) / (1 - beta1^(t+1)) * m / (sqrt(s) + eps_hat)
 * i.e. Adam (Kingma and Ba, in the epsilon-hat form the paper's constant
 * names) on the gradient rescaled by LARC's clipped local rate, with the
 * global rate on a power-1 polynomial decay.  The paper's values: eta0 =
 * 2e-3, eta_min = 1e-4, beta1 = 0.9, beta2 = 0.999, eps_hat = 1e-8, coef =
 * 0.002, fallback = 6.25e-5, clip = 1; t_decay is not given there.
 * t counts the updates already applied (0 for the first): the decay starts
 * from eta0, Adam's bias corrections count from 1.  The clamp of t at
 * t_decay is a reading (the paper leaves the rate after t_decay open).
 * ------------------------------------------------------------------------ */
typedef struct cf_adam_larc_hparams {
  double eta0, eta_min; /* global rate at t = 0 and from t = t_decay on */
  int64_t t_decay;      /* length of the linear decay, > 0 */
  double beta1, beta2;  /* Adam's moment decays, in [0, 1) */
  double eps_hat;       /* >= 0 */
  double larc_coef;     /* eta* = coef * ||v|| / ||g|| */
  double larc_fallback; /* eta* when either norm is zero */
  double larc_clip;     /* eta+ = min(eta*, clip) */
} cf_adam_larc_hparams;

/* Most parameter groups one call takes. */
#define CF_ADAM_MAX_GROUPS 128

/* Bytes of device workspace cf_adam_larc_step needs for these groups (16
 * per chunk; 0 when every group is empty or the arguments are invalid).
 * offsets: host array of ngroups + 1 element offsets, as below. */
size_t cf_adam_larc_workspace_size(int32_t ngroups, const int64_t *offsets);

/* One update of every group.  offsets (HOST memory, ngroups + 1 entries,
 * non-decreasing): group l is elements [offsets[l], offsets[l+1]) of the
 * flat fp32 device arrays v (parameters, updated in place), g (gradient,
 * read only), m and s (Adam's first and second moments, updated in place;
 * zero before the first update).  Every group start offsets[l], l <
 * ngroups, must be a multiple of 4 (CF_ERR_ALIGNMENT); group lengths are
 * free.  v16: NULL, or a bf16 device array that receives RNE(v) after the
 * update at the same offsets (the copy the convolutions of a bf16 step
 * read).  ws: device workspace of cf_adam_larc_workspace_size() bytes; its
 * contents need no initialisation.  All device pointers 16-byte aligned;
 * v, g, m, s, v16 and ws must not overlap (CF_ERR_ALIAS).  Elements outside
 * the groups are not touched.  The norms are summed in fp64 in a fixed
 * order and the update is evaluated in fp64 with one rounding per fp32
 * store: results are deterministic.  More than CF_ADAM_MAX_GROUPS groups:
 * CF_ERR_UNSUPPORTED.  Invalid hyperparameters (non-finite values, beta
 * outside [0, 1), eps_hat < 0, t < 0, t_decay <= 0): CF_ERR_INVALID_ARG. */
cf_status cf_adam_larc_step(int32_t ngroups, const int64_t *offsets, int64_t t,
                            const cf_adam_larc_hparams *hp, float *v, const float *g, float *m,
                            float *s, void *v16, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Fully-connected head and loss (Section III-A: three fully-connected layers
 * follow the convolutions, each with leaky ReLU -- applied by
 * cf_bias_lrelu_fwd / _bwd with nvox = m rows and c = n features -- the last
 * with three outputs, one per regressed cosmological parameter).
 *
 * A layer maps the m rows of x [m][k] (for the first layer: each sample's
 * NDHWC activation flattened in memory order, k = d*h*w*c) to
 *   z[i][j] = sum_{l < k} x[i][l] W[l][j],    W stored [k][n] (row l = input l).
 * x, W, z, dz, dx are in dtype; dW is fp32; products and sums are fp32.
 * Sizes: m >= 0 (m == 0 is a no-op), 1 <= k < 2^31, 1 <= n <= 65536 and
 * k * n < 2^40.  All device pointers 16-byte aligned; outputs must not
 * overlap inputs (CF_ERR_ALIAS).  Every sum has an order fixed by the sizes:
 * results are deterministic.  Bandwidth-bound: each call streams W (or dW)
 * through HBM once per 8 rows of the batch.
 * ------------------------------------------------------------------------ */

/* Bytes of device workspace cf_fc_fwd needs (fp32 partial sums of the split
 * over k; 0 for invalid sizes). */
size_t cf_fc_fwd_workspace_size(int32_t m, int32_t k, int32_t n);

/* z = x W (see above).  ws: cf_fc_fwd_workspace_size() bytes, contents
 * need no initialisation, must not overlap x, W or z. */
cf_status cf_fc_fwd(int32_t m, int32_t k, int32_t n, int32_t dtype, const void *x, const void *w,
                    void *z, void *ws, size_t ws_bytes, void *stream);

/* Backward data, the adjoint in x:  dx[i][l] = sum_j dz[i][j] W[l][j].
 * dz [m][n], W [k][n], dx [m][k]. */
cf_status cf_fc_bwd_data(int32_t m, int32_t k, int32_t n, int32_t dtype, const void *dz,
                         const void *w, void *dx, void *stream);

/* Backward weights, the adjoint in W:  dW[l][j] = sum_{i < m} x[i][l] dz[i][j]
 * (summed over the batch rows in order), dW fp32 [k][n], overwritten.  m == 0
 * writes dW = 0. */
cf_status cf_fc_bwd_weight(int32_t m, int32_t k, int32_t n, int32_t dtype, const void *x,
                           const void *dz, float *dw, void *stream);

/* Loss.  The paper does not name it; it is read as the mean squared error
 * of the regressed parameters over the batch:
 *   loss = (1/(m n)) sum_{i,j} (p[i][j] - t[i][j])^2,
 *   dp[i][j] = 2 (p[i][j] - t[i][j]) / (m n)      (dL/dp, rounded once to dtype).
 * p, dp [m][n] in dtype; t [m][n] fp32; loss: one fp32 on the device.  dp may
 * be NULL (loss only).  m, n >= 1 and m * n < 2^31.  One workgroup. */
cf_status cf_mse_loss(int32_t m, int32_t n, int32_t dtype, const void *p, const float *t,
                      float *loss, void *dp, void *stream);

/* The whole head in one call (Section III-A: fully-connected layers with
 * leaky ReLU after the convolutions; the loss as cf_mse_loss reads it):
 * forward, loss and backward of nlayers layers of widths dims[0] -> dims[1]
 * -> ... -> dims[nlayers], in four kernel launches -- the first layer's
 * split-K forward, its column sums with bias and leaky ReLU, one workgroup
 * for the rest of the forward, the loss and the later layers' backward
 * (their weights and activations held in LDS), and one pass over the first
 * layer's W for its dW and dx.  The results are
 * those of the per-layer calls (cf_fc_fwd, cf_bias_lrelu_fwd, cf_mse_loss,
 * cf_bias_lrelu_bwd, cf_fc_bwd_weight, cf_fc_bwd_data) with the same rounding
 * points; the first layer's y, dW and dx are bitwise those calls' results
 * (given the same dz), the later layers' sums take their own fixed order.
 * Deterministic.
 *   x [m][dims[0]] (dtype), w[i] [dims[i]][dims[i+1]] (dtype), b[i] fp32
 *   [dims[i+1]], target fp32 [m][dims[nlayers]];
 *   outputs: y[i] [m][dims[i+1]] = lrelu(z + b) (dtype); loss (one fp32);
 *   dz[i] [m][dims[i+1]] (dtype) = dL/dy[i] * slope (dL/dy of the last layer
 *   is the loss gradient rounded to dtype); db[i] fp32 [dims[i+1]]; dw[i] fp32
 *   [dims[i]][dims[i+1]]; dx[i] [m][dims[i]] (dtype) the gradient of layer
 *   i's input (dx[0]: of x).
 * Limits (else CF_ERR_UNSUPPORTED, nothing launched): 2 <= nlayers <= 4,
 * 1 <= m <= 8; dims[0] a multiple of 8 below 2^31; dims[1] / V a power of
 * two from 8 to 64 (V = 8 for bf16, 4 for fp32); every later width <= 512,
 * m * (dims[1] + ... + dims[nlayers]) <= 8192 and the sum over the later
 * layers of dims[i] * (dims[i+1] + 1) <= 16384.  Every pointer (the arrays
 * are host arrays of nlayers device pointers) non-NULL and 16-byte aligned;
 * no output may overlap an input or another output (CF_ERR_ALIAS).
 * ws: cf_fc_head_workspace_size() bytes (the first layer's partial sums),
 * no initialisation needed. */
size_t cf_fc_head_workspace_size(int32_t m, int32_t nlayers, const int32_t *dims);
cf_status cf_fc_head(int32_t m, int32_t nlayers, const int32_t *dims, int32_t dtype, const void *x,
                     const void *const *w, const float *const *b, float alpha, const float *target, void *const *y,
                     void *const *dz, void *const *dx, float *const *dw, float *const *db, float *loss, void *ws,
                     size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* COSMOFLOW_H */
