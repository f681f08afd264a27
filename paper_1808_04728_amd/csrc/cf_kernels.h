// cf_kernels.h -- host-side launchers of the gfx950 kernels (internal).
//
// The C ABI layer (cf_api.cpp) validates arguments, derives the geometry
// below and calls these launchers; they only pick a kernel variant and
// launch it on the given stream.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace cf {

// Compute units of a gfx950 device (MI350X / MI355X: 8 XCDs x 32 CUs).  The
// library is built for gfx950 only, so persistent grids are sized from this
// constant instead of a per-launch device query; on a partitioned device with
// fewer CUs the same grid simply queues more workgroups per CU (same results:
// no partition of work or summation order depends on it).
constexpr int kNumCUs = 256;

// Fully resolved geometry of one convolution layer.
struct ConvShape {
  int n, d, h, w;        // input extent
  int ci, co;            // channels
  int kd, kh, kw;        // kernel
  int sd, sh, sw;        // strides
  int pd, ph, pw;        // padding before (after = whatever SAME leaves)
  int od, oh, ow;        // output extent
  int dtype;             // DT_F32 / DT_BF16
};

// First-layer (few input channels) kernels, conv_smallc.hip.
struct SmallcParams {
  int n, d, h, w, ci, co;
  int kd, kh, kw, pd, ph, pw;
  int od, oh, ow;
  int pod, poh, pow_;   // pooled extents (floor(o/2))
  int tiles_per_block;  // backward-weights: output tiles folded into one workgroup
};
// 16 -> 32 channel stride-1 forward (bf16), conv_c16.hip.  epi: 0 store z,
// 1 bias + lReLU -> y (+ mask if non-null), 2 bias + lReLU + mask + 2^3 pool.
struct C16Params {
  int n, d, h, w;
  int pd, ph, pw;
  int od, oh, ow;
  int pod, poh, pow_;
  int x_bytes;  // forward: extent of the range-checked input buffer
  int g_bytes;  // backward-data: extent of dz (or of the pooled gradient, fused)
  int m_bytes;  // backward-data, fused: extent of the slope mask
};
bool c16_fwd_supported(const ConvShape &s);
// backward data of the same layers (conv_c16_bwd.hip); fused: g is the pooled-output
// gradient and mask the forward's slope mask, else g is dz
bool c16_bwd_supported(const ConvShape &s);
// backward weights of the 4^3 16 -> 32 layer (conv_c16_wgrad.hip); fused as above, db only when fused;
// dz_out (fused only, may be null) receives the rebuilt dz [n,od,oh,ow,32] in bf16
bool c16_wgrad_supported(const ConvShape &s);
size_t c16_wgrad_workspace(const ConvShape &s);
hipError_t launch_conv_bwd_weight_c16(const ConvShape &s, const void *x, const void *g, const uint32_t *mask,
                                      float alpha, float *dw, float *db, void *ws, bool fused, void *dz_out,
                                      hipStream_t st);
hipError_t launch_conv_bwd_data_c16(const ConvShape &s, const void *g, const uint32_t *mask, const void *w,
                                    float alpha, void *dx, bool fused, hipStream_t st);
hipError_t launch_conv_fwd_c16(const ConvShape &s, const void *x, const void *w, const float *bias, float alpha,
                               void *out, uint32_t *mask, int epi, hipStream_t st);

bool smallc_supported(const ConvShape &s, bool fused);
hipError_t launch_conv_fwd_smallc(const ConvShape &s, const void *x, const void *w, const float *bias,
                                  float alpha, void *out, uint16_t *mask, bool fused, hipStream_t st);
// bf16 first layer (1 -> 16 channels, 3^3, stride 1) with the pooled epilogue,
// even output extents: voxel-pair windows, conv_smallc_pair.hip.
bool l1pair_supported(const ConvShape &s);
hipError_t launch_l1pair_fwd(const ConvShape &s, const void *x, const void *w, const float *bias, float alpha,
                             void *out, uint16_t *mask, hipStream_t st);
bool smallc_wgrad_fused_supported(const ConvShape &s);
size_t smallc_wgrad_fused_workspace(const ConvShape &s);
// the same layer unfused (dz given), bf16, one input channel, 16 outputs: partials in ws
bool smallc_wgrad_dz_supported(const ConvShape &s);
size_t smallc_wgrad_dz_workspace(const ConvShape &s);
hipError_t launch_smallc_wgrad_dz(const ConvShape &s, const void *x, const void *dz, float *dw, void *ws,
                                  hipStream_t st);
hipError_t launch_smallc_wgrad_fused(const ConvShape &s, const void *x, const void *dp, const uint16_t *mask,
                                     float alpha, float *dw, float *db, void *ws, hipStream_t st);

// Deep-layer implicit GEMM (>= 32 contracted channels, bf16), conv_direct.hip.
// act: bias + leaky ReLU epilogue (out = y), optional 1-bit slope mask.
bool direct_supported(const ConvShape &s, bool fwd);
hipError_t launch_conv_fwd_direct(const ConvShape &s, const void *x, const void *w, const float *bias, float alpha,
                                  void *out, void *mask, bool act, hipStream_t st);
// pooled forward of a deep layer (bias + lReLU + slope mask + 2^3 pool; out = pooled output)
bool direct_pool_supported(const ConvShape &s);
hipError_t launch_conv_fwd_direct_pool(const ConvShape &s, const void *x, const void *w, const float *bias,
                                       float alpha, void *out, void *mask, hipStream_t st);
hipError_t launch_conv_bwd_data_direct(const ConvShape &s, const void *dz, const void *w, void *dx,
                                       hipStream_t st);
// backward-data of a fused deep layer (register kernel): gm = GRAD_POOL, g = pooled-output
// gradient, aux = slope mask; gm = GRAD_DYY, g = dy, aux = y; dz formed from them per load
hipError_t launch_conv_bwd_data_direct_fused(const ConvShape &s, const void *g, const void *aux, int gm, float alpha,
                                             const void *w, void *dx, hipStream_t st);
// their weight gradient (bf16, ci % 8 == 0, co % 64 == 0), conv_direct_wgrad.hip: K-split
// partials in ws, summed into dw (and db, fused) by launch_sum_rows.  gm selects the
// gradient operand: DWG_DZ g = dz; DWG_POOL g = pooled-output gradient, aux = slope
// mask (bit per conv-output element); DWG_DYY g = dy, aux = the activation y
enum : int { DWG_DZ = 0, DWG_POOL = 1, DWG_DYY = 3 };
bool direct_wgrad_supported(const ConvShape &s);
size_t direct_wgrad_workspace(const ConvShape &s, bool fused);
hipError_t launch_conv_bwd_weight_direct(const ConvShape &s, const void *x, const void *g, const void *aux, int gm,
                                         float alpha, float *dw, float *db, void *ws, hipStream_t st);

// fp32 implicit GEMM on v_mfma_f32_16x16x4_f32 (conv_f32.hip): forward for
// ci % 16 == 0 and co % 32 == 0, backward-data for co % 16 == 0 and ci % 16 == 0.
// epi: 0 store z, 1 bias + lReLU (+ mask if non-null), 2 bias + lReLU + mask +
// 2^3 pool (f32conv_pool_supported: stride 1, 32 output channels)
bool f32conv_supported(const ConvShape &s, bool fwd);
bool f32conv_pool_supported(const ConvShape &s);
hipError_t launch_conv_fwd_f32(const ConvShape &s, const float *x, const float *w, const float *bias, float alpha,
                               float *out, uint8_t *mask, int epi, hipStream_t st);
// y non-null: the A operand is dz = dy * (y > 0 ? 1 : alpha) from dy (the dz argument) and y
hipError_t launch_conv_bwd_data_f32(const ConvShape &s, const float *dz, const float *w, float *dx, hipStream_t st,
                                    const float *y = nullptr, float alpha = 0.f);

// fp32 backward-weights on v_mfma_f32_16x16x4_f32 (conv_f32_wgrad.hip), ci % 16 == 0,
// co % 16 == 0: voxel slices' partials in ws, summed by launch_sum_rows.  fused (the
// pooled 16 -> 32 layer, 32 output channels): g is the pooled-output gradient and
// mask the forward's slope mask; db and (if dz_out) the rebuilt dz come from the
// same pass
bool f32wgrad_supported(const ConvShape &s);
// the fused first layer in fp32 (one input channel, 16 outputs, 2^3 or 3^3): register-streamed
// input windows, the bias gradient as an MFMA row of ones (conv_f32_wgrad.hip)
bool l1f32_wgrad_supported(const ConvShape &s);
size_t l1f32_wgrad_workspace(const ConvShape &s);
hipError_t launch_l1_wgrad_f32(const ConvShape &s, const float *x, const float *dp, const uint16_t *mask,
                               float alpha, float *dw, float *db, void *ws, hipStream_t st);
bool f32wgrad_fused_supported(const ConvShape &s);
// gm: 0 g = dz; 1 g = pooled gradient, aux = slope mask; 3 g = dy, aux = the activation y
size_t f32wgrad_workspace(const ConvShape &s, int gm);
// fp32 backward of an unpooled fused layer (dz = dy * slope(y)): dW, db and dx
// in one launch where the planners pick the instantiated tile shapes, else the
// two launches in sequence; workspace as the (dy, y) weight gradient's.
hipError_t launch_conv_bwd_fused_f32(const ConvShape &s, const float *x, const float *dy, const float *y,
                                     const float *w, float alpha, float *dw, float *db, float *dx, void *ws,
                                     hipStream_t st);
// fp32 weight and data gradients of a layer from a stored dz: one launch where
// the planners pick the instantiated tile shapes, else the two launches in
// sequence; workspace as cf_conv3d_bwd_weight's.
hipError_t launch_conv_bwd_f32(const ConvShape &s, const float *x, const float *dz, const float *w, float *dw,
                               float *dx, void *ws, hipStream_t st);
// both backward products of a layer from a stored dz (conv_igemm.hip's dispatch)
hipError_t launch_conv_bwd(const ConvShape &s, const void *x, const void *dz, const void *w, float *dw, void *dx,
                           void *ws, hipStream_t st);
hipError_t launch_conv_bwd_weight_f32(const ConvShape &s, const float *x, const float *g, const void *aux,
                                      float alpha, float *dw, float *db, void *ws, int gm, float *dz_out,
                                      hipStream_t st);

hipError_t launch_conv_fwd(const ConvShape &s, const void *x, const void *w, void *z,
                           hipStream_t st);
hipError_t launch_conv_bwd_data(const ConvShape &s, const void *dz, const void *w, void *dx,
                                hipStream_t st);
size_t conv_bwd_weight_workspace(const ConvShape &s);
hipError_t launch_conv_bwd_weight(const ConvShape &s, const void *x, const void *dz, float *dw,
                                  void *ws, hipStream_t st);

hipError_t launch_bias_lrelu_fwd(int64_t nvox, int c, int dtype, const void *z,
                                 const float *bias, float alpha, void *y, hipStream_t st);
size_t bias_lrelu_bwd_workspace(int64_t nvox, int c);
hipError_t launch_bias_lrelu_bwd(int64_t nvox, int c, int dtype, const void *dy, const void *y,
                                 float alpha, void *dz, float *db, void *ws, hipStream_t st);

// out[c] = sum_{r < rows} part[r * cols + c], in an order fixed by (rows, cols).
// dz of a pooled layer from the pooled-output gradient and the slope mask (the
// adjoints of the 2^3 pool and of the leaky ReLU in one pass), db partials summed
// by launch_sum_rows (eltwise.hip); d, h, w = the conv-output extent
bool pool_lrelu_bwd_supported(long long nvox, int c, int dtype);
size_t pool_lrelu_bwd_workspace(int64_t nvox, int c);
hipError_t launch_pool_lrelu_bwd(int n, int d, int h, int w, int c, int dtype, const void *g, const void *mask,
                                 float alpha, void *dz, float *db, void *ws, hipStream_t st);
hipError_t launch_sum_rows(const float *part, float *out, int rows, int cols, hipStream_t st);
// one pending column sum out[c] = sum_r part[r][c] of a [rows][cols] fp32 matrix
struct SumJob {
  const float *part;
  float *out;
  int rows, cols;
};
// While a collector is installed on the calling thread, launch_sum_rows records
// its job there instead of launching it (the deferred entry points).
struct SumCollector {
  static constexpr int CAP = 4;
  int n;
  SumJob job[CAP];
};
void set_sum_collector(SumCollector *c);
// all jobs in as few launches as possible (same bits as one launch per job)
hipError_t launch_sum_batch(const SumJob *jobs, int n, hipStream_t st);

// Scratch region of the allocation-free backward-weights entry point
// (noalloc.hip): a file-scope device array of this many bytes per GPU.
constexpr size_t kNoallocScratchBytes = 16u << 20;
// device address of the current device's scratch region (resolved once per
// device with hipGetSymbolAddress, with that device current)
hipError_t noalloc_scratch(void **ptr);

// out[0..n) = 0 (a fill kernel, never hipMemsetAsync).
hipError_t launch_fill_zero(float *out, long long n, hipStream_t st);

hipError_t launch_avgpool_fwd(int n, int d, int h, int w, int c, int k, int dtype,
                              const void *y, void *p, hipStream_t st);
hipError_t launch_avgpool_bwd(int n, int d, int h, int w, int c, int k, int dtype,
                              const void *dp, void *dy, hipStream_t st);

// Parameter update (optim.hip): Adam + LARC + linear learning-rate decay over
// parameter groups of flat fp32 arrays.  Passed by value as a kernel argument.
constexpr int kOptMaxGroups = 128;
struct OptGroups {
  int n;                             // groups
  int chunk0[kOptMaxGroups + 1];     // first chunk of each group; chunk0[n] = all chunks
  int shift[kOptMaxGroups];          // a chunk of group l holds 1024 << shift[l] elements
  long long off[kOptMaxGroups + 1];  // element offsets; group l is [off[l], off[l+1])
};
struct OptHparams {
  double eta0, eta_min;
  long long t_decay;
  double beta1, beta2, eps_hat, coef, fallback, clip;
};
// fills G from n + 1 offsets (off[l] % 4 == 0 for l < n), returns the chunk count
int plan_opt_groups(int n, const long long *off, OptGroups *G);
// part: 2 doubles per chunk (caller workspace); v16 may be null
hipError_t launch_adam_larc(const OptGroups &G, int chunks, const OptHparams &hp, long long t, float *v,
                            const float *g, float *m, float *s, uint16_t *v16, double *part, hipStream_t st);

// Fully-connected layers (fc.hip): rows x[M][K], W[K][N], z[M][N].
size_t fc_fwd_workspace(int M, int K, int N);
hipError_t launch_fc_fwd(int M, int K, int N, int dtype, const void *x, const void *w, void *y, void *ws,
                         hipStream_t st);
hipError_t launch_fc_bwd_data(int M, int K, int N, int dtype, const void *dz, const void *w, void *dx,
                              hipStream_t st);
hipError_t launch_fc_bwd_weight(int M, int K, int N, int dtype, const void *x, const void *dz, float *dw,
                                hipStream_t st);
// mean squared error over n predictions; inv = 1 / n; dp may be null
// The whole head (fc.hip): first layer split-K forward and its column sums
// with bias and leaky ReLU, one workgroup for the rest of the forward, the
// loss and the later layers' backward, one pass for the first layer's dW and dx.
bool fc_head_supported(int M, int L, const int *dims, int dtype);
size_t fc_head_workspace(int M, int L, const int *dims);
hipError_t launch_fc_head(int M, int L, const int *dims, int dtype, const void *x, const void *const *w,
                          const float *const *b, float alpha, const float *target, void *const *y, void *const *dz,
                          void *const *dx, float *const *dw, float *const *db, float *loss, void *ws,
                          hipStream_t st);
hipError_t launch_mse_loss(long long n, int dtype, const void *p, const float *t, float *loss, void *dp,
                           float inv, hipStream_t st);

}  // namespace cf
