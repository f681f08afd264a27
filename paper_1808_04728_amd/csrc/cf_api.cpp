// cf_api.cpp -- the C ABI (include/cosmoflow.h): host-side argument
// validation, geometry, and dispatch to the gfx950 kernel launchers.
//
// Every check runs on the host before anything is launched, so a rejected
// call touches neither the device nor the outputs.

#include "../../include/cosmoflow.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "cf_common.h"
#include "cf_kernels.h"

namespace {

thread_local std::string g_last_error;

cf_status fail(cf_status code, const std::string &msg) {
  g_last_error = msg;
  return code;
}

cf_status ok() {
  g_last_error.clear();
  return CF_OK;
}

bool debug_sync() {
  static int v = [] {
    const char *e = std::getenv("CF_DEBUG_SYNC");
    return (e && e[0] && e[0] != '0') ? 1 : 0;
  }();
  return v != 0;
}

cf_status finish(hipError_t e, hipStream_t st, const char *what) {
  if (e == hipSuccess && debug_sync()) e = hipStreamSynchronize(st);
  if (e != hipSuccess)
    return fail(CF_ERR_LAUNCH, std::string(what) + ": " + hipGetErrorString(e));
  return ok();
}

size_t elem_size(int dtype) { return dtype == CF_BF16 ? 2 : 4; }

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

bool overlap(const void *a, size_t na, const void *b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + nb && b0 < a0 + na;
}

constexpr long long kMaxRows = (1LL << 31) - 1;

// Validate a convolution descriptor and resolve its geometry.
cf_status resolve(const cf_conv3d_desc *d, cf::ConvShape *s) {
  if (!d) return fail(CF_ERR_INVALID_ARG, "desc is NULL");
  if (d->n < 0) return fail(CF_ERR_INVALID_ARG, "batch n must be >= 0");
  if (d->d <= 0 || d->h <= 0 || d->w <= 0)
    return fail(CF_ERR_INVALID_ARG, "spatial extents d, h, w must be > 0");
  if (d->c_in <= 0 || d->c_out <= 0) return fail(CF_ERR_INVALID_ARG, "channels must be > 0");
  if (d->kd <= 0 || d->kh <= 0 || d->kw <= 0) return fail(CF_ERR_INVALID_ARG, "kernel extents must be > 0");
  if (d->sd <= 0 || d->sh <= 0 || d->sw <= 0) return fail(CF_ERR_INVALID_ARG, "strides must be > 0");
  if (d->pad != CF_PAD_SAME_TF && d->pad != CF_PAD_VALID) return fail(CF_ERR_INVALID_ARG, "unknown pad mode");
  if (d->dtype != CF_F32 && d->dtype != CF_BF16) return fail(CF_ERR_INVALID_ARG, "unknown dtype");
  const int in[3] = {d->d, d->h, d->w}, k[3] = {d->kd, d->kh, d->kw}, st[3] = {d->sd, d->sh, d->sw};
  int out[3], pb[3];
  for (int a = 0; a < 3; ++a) {
    if (d->pad == CF_PAD_SAME_TF) {
      out[a] = (in[a] + st[a] - 1) / st[a];
      long long tot = (long long)(out[a] - 1) * st[a] + k[a] - in[a];
      if (tot < 0) tot = 0;
      pb[a] = (int)(tot / 2);
    } else {
      if (k[a] > in[a]) return fail(CF_ERR_INVALID_ARG, "VALID convolution: kernel larger than input");
      out[a] = (in[a] - k[a]) / st[a] + 1;
      pb[a] = 0;
    }
  }
  const long long taps = (long long)k[0] * k[1] * k[2];
  if (taps * d->c_in >= kMaxRows || taps * d->c_out >= kMaxRows)
    return fail(CF_ERR_INVALID_ARG, "kernel volume x channels overflows 32 bits");
  const long long vin = (long long)d->n * in[0] * in[1] * in[2];
  const long long vout = (long long)d->n * out[0] * out[1] * out[2];
  if (vin >= kMaxRows || vout >= kMaxRows) return fail(CF_ERR_INVALID_ARG, "too many voxels (>= 2^31)");
  s->n = d->n; s->d = in[0]; s->h = in[1]; s->w = in[2];
  s->ci = d->c_in; s->co = d->c_out;
  s->kd = k[0]; s->kh = k[1]; s->kw = k[2];
  s->sd = st[0]; s->sh = st[1]; s->sw = st[2];
  s->pd = pb[0]; s->ph = pb[1]; s->pw = pb[2];
  s->od = out[0]; s->oh = out[1]; s->ow = out[2];
  s->dtype = d->dtype == CF_BF16 ? cf::DT_BF16 : cf::DT_F32;
  return CF_OK;
}

struct Sizes {
  size_t x, w, z;
};

Sizes conv_bytes(const cf::ConvShape &s) {
  const size_t es = s.dtype == cf::DT_BF16 ? 2 : 4;
  Sizes r;
  r.x = (size_t)s.n * s.d * s.h * s.w * s.ci * es;
  r.w = (size_t)s.kd * s.kh * s.kw * s.ci * s.co * es;
  r.z = (size_t)s.n * s.od * s.oh * s.ow * s.co * es;
  return r;
}

cf_status check_ptrs(std::initializer_list<const void *> ptrs) {
  for (const void *p : ptrs) {
    if (!p) return fail(CF_ERR_INVALID_ARG, "NULL tensor pointer");
    if (!aligned16(p)) return fail(CF_ERR_ALIGNMENT, "tensor pointer not 16-byte aligned");
  }
  return CF_OK;
}

}  // namespace

namespace {
// runs `call` with the fixed-order column sums recorded instead of launched
template <class F>
cf_status deferred(cf_reduction *pending, int32_t *npending, F call) {
  if (!pending || !npending) return fail(CF_ERR_INVALID_ARG, "pending / npending is NULL");
  *npending = 0;
  cf::SumCollector col{};
  cf::set_sum_collector(&col);
  const cf_status r = call();
  cf::set_sum_collector(nullptr);
  if (r != CF_OK) return r;
  for (int i = 0; i < col.n; ++i)
    pending[i] = cf_reduction{col.job[i].part, col.job[i].out, col.job[i].rows, col.job[i].cols};
  *npending = col.n;
  return CF_OK;
}
}  // namespace

namespace {
// validates the group table and fills the kernel's plan; chunks = 0 when every group is empty
cf_status adam_plan(int32_t ngroups, const int64_t *offsets, cf::OptGroups *G, int *chunks) {
  if (ngroups < 0) return fail(CF_ERR_INVALID_ARG, "adam_larc: ngroups must be >= 0");
  if (ngroups > CF_ADAM_MAX_GROUPS) return fail(CF_ERR_UNSUPPORTED, "adam_larc: more than CF_ADAM_MAX_GROUPS groups");
  if (!offsets) return fail(CF_ERR_INVALID_ARG, "adam_larc: offsets is NULL");
  if (offsets[0] < 0) return fail(CF_ERR_INVALID_ARG, "adam_larc: negative offset");
  for (int l = 0; l < ngroups; ++l) {
    if (offsets[l + 1] < offsets[l]) return fail(CF_ERR_INVALID_ARG, "adam_larc: offsets must be non-decreasing");
    if (offsets[l] % 4 != 0) return fail(CF_ERR_ALIGNMENT, "adam_larc: a group start is not a multiple of 4");
  }
  if (offsets[ngroups] >= (1LL << 40)) return fail(CF_ERR_INVALID_ARG, "adam_larc: too many elements");
  static_assert(cf::kOptMaxGroups == CF_ADAM_MAX_GROUPS, "group table size");
  std::vector<long long> off(offsets, offsets + ngroups + 1);
  *chunks = cf::plan_opt_groups(ngroups, off.data(), G);
  return CF_OK;
}
}  // namespace

extern "C" {

const char *cf_version(void) { return "cosmoflow-gfx950 0.1.0"; }

const char *cf_last_error(void) { return g_last_error.c_str(); }

cf_status cf_conv3d_out_shape(const cf_conv3d_desc *desc, int32_t out_dhw[3]) {
  cf::ConvShape s;
  cf_status r = resolve(desc, &s);
  if (r != CF_OK) return r;
  if (!out_dhw) return fail(CF_ERR_INVALID_ARG, "out_dhw is NULL");
  out_dhw[0] = s.od;
  out_dhw[1] = s.oh;
  out_dhw[2] = s.ow;
  return ok();
}

cf_status cf_conv3d_fwd(const cf_conv3d_desc *desc, const void *x, const void *w, void *z,
                        void *stream) {
  cf::ConvShape s;
  cf_status r = resolve(desc, &s);
  if (r != CF_OK) return r;
  if (s.n == 0) return ok();
  if ((r = check_ptrs({x, w, z})) != CF_OK) return r;
  Sizes b = conv_bytes(s);
  if (overlap(z, b.z, x, b.x) || overlap(z, b.z, w, b.w))
    return fail(CF_ERR_ALIAS, "conv3d_fwd: z overlaps x or W");
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_conv_fwd(s, x, w, z, st), st, "cf_conv3d_fwd");
}

// check_only: validate every argument and return without launching
static cf_status bwd_data(const cf_conv3d_desc *desc, const void *dz, const void *w, void *dx, void *stream,
                          bool check_only) {
  cf::ConvShape s;
  cf_status r = resolve(desc, &s);
  if (r != CF_OK) return r;
  if (s.n == 0) return ok();
  if ((r = check_ptrs({dz, w, dx})) != CF_OK) return r;
  Sizes b = conv_bytes(s);
  if (overlap(dx, b.x, dz, b.z) || overlap(dx, b.x, w, b.w))
    return fail(CF_ERR_ALIAS, "conv3d_bwd_data: dx overlaps dz or W");
  if (check_only) return CF_OK;
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_conv_bwd_data(s, dz, w, dx, st), st, "cf_conv3d_bwd_data");
}

cf_status cf_conv3d_bwd_data(const cf_conv3d_desc *desc, const void *dz, const void *w, void *dx,
                             void *stream) {
  return bwd_data(desc, dz, w, dx, stream, false);
}

size_t cf_conv3d_bwd_weight_workspace_size(const cf_conv3d_desc *desc) {
  cf::ConvShape s;
  std::string keep = g_last_error;
  if (resolve(desc, &s) != CF_OK) {
    g_last_error = keep;
    return 0;
  }
  if (s.n == 0) return 0;
  return cf::conv_bwd_weight_workspace(s);
}

static cf_status bwd_weight(const cf_conv3d_desc *desc, const void *x, const void *dz, float *dw, void *ws,
                            size_t ws_bytes, void *stream, bool check_only) {
  cf::ConvShape s;
  cf_status r = resolve(desc, &s);
  if (r != CF_OK) return r;
  hipStream_t st = (hipStream_t)stream;
  Sizes b = conv_bytes(s);
  const size_t dw_bytes = (size_t)s.kd * s.kh * s.kw * s.ci * s.co * sizeof(float);
  if (s.n == 0) {
    if ((r = check_ptrs({dw})) != CF_OK) return r;
    if (check_only) return CF_OK;
    // the sum over an empty batch is zero
    return finish(cf::launch_fill_zero(dw, (long long)(dw_bytes / sizeof(float)), st), st,
                  "cf_conv3d_bwd_weight");
  }
  if ((r = check_ptrs({x, dz, dw})) != CF_OK) return r;
  const size_t need = cf::conv_bwd_weight_workspace(s);
  if (need > 0 && (!ws || ws_bytes < need))
    return fail(CF_ERR_WORKSPACE, "conv3d_bwd_weight: workspace smaller than cf_conv3d_bwd_weight_workspace_size()");
  if (ws && !aligned16(ws)) return fail(CF_ERR_ALIGNMENT, "workspace not 16-byte aligned");
  if (overlap(dw, dw_bytes, x, b.x) || overlap(dw, dw_bytes, dz, b.z))
    return fail(CF_ERR_ALIAS, "conv3d_bwd_weight: dW overlaps x or dz");
  if (overlap(ws, need, x, b.x) || overlap(ws, need, dz, b.z) || overlap(ws, need, dw, dw_bytes))
    return fail(CF_ERR_ALIAS, "conv3d_bwd_weight: workspace overlaps a tensor");
  if (check_only) return CF_OK;
  return finish(cf::launch_conv_bwd_weight(s, x, dz, dw, ws, st), st, "cf_conv3d_bwd_weight");
}

cf_status cf_conv3d_bwd_weight(const cf_conv3d_desc *desc, const void *x, const void *dz, float *dw,
                               void *ws, size_t ws_bytes, void *stream) {
  return bwd_weight(desc, x, dz, dw, ws, ws_bytes, stream, false);
}

cf_status cf_conv3d_bwd(const cf_conv3d_desc *desc, const void *x, const void *dz, const void *w, float *dw,
                        void *dx, void *ws, size_t ws_bytes, void *stream) {
  cf_status r = bwd_weight(desc, x, dz, dw, ws, ws_bytes, stream, true);
  if (r != CF_OK) return r;
  if ((r = bwd_data(desc, dz, w, dx, stream, true)) != CF_OK) return r;
  cf::ConvShape s;
  resolve(desc, &s);
  if (s.n == 0) return bwd_weight(desc, x, dz, dw, ws, ws_bytes, stream, false);  // dW = 0, dx empty
  const size_t dxb = conv_bytes(s).x, dwb = (size_t)s.kd * s.kh * s.kw * s.ci * s.co * sizeof(float);
  if (overlap(dx, dxb, dw, dwb) || overlap(dx, dxb, x, conv_bytes(s).x) ||
      overlap(dx, dxb, ws, cf::conv_bwd_weight_workspace(s)))
    return fail(CF_ERR_ALIAS, "cf_conv3d_bwd: dx overlaps x, dW or the workspace");
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_conv_bwd(s, x, dz, w, dw, dx, ws, st), st, "cf_conv3d_bwd");
}

static_assert(cf::kNoallocScratchBytes == CF_NOALLOC_SCRATCH_BYTES, "scratch region size");

cf_status cf_conv3d_bwd_weight_noalloc(const cf_conv3d_desc *desc, const void *x, const void *dz, float *dw,
                                       void *stream) {
  cf::ConvShape s;
  cf_status r = resolve(desc, &s);
  if (r != CF_OK) return r;
  const size_t need = s.n == 0 ? 0 : cf::conv_bwd_weight_workspace(s);
  if (need > cf::kNoallocScratchBytes)
    return fail(CF_ERR_UNSUPPORTED, "cf_conv3d_bwd_weight_noalloc: the split reduction needs " +
                                        std::to_string(need) + " bytes of partials, more than the " +
                                        std::to_string(cf::kNoallocScratchBytes) +
                                        "-byte library scratch region (use cf_conv3d_bwd_weight with a workspace)");
  void *ws = nullptr;
  if (need > 0) {
    const hipError_t e = cf::noalloc_scratch(&ws);
    if (e != hipSuccess)
      return fail(CF_ERR_LAUNCH, std::string("cf_conv3d_bwd_weight_noalloc: scratch region: ") + hipGetErrorString(e));
  }
  return cf_conv3d_bwd_weight(desc, x, dz, dw, ws, need, stream);
}

cf_status cf_bias_lrelu_fwd(int64_t nvox, int32_t c, int32_t dtype, const void *z, const float *bias,
                            float alpha, void *y, void *stream) {
  if (nvox < 0) return fail(CF_ERR_INVALID_ARG, "nvox must be >= 0");
  if (c <= 0) return fail(CF_ERR_INVALID_ARG, "channels must be > 0");
  if (dtype != CF_F32 && dtype != CF_BF16) return fail(CF_ERR_INVALID_ARG, "unknown dtype");
  if (!std::isfinite(alpha)) return fail(CF_ERR_INVALID_ARG, "alpha must be finite");
  if (nvox == 0) return ok();
  cf_status r;
  if ((r = check_ptrs({z, y})) != CF_OK) return r;
  if (!bias) return fail(CF_ERR_INVALID_ARG, "bias is NULL");
  const size_t bytes = (size_t)nvox * c * elem_size(dtype);
  if (y != z && overlap(y, bytes, z, bytes))
    return fail(CF_ERR_ALIAS, "bias_lrelu_fwd: y partially overlaps z");
  if (overlap(y, bytes, bias, (size_t)c * 4)) return fail(CF_ERR_ALIAS, "bias_lrelu_fwd: y overlaps bias");
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_bias_lrelu_fwd(nvox, c, dtype == CF_BF16 ? cf::DT_BF16 : cf::DT_F32, z, bias,
                                          alpha, y, st),
                st, "cf_bias_lrelu_fwd");
}

size_t cf_bias_lrelu_bwd_workspace_size(int64_t nvox, int32_t c) {
  if (nvox <= 0 || c <= 0) return 0;
  return cf::bias_lrelu_bwd_workspace(nvox, c);
}

cf_status cf_bias_lrelu_bwd(int64_t nvox, int32_t c, int32_t dtype, const void *dy, const void *y,
                            float alpha, void *dz, float *db, void *ws, size_t ws_bytes,
                            void *stream) {
  if (nvox < 0) return fail(CF_ERR_INVALID_ARG, "nvox must be >= 0");
  if (c <= 0) return fail(CF_ERR_INVALID_ARG, "channels must be > 0");
  if (c > 2048) return fail(CF_ERR_UNSUPPORTED, "bias_lrelu_bwd: more than 2048 channels");
  if (dtype != CF_F32 && dtype != CF_BF16) return fail(CF_ERR_INVALID_ARG, "unknown dtype");
  if (!std::isfinite(alpha)) return fail(CF_ERR_INVALID_ARG, "alpha must be finite");
  hipStream_t st = (hipStream_t)stream;
  const int dt = dtype == CF_BF16 ? cf::DT_BF16 : cf::DT_F32;
  if (nvox == 0) {
    if (!db) return ok();
    if (!aligned16(db)) return fail(CF_ERR_ALIGNMENT, "db not 16-byte aligned");
    return finish(cf::launch_bias_lrelu_bwd(0, c, dt, nullptr, nullptr, alpha, nullptr, db, nullptr, st),
                  st, "cf_bias_lrelu_bwd");
  }
  cf_status r;
  if ((r = check_ptrs({dy, y, dz})) != CF_OK) return r;
  const size_t bytes = (size_t)nvox * c * elem_size(dtype);
  if (dz != dy && overlap(dz, bytes, dy, bytes))
    return fail(CF_ERR_ALIAS, "bias_lrelu_bwd: dz partially overlaps dy");
  if (overlap(dz, bytes, y, bytes)) return fail(CF_ERR_ALIAS, "bias_lrelu_bwd: dz overlaps y");
  if (db) {
    if (!aligned16(db)) return fail(CF_ERR_ALIGNMENT, "db not 16-byte aligned");
    const size_t need = cf::bias_lrelu_bwd_workspace(nvox, c);
    if (!ws || ws_bytes < need)
      return fail(CF_ERR_WORKSPACE, "bias_lrelu_bwd: workspace smaller than cf_bias_lrelu_bwd_workspace_size()");
    if (!aligned16(ws)) return fail(CF_ERR_ALIGNMENT, "workspace not 16-byte aligned");
    if (overlap(db, (size_t)c * 4, dz, bytes) || overlap(ws, need, dz, bytes) ||
        overlap(ws, need, dy, bytes) || overlap(ws, need, y, bytes) || overlap(ws, need, db, (size_t)c * 4))
      return fail(CF_ERR_ALIAS, "bias_lrelu_bwd: db or workspace overlaps a tensor");
  }
  return finish(cf::launch_bias_lrelu_bwd(nvox, c, dt, dy, y, alpha, dz, db, ws, st), st,
                "cf_bias_lrelu_bwd");
}

size_t cf_avgpool3d_lrelu_bwd_workspace_size(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c) {
  if (n <= 0 || d <= 0 || h <= 0 || w <= 0 || c <= 0) return 0;
  return cf::pool_lrelu_bwd_workspace((int64_t)n * d * h * w, c);
}

cf_status cf_avgpool3d_lrelu_bwd(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c, int32_t dtype,
                                 const void *dp, const void *mask, float alpha, void *dz, float *db, void *ws,
                                 size_t ws_bytes, void *stream) {
  if (n < 0) return fail(CF_ERR_INVALID_ARG, "batch n must be >= 0");
  if (d <= 0 || h <= 0 || w <= 0 || c <= 0) return fail(CF_ERR_INVALID_ARG, "extents and channels must be > 0");
  if (dtype != CF_F32 && dtype != CF_BF16) return fail(CF_ERR_INVALID_ARG, "unknown dtype");
  if (!std::isfinite(alpha) || alpha < 0.f) return fail(CF_ERR_INVALID_ARG, "alpha must be finite and >= 0");
  const int dt = dtype == CF_BF16 ? cf::DT_BF16 : cf::DT_F32;
  const int64_t nvox = (int64_t)n * d * h * w;
  if (!cf::pool_lrelu_bwd_supported(nvox, c, dt))
    return fail(CF_ERR_UNSUPPORTED, "avgpool3d_lrelu_bwd: channels must be a power-of-two multiple (at most 64) of "
                                    "the 16-byte vector, at most 256, and the tensor below 2^31 elements");
  hipStream_t st = (hipStream_t)stream;
  if (nvox == 0) {
    if (!db) return ok();
    if (!aligned16(db)) return fail(CF_ERR_ALIGNMENT, "db not 16-byte aligned");
    return finish(cf::launch_pool_lrelu_bwd(0, d, h, w, c, dt, nullptr, nullptr, alpha, nullptr, db, nullptr, st), st,
                  "cf_avgpool3d_lrelu_bwd");
  }
  cf_status r;
  if ((r = check_ptrs({dp, mask, dz})) != CF_OK) return r;
  const size_t es = elem_size(dtype);
  const size_t bz = (size_t)nvox * c * es, bp = (size_t)n * (d / 2) * (h / 2) * (w / 2) * c * es;
  const size_t bm = ((size_t)nvox * c + 31) / 32 * 4;
  if (overlap(dz, bz, dp, bp) || overlap(dz, bz, mask, bm))
    return fail(CF_ERR_ALIAS, "avgpool3d_lrelu_bwd: dz overlaps an input");
  if (db) {
    if (!aligned16(db)) return fail(CF_ERR_ALIGNMENT, "db not 16-byte aligned");
    const size_t need = cf::pool_lrelu_bwd_workspace(nvox, c);
    if (!ws || ws_bytes < need)
      return fail(CF_ERR_WORKSPACE, "avgpool3d_lrelu_bwd: workspace smaller than the size query");
    if (!aligned16(ws)) return fail(CF_ERR_ALIGNMENT, "workspace not 16-byte aligned");
    if (overlap(db, (size_t)c * 4, dz, bz) || overlap(ws, need, dz, bz) || overlap(ws, need, dp, bp) ||
        overlap(ws, need, mask, bm) || overlap(ws, need, db, (size_t)c * 4) || overlap(db, (size_t)c * 4, dp, bp) ||
        overlap(db, (size_t)c * 4, mask, bm))
      return fail(CF_ERR_ALIAS, "avgpool3d_lrelu_bwd: db or workspace overlaps a tensor");
  }
  return finish(cf::launch_pool_lrelu_bwd(n, d, h, w, c, dt, dp, mask, alpha, dz, db, ws, st), st,
                "cf_avgpool3d_lrelu_bwd");
}

static cf_status pool_check(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c, int32_t k,
                            int32_t s, int32_t dtype) {
  if (n < 0) return fail(CF_ERR_INVALID_ARG, "batch n must be >= 0");
  if (d <= 0 || h <= 0 || w <= 0 || c <= 0) return fail(CF_ERR_INVALID_ARG, "extents and channels must be > 0");
  if (k <= 0 || s <= 0) return fail(CF_ERR_INVALID_ARG, "window and stride must be > 0");
  if (dtype != CF_F32 && dtype != CF_BF16) return fail(CF_ERR_INVALID_ARG, "unknown dtype");
  if (k != s) return fail(CF_ERR_UNSUPPORTED, "avgpool3d: only non-overlapping windows (k == s)");
  if (d < k || h < k || w < k) return fail(CF_ERR_INVALID_ARG, "avgpool3d: window larger than input");
  if ((long long)n * d * h * w >= kMaxRows) return fail(CF_ERR_INVALID_ARG, "too many voxels (>= 2^31)");
  return CF_OK;
}

cf_status cf_avgpool3d_fwd(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c, int32_t k, int32_t s,
                           int32_t dtype, const void *y, void *p, void *stream) {
  cf_status r = pool_check(n, d, h, w, c, k, s, dtype);
  if (r != CF_OK) return r;
  if (n == 0) return ok();
  if ((r = check_ptrs({y, p})) != CF_OK) return r;
  const size_t es = elem_size(dtype);
  const size_t by = (size_t)n * d * h * w * c * es;
  const size_t bp = (size_t)n * ((d - k) / s + 1) * ((h - k) / s + 1) * ((w - k) / s + 1) * c * es;
  if (overlap(y, by, p, bp)) return fail(CF_ERR_ALIAS, "avgpool3d_fwd: p overlaps y");
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_avgpool_fwd(n, d, h, w, c, k, dtype == CF_BF16 ? cf::DT_BF16 : cf::DT_F32, y, p, st),
                st, "cf_avgpool3d_fwd");
}

cf_status cf_avgpool3d_bwd(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c, int32_t k, int32_t s,
                           int32_t dtype, const void *dp, void *dy, void *stream) {
  cf_status r = pool_check(n, d, h, w, c, k, s, dtype);
  if (r != CF_OK) return r;
  if (n == 0) return ok();
  if ((r = check_ptrs({dp, dy})) != CF_OK) return r;
  const size_t es = elem_size(dtype);
  const size_t by = (size_t)n * d * h * w * c * es;
  const size_t bp = (size_t)n * ((d - k) / s + 1) * ((h - k) / s + 1) * ((w - k) / s + 1) * c * es;
  if (overlap(dy, by, dp, bp)) return fail(CF_ERR_ALIAS, "avgpool3d_bwd: dy overlaps dp");
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_avgpool_bwd(n, d, h, w, c, k, dtype == CF_BF16 ? cf::DT_BF16 : cf::DT_F32, dp, dy, st),
                st, "cf_avgpool3d_bwd");
}

// ---------------------------------------------------------------------------
// Fused layer variants
// ---------------------------------------------------------------------------

static int32_t fused_mask(const cf::ConvShape &s, uint32_t flags) {
  int32_t m = 0;
  if (flags & ~(CF_FUSE_POOL2 | CF_FUSE_MASK)) return 0;
  // the mask flag only asks the forward for the mask; with the pool it is implied
  const bool ymode = flags == 0;  // unpooled backward from (dy, y)
  if (flags & CF_FUSE_POOL2) flags = CF_FUSE_POOL2;
  if (flags == CF_FUSE_POOL2) {
    if (cf::smallc_supported(s, true)) m |= 1;
    if (cf::smallc_wgrad_fused_supported(s) || cf::c16_wgrad_supported(s)) m |= 2;
  }
  if (cf::c16_fwd_supported(s)) m |= 1;  // with or without the pool
  if ((flags == 0 || flags == CF_FUSE_MASK) && (cf::direct_supported(s, true) || cf::f32conv_supported(s, true)))
    m |= 1;
  if (ymode && cf::f32wgrad_supported(s)) m |= 2 | 8;
  if (ymode && cf::f32conv_supported(s, false)) m |= 4;
  if (flags == CF_FUSE_POOL2 && cf::f32conv_pool_supported(s)) m |= 1;
  if (flags == CF_FUSE_POOL2 && cf::c16_bwd_supported(s)) m |= 4;
  if (flags == CF_FUSE_POOL2 && cf::c16_wgrad_supported(s) && !cf::smallc_wgrad_fused_supported(s)) m |= 8;
  if (flags == CF_FUSE_POOL2 && cf::f32wgrad_fused_supported(s) && !cf::smallc_wgrad_fused_supported(s)) m |= 2 | 8;
  // bf16 deep layers: pooled forward, and both backward kernels forming dz from
  // (pooled gradient, mask) or (dy, y) as they load it (no dz output)
  if (flags == CF_FUSE_POOL2 && cf::direct_pool_supported(s)) m |= 1;
  if ((flags == CF_FUSE_POOL2 || ymode) && s.dtype == cf::DT_BF16 && cf::direct_wgrad_supported(s)) m |= 2;
  if ((flags == CF_FUSE_POOL2 || ymode) && cf::direct_supported(s, false)) m |= 4;
  return m;
}

int32_t cf_conv3d_fused_supported(const cf_conv3d_desc *desc, uint32_t flags) {
  cf::ConvShape s;
  std::string keep = g_last_error;
  if (resolve(desc, &s) != CF_OK) {
    g_last_error = keep;
    return 0;
  }
  return fused_mask(s, flags);
}

static size_t mask_bytes(const cf::ConvShape &s) {
  const size_t bits = (size_t)s.n * s.od * s.oh * s.ow * s.co;
  return (bits + 31) / 32 * 4;
}

static size_t fused_wgrad_workspace(const cf::ConvShape &s, uint32_t flags) {
  const bool deep16 = s.dtype == cf::DT_BF16 && cf::direct_wgrad_supported(s);
  if (!(flags & CF_FUSE_POOL2))  // (dy, y)
    return deep16 ? cf::direct_wgrad_workspace(s, true) : cf::f32wgrad_workspace(s, 3);
  if (cf::smallc_wgrad_fused_supported(s)) return cf::smallc_wgrad_fused_workspace(s);
  if (cf::f32wgrad_fused_supported(s)) return cf::f32wgrad_workspace(s, 1);
  if (deep16) return cf::direct_wgrad_workspace(s, true);
  return cf::c16_wgrad_workspace(s);
}

// bytes of the 2^3 stride-2 pooled conv output (floor extents)
static size_t pooled_bytes(const cf::ConvShape &s) {
  const size_t es = s.dtype == cf::DT_BF16 ? 2 : 4;
  return (size_t)s.n * (s.od / 2) * (s.oh / 2) * (s.ow / 2) * s.co * es;
}

size_t cf_conv3d_mask_bytes(const cf_conv3d_desc *desc) {
  cf::ConvShape s;
  std::string keep = g_last_error;
  if (resolve(desc, &s) != CF_OK) {
    g_last_error = keep;
    return 0;
  }
  return mask_bytes(s);
}

cf_status cf_conv3d_fwd_fused(const cf_conv3d_desc *desc, const void *x, const void *w, const float *bias,
                              float alpha, uint32_t flags, void *out, void *mask, void *stream) {
  cf::ConvShape s;
  cf_status r = resolve(desc, &s);
  if (r != CF_OK) return r;
  if (!std::isfinite(alpha) || alpha < 0.f) return fail(CF_ERR_INVALID_ARG, "alpha must be finite and >= 0");
  if (flags & ~(CF_FUSE_POOL2 | CF_FUSE_MASK)) return fail(CF_ERR_INVALID_ARG, "unknown flags");
  if (!(fused_mask(s, flags) & 1))
    return fail(CF_ERR_UNSUPPORTED, "conv3d_fwd_fused: no fused kernel for this layer shape / flags");
  if (s.n == 0) return ok();
  const bool pool = (flags & CF_FUSE_POOL2) != 0;
  if ((r = check_ptrs({x, w, out})) != CF_OK) return r;
  if (pool && !mask) return fail(CF_ERR_INVALID_ARG, "conv3d_fwd_fused: the pooled variant needs the mask");
  if ((flags & CF_FUSE_MASK) && !mask) return fail(CF_ERR_INVALID_ARG, "conv3d_fwd_fused: CF_FUSE_MASK needs the mask");
  if (mask && !aligned16(mask)) return fail(CF_ERR_ALIGNMENT, "mask not 16-byte aligned");
  if (!bias) return fail(CF_ERR_INVALID_ARG, "bias is NULL");
  Sizes b = conv_bytes(s);
  const size_t ob = pool ? pooled_bytes(s) : b.z;
  const size_t mb = mask_bytes(s);
  if (overlap(out, ob, x, b.x) || overlap(out, ob, w, b.w) || overlap(mask, mb, x, b.x) ||
      overlap(mask, mb, w, b.w) || overlap(mask, mb, out, ob) || overlap(bias, (size_t)s.co * 4, out, ob) ||
      overlap(bias, (size_t)s.co * 4, mask, mb))
    return fail(CF_ERR_ALIAS, "conv3d_fwd_fused: an output overlaps an input");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e;
  if (pool && cf::l1pair_supported(s))
    e = cf::launch_l1pair_fwd(s, x, w, bias, alpha, out, (uint16_t *)mask, st);
  else if (pool && cf::smallc_supported(s, true))
    e = cf::launch_conv_fwd_smallc(s, x, w, bias, alpha, out, (uint16_t *)mask, true, st);
  else if (cf::f32conv_supported(s, true) && !cf::c16_fwd_supported(s))
    e = cf::launch_conv_fwd_f32(s, (const float *)x, (const float *)w, bias, alpha, (float *)out, (uint8_t *)mask,
                                pool ? 2 : 1, st);
  else if (!pool && !cf::c16_fwd_supported(s))
    e = cf::launch_conv_fwd_direct(s, x, w, bias, alpha, out, mask, true, st);
  else if (pool && cf::direct_pool_supported(s))
    e = cf::launch_conv_fwd_direct_pool(s, x, w, bias, alpha, out, mask, st);
  else
    e = cf::launch_conv_fwd_c16(s, x, w, bias, alpha, out, (uint32_t *)mask, pool ? 2 : 1, st);
  return finish(e, st, "cf_conv3d_fwd_fused");
}

size_t cf_conv3d_bwd_weight_fused_workspace_size(const cf_conv3d_desc *desc, uint32_t flags) {
  cf::ConvShape s;
  std::string keep = g_last_error;
  if (resolve(desc, &s) != CF_OK || !(fused_mask(s, flags) & 2) || s.n == 0) {
    g_last_error = keep;
    return 0;
  }
  return fused_wgrad_workspace(s, flags);
}

// check_only: validate every argument and return without launching
static cf_status bwd_weight_fused(const char *name, const cf_conv3d_desc *desc, const void *x, const void *g,
                                  const void *mask, float alpha, uint32_t flags, float *dw, float *db, void *dz,
                                  void *ws, size_t ws_bytes, void *stream, bool check_only = false) {
  cf::ConvShape s;
  cf_status r = resolve(desc, &s);
  if (r != CF_OK) return r;
  if (!std::isfinite(alpha) || alpha < 0.f) return fail(CF_ERR_INVALID_ARG, "alpha must be finite and >= 0");
  if (flags & ~(CF_FUSE_POOL2 | CF_FUSE_MASK)) return fail(CF_ERR_INVALID_ARG, "unknown flags");
  if (!(fused_mask(s, flags) & (dz ? 8 : 2)))
    return fail(CF_ERR_UNSUPPORTED, std::string(name) + ": no fused kernel for this layer shape / flags");
  const bool pool = (flags & CF_FUSE_POOL2) != 0;
  hipStream_t st = (hipStream_t)stream;
  const size_t dw_bytes = (size_t)s.kd * s.kh * s.kw * s.ci * s.co * sizeof(float);
  if (s.n == 0) {
    if ((r = check_ptrs({dw, db})) != CF_OK) return r;
    if (check_only) return CF_OK;
    hipError_t e = cf::launch_fill_zero(dw, (long long)(dw_bytes / 4), st);
    if (e == hipSuccess) e = cf::launch_fill_zero(db, s.co, st);
    return finish(e, st, name);
  }
  if ((r = check_ptrs({x, g, mask, dw, db})) != CF_OK) return r;
  if (dz && (r = check_ptrs({dz})) != CF_OK) return r;
  const size_t need = fused_wgrad_workspace(s, flags);
  if (!ws || ws_bytes < need) return fail(CF_ERR_WORKSPACE, std::string(name) + ": workspace smaller than the size query");
  if (!aligned16(ws)) return fail(CF_ERR_ALIGNMENT, "workspace not 16-byte aligned");
  Sizes b = conv_bytes(s);
  // pooled: g = pooled-output gradient, mask = slope mask; else g = dy, mask = y
  const size_t gb = pool ? pooled_bytes(s) : b.z, mb = pool ? mask_bytes(s) : b.z, dbb = (size_t)s.co * 4;
  const void *ins[3] = {x, g, mask};
  const size_t insz[3] = {b.x, gb, mb};
  for (int i = 0; i < 3; ++i)
    if (overlap(dw, dw_bytes, ins[i], insz[i]) || overlap(db, dbb, ins[i], insz[i]) ||
        overlap(ws, need, ins[i], insz[i]) || (dz && overlap(dz, b.z, ins[i], insz[i])))
      return fail(CF_ERR_ALIAS, std::string(name) + ": an output or the workspace overlaps an input");
  if (overlap(dw, dw_bytes, db, dbb) || overlap(ws, need, dw, dw_bytes) || overlap(ws, need, db, dbb))
    return fail(CF_ERR_ALIAS, std::string(name) + ": outputs / workspace overlap");
  if (dz && (overlap(dz, b.z, dw, dw_bytes) || overlap(dz, b.z, db, dbb) || overlap(dz, b.z, ws, need)))
    return fail(CF_ERR_ALIAS, std::string(name) + ": dz overlaps another output or the workspace");
  if (check_only) return CF_OK;
  hipError_t e;
  const bool deep16 = s.dtype == cf::DT_BF16 && cf::direct_wgrad_supported(s);
  if (!pool && deep16)
    e = cf::launch_conv_bwd_weight_direct(s, x, g, mask, cf::DWG_DYY, alpha, dw, db, ws, st);
  else if (!pool)
    e = cf::launch_conv_bwd_weight_f32(s, (const float *)x, (const float *)g, mask, alpha, dw, db, ws, 3, (float *)dz,
                                       st);
  else if (cf::smallc_wgrad_fused_supported(s))
    e = cf::launch_smallc_wgrad_fused(s, x, g, (const uint16_t *)mask, alpha, dw, db, ws, st);
  else if (cf::f32wgrad_fused_supported(s))
    e = cf::launch_conv_bwd_weight_f32(s, (const float *)x, (const float *)g, mask, alpha, dw, db, ws, 1, (float *)dz,
                                       st);
  else if (deep16)
    e = cf::launch_conv_bwd_weight_direct(s, x, g, mask, cf::DWG_POOL, alpha, dw, db, ws, st);
  else
    e = cf::launch_conv_bwd_weight_c16(s, x, g, (const uint32_t *)mask, alpha, dw, db, ws, true, dz, st);
  return finish(e, st, name);
}

cf_status cf_conv3d_bwd_weight_fused(const cf_conv3d_desc *desc, const void *x, const void *g, const void *mask,
                                     float alpha, uint32_t flags, float *dw, float *db, void *ws, size_t ws_bytes,
                                     void *stream) {
  return bwd_weight_fused("cf_conv3d_bwd_weight_fused", desc, x, g, mask, alpha, flags, dw, db, nullptr, ws,
                          ws_bytes, stream);
}

cf_status cf_conv3d_bwd_weight_fused_dz(const cf_conv3d_desc *desc, const void *x, const void *g, const void *mask,
                                        float alpha, uint32_t flags, float *dw, float *db, void *dz, void *ws,
                                        size_t ws_bytes, void *stream) {
  if (!dz && desc && desc->n > 0) return fail(CF_ERR_INVALID_ARG, "cf_conv3d_bwd_weight_fused_dz: dz is NULL");
  return bwd_weight_fused("cf_conv3d_bwd_weight_fused_dz", desc, x, g, mask, alpha, flags, dw, db, dz, ws,
                          ws_bytes, stream);
}

static cf_status bwd_data_fused(const cf_conv3d_desc *desc, const void *g, const void *mask, const void *w,
                                float alpha, uint32_t flags, void *dx, void *stream, bool check_only) {
  cf::ConvShape s;
  cf_status r = resolve(desc, &s);
  if (r != CF_OK) return r;
  if (!std::isfinite(alpha) || alpha < 0.f) return fail(CF_ERR_INVALID_ARG, "alpha must be finite and >= 0");
  if (flags & ~(CF_FUSE_POOL2 | CF_FUSE_MASK)) return fail(CF_ERR_INVALID_ARG, "unknown flags");
  if (!(fused_mask(s, flags) & 4))
    return fail(CF_ERR_UNSUPPORTED, "conv3d_bwd_data_fused: no fused kernel for this layer shape / flags");
  if (s.n == 0) return ok();
  if ((r = check_ptrs({g, mask, w, dx})) != CF_OK) return r;
  Sizes b = conv_bytes(s);
  const bool pool = (flags & CF_FUSE_POOL2) != 0;
  const size_t gb = pool ? pooled_bytes(s) : b.z, mb = pool ? mask_bytes(s) : b.z;
  if (overlap(dx, b.x, g, gb) || overlap(dx, b.x, mask, mb) || overlap(dx, b.x, w, b.w))
    return fail(CF_ERR_ALIAS, "conv3d_bwd_data_fused: dx overlaps an input");
  if (check_only) return CF_OK;
  hipStream_t st = (hipStream_t)stream;
  hipError_t e;
  if (pool && cf::c16_bwd_supported(s))
    e = cf::launch_conv_bwd_data_c16(s, g, (const uint32_t *)mask, w, alpha, dx, true, st);
  else if (cf::direct_supported(s, false))  // bf16 deep layers
    e = cf::launch_conv_bwd_data_direct_fused(s, g, mask, pool ? cf::DWG_POOL : cf::DWG_DYY, alpha, w, dx, st);
  else
    e = cf::launch_conv_bwd_data_f32(s, (const float *)g, (const float *)w, (float *)dx, st, (const float *)mask,
                                     alpha);
  return finish(e, st, "cf_conv3d_bwd_data_fused");
}

cf_status cf_conv3d_bwd_data_fused(const cf_conv3d_desc *desc, const void *g, const void *mask, const void *w,
                                   float alpha, uint32_t flags, void *dx, void *stream) {
  return bwd_data_fused(desc, g, mask, w, alpha, flags, dx, stream, false);
}

cf_status cf_conv3d_bwd_fused(const cf_conv3d_desc *desc, const void *x, const void *g, const void *mask,
                              const void *w, float alpha, uint32_t flags, float *dw, float *db, void *dx, void *ws,
                              size_t ws_bytes, void *stream) {
  const char *name = "cf_conv3d_bwd_fused";
  cf_status r = bwd_weight_fused(name, desc, x, g, mask, alpha, flags, dw, db, nullptr, ws, ws_bytes, stream, true);
  if (r != CF_OK) return r;
  if ((r = bwd_data_fused(desc, g, mask, w, alpha, flags, dx, stream, true)) != CF_OK) return r;
  cf::ConvShape s;
  resolve(desc, &s);
  if (s.n > 0) {
    const size_t dxb = conv_bytes(s).x, dwb = (size_t)s.kd * s.kh * s.kw * s.ci * s.co * sizeof(float);
    if (overlap(dx, dxb, dw, dwb) || overlap(dx, dxb, db, (size_t)s.co * 4) ||
        overlap(dx, dxb, ws, fused_wgrad_workspace(s, flags)))
      return fail(CF_ERR_ALIAS, "cf_conv3d_bwd_fused: dx overlaps dW, db or the workspace");
  }
  // fp32 unpooled layers: both products from (dy, y) in one launch where the
  // kernels allow; everything else is the two calls in sequence
  if (s.n > 0 && s.dtype == cf::DT_F32 && !(flags & CF_FUSE_POOL2)) {
    hipStream_t st = (hipStream_t)stream;
    return finish(cf::launch_conv_bwd_fused_f32(s, (const float *)x, (const float *)g, (const float *)mask,
                                                (const float *)w, alpha, dw, db, (float *)dx, ws, st),
                  st, name);
  }
  if ((r = bwd_weight_fused(name, desc, x, g, mask, alpha, flags, dw, db, nullptr, ws, ws_bytes, stream)) != CF_OK)
    return r;
  return bwd_data_fused(desc, g, mask, w, alpha, flags, dx, stream, false);
}

// ---------------------------------------------------------------------------
// Deferred gradient sums
// ---------------------------------------------------------------------------


cf_status cf_reduce_partials(int32_t n, const cf_reduction *jobs, void *stream) {
  if (n < 0) return fail(CF_ERR_INVALID_ARG, "n must be >= 0");
  if (n == 0) return ok();
  if (!jobs) return fail(CF_ERR_INVALID_ARG, "jobs is NULL");
  std::vector<cf::SumJob> v;
  v.reserve(n);
  for (int32_t i = 0; i < n; ++i) {
    const cf_reduction &j = jobs[i];
    if (j.rows < 0 || j.cols < 0) return fail(CF_ERR_INVALID_ARG, "reduction with negative rows or cols");
    if (j.cols == 0) continue;
    if (!j.out || (j.rows > 0 && !j.part)) return fail(CF_ERR_INVALID_ARG, "reduction with a NULL pointer");
    if (((uintptr_t)j.out & 3) || ((uintptr_t)j.part & 3))
      return fail(CF_ERR_ALIGNMENT, "reduction pointers must be 4-byte aligned");
    if (overlap(j.out, (size_t)j.cols * 4, j.part, (size_t)j.rows * j.cols * 4))
      return fail(CF_ERR_ALIAS, "reduction output overlaps its partials");
    v.push_back(cf::SumJob{j.part, j.out, j.rows, j.cols});
  }
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_sum_batch(v.data(), (int)v.size(), st), st, "cf_reduce_partials");
}

cf_status cf_conv3d_bwd_weight_deferred(const cf_conv3d_desc *desc, const void *x, const void *dz, float *dw,
                                        void *ws, size_t ws_bytes, cf_reduction *pending, int32_t *npending,
                                        void *stream) {
  return deferred(pending, npending, [&] { return cf_conv3d_bwd_weight(desc, x, dz, dw, ws, ws_bytes, stream); });
}

cf_status cf_bias_lrelu_bwd_deferred(int64_t nvox, int32_t c, int32_t dtype, const void *dy, const void *y,
                                     float alpha, void *dz, float *db, void *ws, size_t ws_bytes,
                                     cf_reduction *pending, int32_t *npending, void *stream) {
  return deferred(pending, npending, [&] {
    return cf_bias_lrelu_bwd(nvox, c, dtype, dy, y, alpha, dz, db, ws, ws_bytes, stream);
  });
}

cf_status cf_avgpool3d_lrelu_bwd_deferred(int32_t n, int32_t d, int32_t h, int32_t w, int32_t c, int32_t dtype,
                                          const void *dp, const void *mask, float alpha, void *dz, float *db,
                                          void *ws, size_t ws_bytes, cf_reduction *pending, int32_t *npending,
                                          void *stream) {
  return deferred(pending, npending, [&] {
    return cf_avgpool3d_lrelu_bwd(n, d, h, w, c, dtype, dp, mask, alpha, dz, db, ws, ws_bytes, stream);
  });
}

cf_status cf_conv3d_bwd_weight_fused_deferred(const cf_conv3d_desc *desc, const void *x, const void *g,
                                              const void *mask, float alpha, uint32_t flags, float *dw, float *db,
                                              void *dz, void *ws, size_t ws_bytes, cf_reduction *pending,
                                              int32_t *npending, void *stream) {
  return deferred(pending, npending, [&] {
    return bwd_weight_fused(dz ? "cf_conv3d_bwd_weight_fused_dz" : "cf_conv3d_bwd_weight_fused", desc, x, g, mask,
                            alpha, flags, dw, db, dz, ws, ws_bytes, stream);
  });
}

cf_status cf_conv3d_bwd_deferred(const cf_conv3d_desc *desc, const void *x, const void *dz, const void *w,
                                 float *dw, void *dx, void *ws, size_t ws_bytes, cf_reduction *pending,
                                 int32_t *npending, void *stream) {
  return deferred(pending, npending, [&] { return cf_conv3d_bwd(desc, x, dz, w, dw, dx, ws, ws_bytes, stream); });
}

cf_status cf_conv3d_bwd_fused_deferred(const cf_conv3d_desc *desc, const void *x, const void *g, const void *mask,
                                       const void *w, float alpha, uint32_t flags, float *dw, float *db, void *dx,
                                       void *ws, size_t ws_bytes, cf_reduction *pending, int32_t *npending,
                                       void *stream) {
  return deferred(pending, npending, [&] {
    return cf_conv3d_bwd_fused(desc, x, g, mask, w, alpha, flags, dw, db, dx, ws, ws_bytes, stream);
  });
}


size_t cf_adam_larc_workspace_size(int32_t ngroups, const int64_t *offsets) {
  std::string keep = g_last_error;
  cf::OptGroups G;
  int chunks = 0;
  if (adam_plan(ngroups, offsets, &G, &chunks) != CF_OK) {
    g_last_error = keep;
    return 0;
  }
  return (size_t)chunks * 2 * sizeof(double);
}

cf_status cf_adam_larc_step(int32_t ngroups, const int64_t *offsets, int64_t t, const cf_adam_larc_hparams *hp,
                            float *v, const float *g, float *m, float *s, void *v16, void *ws, size_t ws_bytes,
                            void *stream) {
  cf::OptGroups G;
  int chunks = 0;
  cf_status r = adam_plan(ngroups, offsets, &G, &chunks);
  if (r != CF_OK) return r;
  if (!hp) return fail(CF_ERR_INVALID_ARG, "adam_larc: hp is NULL");
  if (t < 0) return fail(CF_ERR_INVALID_ARG, "adam_larc: t must be >= 0");
  if (hp->t_decay <= 0) return fail(CF_ERR_INVALID_ARG, "adam_larc: t_decay must be > 0");
  const double vals[] = {hp->eta0, hp->eta_min, hp->beta1, hp->beta2, hp->eps_hat,
                         hp->larc_coef, hp->larc_fallback, hp->larc_clip};
  for (double x : vals)
    if (!std::isfinite(x)) return fail(CF_ERR_INVALID_ARG, "adam_larc: hyperparameters must be finite");
  if (hp->beta1 < 0.0 || hp->beta1 >= 1.0 || hp->beta2 < 0.0 || hp->beta2 >= 1.0)
    return fail(CF_ERR_INVALID_ARG, "adam_larc: beta1 and beta2 must lie in [0, 1)");
  if (hp->eps_hat < 0.0) return fail(CF_ERR_INVALID_ARG, "adam_larc: eps_hat must be >= 0");
  if (chunks == 0) return ok();
  if ((r = check_ptrs({v, g, m, s})) != CF_OK) return r;
  if (v16 && !aligned16(v16)) return fail(CF_ERR_ALIGNMENT, "adam_larc: v16 not 16-byte aligned");
  const size_t need = (size_t)chunks * 2 * sizeof(double);
  if (!ws || ws_bytes < need)
    return fail(CF_ERR_WORKSPACE, "adam_larc: workspace smaller than cf_adam_larc_workspace_size()");
  if (!aligned16(ws)) return fail(CF_ERR_ALIGNMENT, "workspace not 16-byte aligned");
  const size_t nb = (size_t)offsets[ngroups] * 4;
  const void *bufs[] = {v, g, m, s, v16, ws};
  const size_t lens[] = {nb, nb, nb, nb, nb / 2, need};
  for (int a = 0; a < 6; ++a)
    for (int b = a + 1; b < 6; ++b)
      if (overlap(bufs[a], lens[a], bufs[b], lens[b]))
        return fail(CF_ERR_ALIAS, "adam_larc: v, g, m, s, v16 and the workspace must not overlap");
  cf::OptHparams h{hp->eta0,  hp->eta_min,   hp->t_decay,       hp->beta1,    hp->beta2,
                   hp->eps_hat, hp->larc_coef, hp->larc_fallback, hp->larc_clip};
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_adam_larc(G, chunks, h, (long long)t, v, g, m, s, (uint16_t *)v16, (double *)ws, st),
                st, "cf_adam_larc_step");
}

}  // extern "C"

// ---- fully-connected head and loss -------------------------------------------

namespace {
cf_status fc_check(int32_t m, int32_t k, int32_t n, int32_t dtype, const char *who) {
  if (m < 0) return fail(CF_ERR_INVALID_ARG, std::string(who) + ": m must be >= 0");
  if (k <= 0 || n <= 0) return fail(CF_ERR_INVALID_ARG, std::string(who) + ": k and n must be > 0");
  if (n > 65536) return fail(CF_ERR_UNSUPPORTED, std::string(who) + ": more than 65536 outputs");
  if ((long long)k * n >= (1LL << 40)) return fail(CF_ERR_UNSUPPORTED, std::string(who) + ": k * n too large");
  if (dtype != CF_F32 && dtype != CF_BF16) return fail(CF_ERR_INVALID_ARG, "unknown dtype");
  return CF_OK;
}
int kdt(int32_t dtype) { return dtype == CF_BF16 ? cf::DT_BF16 : cf::DT_F32; }
}  // namespace

size_t cf_fc_fwd_workspace_size(int32_t m, int32_t k, int32_t n) {
  if (m <= 0 || k <= 0 || n <= 0 || n > 65536 || (long long)k * n >= (1LL << 40)) return 0;
  return cf::fc_fwd_workspace(m, k, n);
}

cf_status cf_fc_fwd(int32_t m, int32_t k, int32_t n, int32_t dtype, const void *x, const void *w, void *z,
                    void *ws, size_t ws_bytes, void *stream) {
  cf_status r = fc_check(m, k, n, dtype, "fc_fwd");
  if (r != CF_OK) return r;
  if (m == 0) return ok();
  if ((r = check_ptrs({x, w, z})) != CF_OK) return r;
  const size_t es = elem_size(dtype);
  const size_t bx = (size_t)m * k * es, bw = (size_t)k * n * es, bz = (size_t)m * n * es;
  const size_t need = cf::fc_fwd_workspace(m, k, n);
  if (!ws || ws_bytes < need) return fail(CF_ERR_WORKSPACE, "fc_fwd: workspace smaller than cf_fc_fwd_workspace_size()");
  if (!aligned16(ws)) return fail(CF_ERR_ALIGNMENT, "workspace not 16-byte aligned");
  if (overlap(z, bz, x, bx) || overlap(z, bz, w, bw)) return fail(CF_ERR_ALIAS, "fc_fwd: z overlaps x or W");
  if (overlap(ws, need, x, bx) || overlap(ws, need, w, bw) || overlap(ws, need, z, bz))
    return fail(CF_ERR_ALIAS, "fc_fwd: workspace overlaps a tensor");
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_fc_fwd(m, k, n, kdt(dtype), x, w, z, ws, st), st, "cf_fc_fwd");
}

cf_status cf_fc_bwd_data(int32_t m, int32_t k, int32_t n, int32_t dtype, const void *dz, const void *w, void *dx,
                         void *stream) {
  cf_status r = fc_check(m, k, n, dtype, "fc_bwd_data");
  if (r != CF_OK) return r;
  if (m == 0) return ok();
  if ((r = check_ptrs({dz, w, dx})) != CF_OK) return r;
  const size_t es = elem_size(dtype);
  const size_t bx = (size_t)m * k * es, bw = (size_t)k * n * es, bz = (size_t)m * n * es;
  if (overlap(dx, bx, dz, bz) || overlap(dx, bx, w, bw)) return fail(CF_ERR_ALIAS, "fc_bwd_data: dx overlaps dz or W");
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_fc_bwd_data(m, k, n, kdt(dtype), dz, w, dx, st), st, "cf_fc_bwd_data");
}

cf_status cf_fc_bwd_weight(int32_t m, int32_t k, int32_t n, int32_t dtype, const void *x, const void *dz, float *dw,
                           void *stream) {
  cf_status r = fc_check(m, k, n, dtype, "fc_bwd_weight");
  if (r != CF_OK) return r;
  hipStream_t st = (hipStream_t)stream;
  if (m == 0) {
    if ((r = check_ptrs({dw})) != CF_OK) return r;
    return finish(cf::launch_fill_zero(dw, (long long)k * n, st), st, "cf_fc_bwd_weight");
  }
  if ((r = check_ptrs({x, dz, dw})) != CF_OK) return r;
  const size_t es = elem_size(dtype);
  const size_t bx = (size_t)m * k * es, bz = (size_t)m * n * es, bw = (size_t)k * n * 4;
  if (overlap(dw, bw, x, bx) || overlap(dw, bw, dz, bz)) return fail(CF_ERR_ALIAS, "fc_bwd_weight: dW overlaps x or dz");
  return finish(cf::launch_fc_bwd_weight(m, k, n, kdt(dtype), x, dz, dw, st), st, "cf_fc_bwd_weight");
}

size_t cf_fc_head_workspace_size(int32_t m, int32_t nlayers, const int32_t *dims) {
  if (!dims || nlayers < 2 || nlayers > 4 || m < 1) return 0;
  int d[5];
  for (int i = 0; i <= nlayers; ++i) {
    if (dims[i] < 1) return 0;
    d[i] = dims[i];
  }
  return cf::fc_head_workspace(m, nlayers, d);
}

cf_status cf_fc_head(int32_t m, int32_t nlayers, const int32_t *dims, int32_t dtype, const void *x,
                     const void *const *w, const float *const *b, float alpha, const float *target, void *const *y,
                     void *const *dz, void *const *dx, float *const *dw, float *const *db, float *loss, void *ws,
                     size_t ws_bytes, void *stream) {
  if (dtype != CF_F32 && dtype != CF_BF16) return fail(CF_ERR_INVALID_ARG, "unknown dtype");
  if (!dims || !w || !b || !y || !dz || !dx || !dw || !db)
    return fail(CF_ERR_INVALID_ARG, "fc_head: NULL dims or pointer array");
  if (nlayers < 2 || nlayers > 4) return fail(CF_ERR_UNSUPPORTED, "fc_head: 2 to 4 layers");
  if (m < 1 || m > 8) return fail(CF_ERR_UNSUPPORTED, "fc_head: 1 to 8 batch rows");
  int d[5];
  for (int i = 0; i <= nlayers; ++i) {
    if (dims[i] < 1) return fail(CF_ERR_INVALID_ARG, "fc_head: every width must be > 0");
    d[i] = dims[i];
  }
  if (!cf::fc_head_supported(m, nlayers, d, kdt(dtype)))
    return fail(CF_ERR_UNSUPPORTED, "fc_head: widths outside the fused head's limits (see cf_fc_head)");
  cf_status r;
  if ((r = check_ptrs({x, target, loss, ws})) != CF_OK) return r;
  const size_t es = elem_size(dtype);
  // (pointer, bytes) of every input and every output
  std::vector<std::pair<const void *, size_t>> in, out;
  in.push_back({x, (size_t)m * d[0] * es});
  in.push_back({target, (size_t)m * d[nlayers] * 4});
  for (int i = 0; i < nlayers; ++i) {
    if ((r = check_ptrs({w[i], b[i], y[i], dz[i], dx[i], dw[i], db[i]})) != CF_OK) return r;
    const size_t kn = (size_t)d[i] * d[i + 1];
    in.push_back({w[i], kn * es});
    in.push_back({b[i], (size_t)d[i + 1] * 4});
    out.push_back({y[i], (size_t)m * d[i + 1] * es});
    out.push_back({dz[i], (size_t)m * d[i + 1] * es});
    out.push_back({dx[i], (size_t)m * d[i] * es});
    out.push_back({dw[i], kn * 4});
    out.push_back({db[i], (size_t)d[i + 1] * 4});
  }
  out.push_back({loss, 4});
  const size_t need = cf::fc_head_workspace(m, nlayers, d);
  if (ws_bytes < need) return fail(CF_ERR_WORKSPACE, "fc_head: workspace smaller than cf_fc_head_workspace_size()");
  out.push_back({ws, need});
  for (size_t i = 0; i < out.size(); ++i) {
    for (const auto &t : in)
      if (overlap(out[i].first, out[i].second, t.first, t.second))
        return fail(CF_ERR_ALIAS, "fc_head: an output or the workspace overlaps an input");
    for (size_t j = i + 1; j < out.size(); ++j)
      if (overlap(out[i].first, out[i].second, out[j].first, out[j].second))
        return fail(CF_ERR_ALIAS, "fc_head: two outputs overlap");
  }
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_fc_head(m, nlayers, d, kdt(dtype), x, w, b, alpha, target, y, dz, dx, dw, db, loss, ws, st),
                st, "cf_fc_head");
}

cf_status cf_mse_loss(int32_t m, int32_t n, int32_t dtype, const void *p, const float *t, float *loss, void *dp,
                      void *stream) {
  if (m <= 0 || n <= 0) return fail(CF_ERR_INVALID_ARG, "mse_loss: m and n must be > 0");
  if ((long long)m * n >= (1LL << 31)) return fail(CF_ERR_UNSUPPORTED, "mse_loss: m * n too large");
  if (dtype != CF_F32 && dtype != CF_BF16) return fail(CF_ERR_INVALID_ARG, "unknown dtype");
  cf_status r;
  if ((r = check_ptrs({p, t, loss})) != CF_OK) return r;
  if (dp && !aligned16(dp)) return fail(CF_ERR_ALIGNMENT, "dp not 16-byte aligned");
  const long long cnt = (long long)m * n;
  const size_t es = elem_size(dtype);
  if (overlap(loss, 4, p, cnt * es) || overlap(loss, 4, t, cnt * 4) || overlap(loss, 4, dp, dp ? cnt * es : 0))
    return fail(CF_ERR_ALIAS, "mse_loss: loss overlaps a tensor");
  if (dp && (overlap(dp, cnt * es, p, cnt * es) || overlap(dp, cnt * es, t, cnt * 4)))
    return fail(CF_ERR_ALIAS, "mse_loss: dp overlaps p or t");
  hipStream_t st = (hipStream_t)stream;
  return finish(cf::launch_mse_loss(cnt, kdt(dtype), p, t, loss, dp, (float)(1.0 / (double)cnt), st), st,
                "cf_mse_loss");
}
