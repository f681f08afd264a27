/*
 * cfref.c -- the CPU oracle for the CosmoFlow 3D-convolution hot path.
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke
 * check and the CPU-baseline leg of the benchmark may load this library.
 * It shares no code, header, table or helper with the GPU library.
 *
 * Everything is computed in IEEE double precision with plain nested loops in
 * the order of the definitions below; there is no blocking, no fusion and no
 * reordering of any sum.  OpenMP is used only to spread *independent* output
 * elements over threads, so each output is one fixed-order sum and the result
 * does not depend on the thread count.
 *
 * Layouts (the only convention the caller must know):
 *   activations  NDHWC   x[n][d][h][w][c]
 *   weights      DHWIO   W[kd][kh][kw][ci][co]
 *
 * Definitions followed (CosmoFlow, arXiv:1808.04728):
 *   - forward convolution: Section III-C, Algorithm 1 and the paragraph after
 *     it.  Each output is an inner product over the kernel taps (kd,kh,kw)
 *     and the input channels; the source voxel of tap k for output o is
 *     o*stride + k - pad_before, i.e. a cross-correlation without kernel
 *     flip (the algorithm indexes SRC[od + kd]).  The update in the
 *     innermost loop of Algorithm 1 is an accumulation into a zeroed DST
 *     (it sums over input-channel blocks and taps); the printed arrow is read
 *     as "+=".  Stride and zero padding generalise the algorithm's
 *     stride-one, unpadded statement in the standard way.
 *   - backward data / backward weights: Section III-C, the paragraphs after
 *     Algorithm 1.  Backward data propagates the output difference signal to
 *     the input; backward weights produces the weight difference signal.
 *     Both are the exact derivatives (adjoints) of the forward map.
 *   - average pooling: Section III-C, last paragraph -- a per-channel
 *     convolution whose weights are all 1/KS^3; Section III-A gives the
 *     stride (2,2,2).
 *   - leaky ReLU: Section III-A, used after every convolution layer.  The
 *     slope for negative inputs (alpha) is a parameter; the derivative at
 *     exactly zero is taken as alpha (the saved output y is <= 0 there).
 *   - bias: not described by the paper; y = lrelu(z + b[c]) with a
 *     per-output-channel bias, db[c] = sum over voxels of dz.
 *   - parameter update: Section III-B ("SGD Optimizer"): Adam on a gradient
 *     rescaled per layer by LARC's clipped local rate, with a global rate on
 *     a linear (power 1) decay.  See ref_adam_larc_step for the readings.
 *   - fully-connected layers: Section III-A (three FC layers after the
 *     convolutions, leaky ReLU on every one, three outputs for the three
 *     cosmological parameters).  A layer maps a row x[m][0..K) to
 *     z[m][j] = sum_k x[m][k] W[k][j] (W stored [K][N], input index major);
 *     its backward maps are the exact adjoints.  The widths of the first two
 *     layers are in Fig. 2, which the text lacks: they are parameters here.
 *   - loss: not named by the paper.  Read as the mean squared error of the
 *     three regressed parameters over the batch,
 *     L = (1 / (M N)) sum_{m,j} (p[m][j] - t[m][j])^2, dL/dp = 2 (p - t) / (M N).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#define IDX5(n, d, h, w, c, D, H, W, C) \
  (((((int64_t)(n) * (D) + (d)) * (H) + (h)) * (W) + (w)) * (C) + (c))
#define WIDX(a, b, e, ci, co, KH, KW, CI, CO) \
  (((((int64_t)(a) * (KH) + (b)) * (KW) + (e)) * (CI) + (ci)) * (CO) + (co))

/* ---------------------------------------------------------------------- */
/* Geometry                                                                 */
/* ---------------------------------------------------------------------- */

/*
 * Output extent and padding of one spatial dimension.
 *   same != 0 : TensorFlow "SAME" rule (the paper's framework is TensorFlow,
 *               Section IV-D): out = ceil(in / s), total padding
 *               max((out-1)*s + k - in, 0), the smaller half before.
 *   same == 0 : "VALID": out = floor((in - k) / s) + 1, no padding.
 * Returns 0 on success, -1 if the kernel does not fit.
 */
int ref_conv_geometry(int in, int k, int s, int same, int *out, int *pad_before) {
  if (in <= 0 || k <= 0 || s <= 0) return -1;
  if (same) {
    int o = (in + s - 1) / s;
    int tot = (o - 1) * s + k - in;
    if (tot < 0) tot = 0;
    *out = o;
    *pad_before = tot / 2;
  } else {
    if (k > in) return -1;
    *out = (in - k) / s + 1;
    *pad_before = 0;
  }
  return 0;
}

/* ---------------------------------------------------------------------- */
/* Convolution (Section III-C, Algorithm 1)                                 */
/* ---------------------------------------------------------------------- */

/*
 * DST[n,od,oh,ow,co] = sum_{kd,kh,kw,ci} W[kd,kh,kw,ci,co] *
 *                      SRC[n, od*sd+kd-pd, oh*sh+kh-ph, ow*sw+kw-pw, ci]
 * with SRC taken as zero outside its extent.
 */
void ref_conv3d_fwd(const double *src, const double *wt, double *dst,
                    int N, int D, int H, int W, int CI, int CO,
                    int KD, int KH, int KW, int sd, int sh, int sw,
                    int pd, int ph, int pw, int OD, int OH, int OW) {
  int64_t total = (int64_t)N * OD * OH * OW;
#pragma omp parallel for schedule(static)
  for (int64_t v = 0; v < total; ++v) {
    int ow = (int)(v % OW);
    int oh = (int)((v / OW) % OH);
    int od = (int)((v / ((int64_t)OW * OH)) % OD);
    int n = (int)(v / ((int64_t)OW * OH * OD));
    for (int co = 0; co < CO; ++co) {
      double acc = 0.0;
      for (int kd = 0; kd < KD; ++kd) {
        int id = od * sd + kd - pd;
        if (id < 0 || id >= D) continue;
        for (int kh = 0; kh < KH; ++kh) {
          int ih = oh * sh + kh - ph;
          if (ih < 0 || ih >= H) continue;
          for (int kw = 0; kw < KW; ++kw) {
            int iw = ow * sw + kw - pw;
            if (iw < 0 || iw >= W) continue;
            for (int ci = 0; ci < CI; ++ci)
              acc += wt[WIDX(kd, kh, kw, ci, co, KH, KW, CI, CO)] *
                     src[IDX5(n, id, ih, iw, ci, D, H, W, CI)];
          }
        }
      }
      dst[IDX5(n, od, oh, ow, co, OD, OH, OW, CO)] = acc;
    }
  }
}

/*
 * Backward data: the adjoint of ref_conv3d_fwd with respect to SRC.
 * dSRC[n,i,ci] = sum over every (output voxel o, tap k) whose source voxel
 * o*s + k - p equals i (per dimension), of sum_co dDST[n,o,co]*W[k,ci,co].
 * Written as a gather: for each tap k, o = (i + p - k) / s must be an
 * integer inside the output extent.
 */
void ref_conv3d_bwd_data(const double *ddst, const double *wt, double *dsrc,
                         int N, int D, int H, int W, int CI, int CO,
                         int KD, int KH, int KW, int sd, int sh, int sw,
                         int pd, int ph, int pw, int OD, int OH, int OW) {
  int64_t total = (int64_t)N * D * H * W;
#pragma omp parallel for schedule(static)
  for (int64_t v = 0; v < total; ++v) {
    int iw = (int)(v % W);
    int ih = (int)((v / W) % H);
    int id = (int)((v / ((int64_t)W * H)) % D);
    int n = (int)(v / ((int64_t)W * H * D));
    for (int ci = 0; ci < CI; ++ci) {
      double acc = 0.0;
      for (int kd = 0; kd < KD; ++kd) {
        int td = id + pd - kd;
        if (td < 0 || td % sd != 0 || td / sd >= OD) continue;
        int od = td / sd;
        for (int kh = 0; kh < KH; ++kh) {
          int th = ih + ph - kh;
          if (th < 0 || th % sh != 0 || th / sh >= OH) continue;
          int oh = th / sh;
          for (int kw = 0; kw < KW; ++kw) {
            int tw = iw + pw - kw;
            if (tw < 0 || tw % sw != 0 || tw / sw >= OW) continue;
            int ow = tw / sw;
            for (int co = 0; co < CO; ++co)
              acc += ddst[IDX5(n, od, oh, ow, co, OD, OH, OW, CO)] *
                     wt[WIDX(kd, kh, kw, ci, co, KH, KW, CI, CO)];
          }
        }
      }
      dsrc[IDX5(n, id, ih, iw, ci, D, H, W, CI)] = acc;
    }
  }
}

/*
 * Backward weights: the adjoint of ref_conv3d_fwd with respect to W.
 * dW[k,ci,co] = sum_{n,o} SRC[n, o*s + k - p, ci] * dDST[n,o,co]
 * (zero where the source voxel lies in the padding).
 */
void ref_conv3d_bwd_weight(const double *src, const double *ddst, double *dwt,
                           int N, int D, int H, int W, int CI, int CO,
                           int KD, int KH, int KW, int sd, int sh, int sw,
                           int pd, int ph, int pw, int OD, int OH, int OW) {
  int64_t total = (int64_t)KD * KH * KW * CI;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < total; ++r) {
    int ci = (int)(r % CI);
    int kw = (int)((r / CI) % KW);
    int kh = (int)((r / ((int64_t)CI * KW)) % KH);
    int kd = (int)(r / ((int64_t)CI * KW * KH));
    for (int co = 0; co < CO; ++co) {
      double acc = 0.0;
      for (int n = 0; n < N; ++n)
        for (int od = 0; od < OD; ++od) {
          int id = od * sd + kd - pd;
          if (id < 0 || id >= D) continue;
          for (int oh = 0; oh < OH; ++oh) {
            int ih = oh * sh + kh - ph;
            if (ih < 0 || ih >= H) continue;
            for (int ow = 0; ow < OW; ++ow) {
              int iw = ow * sw + kw - pw;
              if (iw < 0 || iw >= W) continue;
              acc += src[IDX5(n, id, ih, iw, ci, D, H, W, CI)] *
                     ddst[IDX5(n, od, oh, ow, co, OD, OH, OW, CO)];
            }
          }
        }
      dwt[WIDX(kd, kh, kw, ci, co, KH, KW, CI, CO)] = acc;
    }
  }
}

/* Single-element evaluators, for sampled checks of full-size tensors.     */

double ref_conv3d_fwd_point(const double *src, const double *wt,
                            int D, int H, int W, int CI, int CO,
                            int KD, int KH, int KW, int sd, int sh, int sw,
                            int pd, int ph, int pw,
                            int n, int od, int oh, int ow, int co) {
  double acc = 0.0;
  for (int kd = 0; kd < KD; ++kd) {
    int id = od * sd + kd - pd;
    if (id < 0 || id >= D) continue;
    for (int kh = 0; kh < KH; ++kh) {
      int ih = oh * sh + kh - ph;
      if (ih < 0 || ih >= H) continue;
      for (int kw = 0; kw < KW; ++kw) {
        int iw = ow * sw + kw - pw;
        if (iw < 0 || iw >= W) continue;
        for (int ci = 0; ci < CI; ++ci)
          acc += wt[WIDX(kd, kh, kw, ci, co, KH, KW, CI, CO)] *
                 src[IDX5(n, id, ih, iw, ci, D, H, W, CI)];
      }
    }
  }
  return acc;
}

double ref_conv3d_bwd_data_point(const double *ddst, const double *wt,
                                 int D, int H, int W, int CI, int CO,
                                 int KD, int KH, int KW, int sd, int sh, int sw,
                                 int pd, int ph, int pw, int OD, int OH, int OW,
                                 int n, int id, int ih, int iw, int ci) {
  (void)D; (void)H; (void)W;
  double acc = 0.0;
  for (int kd = 0; kd < KD; ++kd) {
    int td = id + pd - kd;
    if (td < 0 || td % sd != 0 || td / sd >= OD) continue;
    for (int kh = 0; kh < KH; ++kh) {
      int th = ih + ph - kh;
      if (th < 0 || th % sh != 0 || th / sh >= OH) continue;
      for (int kw = 0; kw < KW; ++kw) {
        int tw = iw + pw - kw;
        if (tw < 0 || tw % sw != 0 || tw / sw >= OW) continue;
        for (int co = 0; co < CO; ++co)
          acc += ddst[IDX5(n, td / sd, th / sh, tw / sw, co, OD, OH, OW, CO)] *
                 wt[WIDX(kd, kh, kw, ci, co, KH, KW, CI, CO)];
      }
    }
  }
  return acc;
}

double ref_conv3d_bwd_weight_point(const double *src, const double *ddst,
                                   int N, int D, int H, int W, int CI, int CO,
                                   int KD, int KH, int KW, int sd, int sh, int sw,
                                   int pd, int ph, int pw, int OD, int OH, int OW,
                                   int kd, int kh, int kw, int ci, int co) {
  (void)KD;
  (void)KH;
  (void)KW;
  double acc = 0.0;
  for (int n = 0; n < N; ++n)
    for (int od = 0; od < OD; ++od) {
      int id = od * sd + kd - pd;
      if (id < 0 || id >= D) continue;
      for (int oh = 0; oh < OH; ++oh) {
        int ih = oh * sh + kh - ph;
        if (ih < 0 || ih >= H) continue;
        for (int ow = 0; ow < OW; ++ow) {
          int iw = ow * sw + kw - pw;
          if (iw < 0 || iw >= W) continue;
          acc += src[IDX5(n, id, ih, iw, ci, D, H, W, CI)] *
                 ddst[IDX5(n, od, oh, ow, co, OD, OH, OW, CO)];
        }
      }
    }
  return acc;
}

/* ---------------------------------------------------------------------- */
/* Bias + leaky ReLU (Section III-A)                                        */
/* ---------------------------------------------------------------------- */

/* y[v,c] = u if u > 0 else alpha*u, with u = z[v,c] + b[c]. */
void ref_bias_lrelu_fwd(const double *z, const double *b, double alpha,
                        double *y, int64_t nvox, int C) {
#pragma omp parallel for schedule(static)
  for (int64_t v = 0; v < nvox; ++v)
    for (int c = 0; c < C; ++c) {
      double u = z[v * C + c] + b[c];
      y[v * C + c] = u > 0.0 ? u : alpha * u;
    }
}

/*
 * dz[v,c] = dy[v,c] * (y[v,c] > 0 ? 1 : alpha);  db[c] = sum_v dz[v,c].
 * The slope is read from the saved output y: for alpha > 0, y > 0 exactly
 * when the pre-activation is > 0.
 */
void ref_bias_lrelu_bwd(const double *dy, const double *y, double alpha,
                        double *dz, double *db, int64_t nvox, int C) {
#pragma omp parallel for schedule(static)
  for (int64_t v = 0; v < nvox; ++v)
    for (int c = 0; c < C; ++c)
      dz[v * C + c] = dy[v * C + c] * (y[v * C + c] > 0.0 ? 1.0 : alpha);
  for (int c = 0; c < C; ++c) {
    double acc = 0.0;
    for (int64_t v = 0; v < nvox; ++v) acc += dz[v * C + c];
    db[c] = acc;
  }
}

/* ---------------------------------------------------------------------- */
/* Average pooling (Section III-C: a per-channel convolution with constant   */
/* weights 1/KS^3; window KS, stride S, outputs floor((in - KS)/S) + 1)      */
/* ---------------------------------------------------------------------- */

void ref_avgpool3d_fwd(const double *y, double *p, int N, int D, int H, int W,
                       int C, int KS, int S) {
  int OD = (D - KS) / S + 1, OH = (H - KS) / S + 1, OW = (W - KS) / S + 1;
  double wgt = 1.0 / ((double)KS * KS * KS);
  int64_t total = (int64_t)N * OD * OH * OW;
#pragma omp parallel for schedule(static)
  for (int64_t v = 0; v < total; ++v) {
    int ow = (int)(v % OW);
    int oh = (int)((v / OW) % OH);
    int od = (int)((v / ((int64_t)OW * OH)) % OD);
    int n = (int)(v / ((int64_t)OW * OH * OD));
    for (int c = 0; c < C; ++c) {
      double acc = 0.0;
      for (int a = 0; a < KS; ++a)
        for (int b = 0; b < KS; ++b)
          for (int e = 0; e < KS; ++e)
            acc += wgt * y[IDX5(n, od * S + a, oh * S + b, ow * S + e, c, D, H, W, C)];
      p[IDX5(n, od, oh, ow, c, OD, OH, OW, C)] = acc;
    }
  }
}

/* Adjoint of ref_avgpool3d_fwd: dy[i] = sum over windows covering i of dp/KS^3. */
void ref_avgpool3d_bwd(const double *dp, double *dy, int N, int D, int H, int W,
                       int C, int KS, int S) {
  int OD = (D - KS) / S + 1, OH = (H - KS) / S + 1, OW = (W - KS) / S + 1;
  double wgt = 1.0 / ((double)KS * KS * KS);
  int64_t total = (int64_t)N * D * H * W;
#pragma omp parallel for schedule(static)
  for (int64_t v = 0; v < total; ++v) {
    int iw = (int)(v % W);
    int ih = (int)((v / W) % H);
    int id = (int)((v / ((int64_t)W * H)) % D);
    int n = (int)(v / ((int64_t)W * H * D));
    for (int c = 0; c < C; ++c) {
      double acc = 0.0;
      for (int a = 0; a < KS; ++a) {
        int td = id - a;
        if (td < 0 || td % S != 0 || td / S >= OD) continue;
        for (int b = 0; b < KS; ++b) {
          int th = ih - b;
          if (th < 0 || th % S != 0 || th / S >= OH) continue;
          for (int e = 0; e < KS; ++e) {
            int tw = iw - e;
            if (tw < 0 || tw % S != 0 || tw / S >= OW) continue;
            acc += wgt * dp[IDX5(n, td / S, th / S, tw / S, c, OD, OH, OW, C)];
          }
        }
      }
      dy[IDX5(n, id, ih, iw, c, D, H, W, C)] = acc;
    }
  }
}

/* ---------------------------------------------------------------------- */
/* Parameter update (Section III-B, "SGD Optimizer")                        */
/* ---------------------------------------------------------------------- */

/*
 * Global learning rate of step t: linear decay from eta0 at t = 0 to eta_min
 * at t = t_decay (the schedule equation of Section III-B, power 1).  The
 * paper does not say what follows t_decay; the rate stays at eta_min (t is
 * clamped), as in TensorFlow's non-cycling polynomial decay.
 */
double ref_lr_schedule(int64_t t, int64_t t_decay, double eta0, double eta_min) {
  const double tc = (double)(t < t_decay ? t : t_decay);
  return (eta0 - eta_min) * (1.0 - tc / (double)t_decay) + eta_min;
}

/*
 * One update of every parameter group (Section III-B equations, in order):
 *   1. eta_t = ref_lr_schedule(t)                            global rate
 *   2. vn = ||v_l||_2, gn = ||g_l||_2                        per group l
 *   3. eta*  = coef * vn / gn if vn != 0 and gn != 0, else fallback
 *   4. eta+  = min(eta*, clip)                               clipped local rate
 *   5. g*    = eta+ * g_l
 *   6. v_l   = Adam(v_l, g*, eta_t)
 * The paper's constants are coef = 0.002, fallback = 6.25e-5, clip = 1,
 * beta1 = 0.9, beta2 = 0.999, eps_hat = 1e-8, eta0 = 2e-3, eta_min = 1e-4.
 *
 * Adam is Kingma and Ba's method in the form the paper's epsilon-hat names
 * (their Section 2, the reformulation at its end; TensorFlow's Adam, which
 * the paper trains with, implements this form): the moments are updated
 *   m = beta1 m + (1 - beta1) g*,   s = beta2 s + (1 - beta2) g*^2,
 * and the step is v -= a_k m / (sqrt(s) + eps_hat) with
 *   a_k = eta_t sqrt(1 - beta2^k) / (1 - beta1^k),
 * where k = t + 1 counts updates from 1 (Adam's bias corrections), while the
 * decay counts them from t = 0 (the first update uses eta0).
 *
 * A group is one parameter tensor (a layer's weights, or its biases): the
 * paper speaks of the parameters "in a layer" without saying whether a
 * layer's weights and biases share one norm; the caller chooses by how it
 * lays out the groups.  Group l holds elements [off[l], off[l+1]) of
 * v, g, m, s.  hp = {eta0, eta_min, beta1, beta2, eps_hat, coef, fallback,
 * clip}.  eta_dag (may be NULL) receives eta+ of every group.
 */
void ref_adam_larc_step(int ngroups, const int64_t *off, int64_t t, int64_t t_decay,
                        const double *hp, double *v, const double *g, double *m,
                        double *s, double *eta_dag) {
  const double eta0 = hp[0], eta_min = hp[1], beta1 = hp[2], beta2 = hp[3];
  const double eps_hat = hp[4], coef = hp[5], fallback = hp[6], clip = hp[7];
  /* 1. */
  const double eta_t = ref_lr_schedule(t, t_decay, eta0, eta_min);
  const double k = (double)(t + 1);
  const double a_k = eta_t * sqrt(1.0 - pow(beta2, k)) / (1.0 - pow(beta1, k));
  for (int l = 0; l < ngroups; ++l) {
    /* 2. */
    double vv = 0.0, gg = 0.0;
    for (int64_t i = off[l]; i < off[l + 1]; ++i) {
      vv += v[i] * v[i];
      gg += g[i] * g[i];
    }
    const double vn = sqrt(vv), gn = sqrt(gg);
    /* 3. and 4. */
    const double star = (vn != 0.0 && gn != 0.0) ? coef * vn / gn : fallback;
    const double dag = star < clip ? star : clip;
    if (eta_dag) eta_dag[l] = dag;
    /* 5. and 6. */
    for (int64_t i = off[l]; i < off[l + 1]; ++i) {
      const double gs = dag * g[i];
      m[i] = beta1 * m[i] + (1.0 - beta1) * gs;
      s[i] = beta2 * s[i] + (1.0 - beta2) * gs * gs;
      v[i] = v[i] - a_k * m[i] / (sqrt(s[i]) + eps_hat);
    }
  }
}

/* ------------------------------------------------------------------------
 * Fully-connected layers (Section III-A) and the loss.
 * x: [M][K] rows (for the first layer, one sample's NDHWC output flattened
 * in memory order), W: [K][N], z / dz: [M][N].
 * ------------------------------------------------------------------------ */

/* z[m][j] = sum over k = 0 .. K-1 (in order) of x[m][k] W[k][j] */
void ref_fc_fwd(const double *x, const double *wt, double *z, int M, int K, int N) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int m = 0; m < M; ++m)
    for (int j = 0; j < N; ++j) {
      double s = 0.0;
      for (int k = 0; k < K; ++k) s += x[(int64_t)m * K + k] * wt[(int64_t)k * N + j];
      z[(int64_t)m * N + j] = s;
    }
}

/* dx[m][k] = sum over j (in order) of dz[m][j] W[k][j]  (adjoint in x) */
void ref_fc_bwd_data(const double *dz, const double *wt, double *dx, int M, int K, int N) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int m = 0; m < M; ++m)
    for (int k = 0; k < K; ++k) {
      double s = 0.0;
      for (int j = 0; j < N; ++j) s += dz[(int64_t)m * N + j] * wt[(int64_t)k * N + j];
      dx[(int64_t)m * K + k] = s;
    }
}

/* dW[k][j] = sum over m (in order) of x[m][k] dz[m][j]  (adjoint in W) */
void ref_fc_bwd_weight(const double *x, const double *dz, double *dw, int M, int K, int N) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int k = 0; k < K; ++k)
    for (int j = 0; j < N; ++j) {
      double s = 0.0;
      for (int m = 0; m < M; ++m) s += x[(int64_t)m * K + k] * dz[(int64_t)m * N + j];
      dw[(int64_t)k * N + j] = s;
    }
}

/* mean squared error over the M x N predictions; dp = dL/dp.  Returns L. */
double ref_mse_loss(const double *p, const double *t, double *dp, int M, int N) {
  const double inv = 1.0 / ((double)M * (double)N);
  double s = 0.0;
  for (int64_t i = 0; i < (int64_t)M * N; ++i) {
    const double e = p[i] - t[i];
    s += e * e;
    dp[i] = 2.0 * e * inv;
  }
  return s * inv;
}
