// fc.hip -- fully-connected layers and the loss for gfx950.
//
// Section III-A: after the convolutions the network has three
// fully-connected layers, each followed by leaky ReLU (applied by the
// bias + leaky ReLU kernels of eltwise.hip), the last with the three outputs
// that regress the cosmological parameters.  A layer maps rows x[m][0..K)
// to z[m][j] = sum_k x[m][k] W[k][j], W stored [K][N] (input index major).
// With a batch of a few rows every pass is bound by reading W (or writing
// dW) once from HBM, so the kernels below stream W with 16-byte loads over
// the whole machine and keep the few batch rows in registers and LDS; no
// pass is recast as a GEMM tile for the matrix cores.
//   forward        split over K: workgroup b sums rows [b KC, (b+1) KC) of
//                  W for all M x N outputs (its phases combined in LDS in
//                  phase order), one partial row per workgroup, then a
//                  fixed-order column sum of the partials rounded once;
//   backward data  one group of G lanes per row k of W: each lane dots its
//                  columns with dz, a lane butterfly completes the row;
//   backward wts   one thread per (k, 4 columns) of dW: sum over the batch
//                  rows in order (the reduction is only M long);
//   loss           mean squared error, one workgroup, fixed-order tree.
// Every sum has an order fixed by the shapes, so results are deterministic.

#include "cf_common.h"
#include "cf_kernels.h"

#include <algorithm>

namespace cf {
namespace {

constexpr int MB = 8;  // batch rows per pass (larger batches take several passes)
constexpr int MH = 4;  // batch rows per LDS round of the forward's phase combine

// ---- forward ------------------------------------------------------------
// Thread t: column group cg = t % cgw (+ cgw, 2 cgw, ... while < cg_n),
// phase t / cgw of np phases; rows k0 + phase + np * u, u < U.
template <int DT, bool VECTOR>
__global__ __launch_bounds__(256) void fc_fwd_kernel(const typename Store<DT>::T *__restrict__ x,
                                                     const typename Store<DT>::T *__restrict__ w,
                                                     float *__restrict__ part, int m0, int mcnt, int K, int N,
                                                     int cgw, int np, int kc) {
  constexpr int V = VECTOR ? Store<DT>::VEC : 1;
  __shared__ float xs[MB * 512];  // x[m0 + m][k0 + kk], kc <= 512
  __shared__ float red[256 * MH * V];  // [phase][batch row][column of the pass] (np * cgw <= 256)
  const int tid = threadIdx.x;
  const int cg_n = N / V;
  const long long k0 = (long long)blockIdx.x * kc;
  const int krows = (int)std::min<long long>(kc, K - k0);
  for (int i = tid; i < MB * kc; i += 256) {
    const int m = i / kc, kk = i - m * kc;
    xs[i] = (m < mcnt && kk < krows) ? to_f32<DT>(x[(long long)(m0 + m) * K + k0 + kk]) : 0.f;
  }
  __syncthreads();
  const int ph = tid / cgw, c_in = tid - ph * cgw;
  float *prow = part + (long long)blockIdx.x * mcnt * N;  // this workgroup's partial row [mcnt][N]
  for (int cbase = 0; cbase < cg_n; cbase += cgw) {
    const int cg = cbase + c_in;
    const bool active = ph < np && cg < cg_n;
    float acc[MB][V];
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
      for (int j = 0; j < V; ++j) acc[m][j] = 0.f;
    if (active) {
#pragma unroll 8
      for (int kk = ph; kk < krows; kk += np) {
        const typename Store<DT>::T *wr = w + (k0 + kk) * N + (long long)cg * V;
        float wv[V];
        if constexpr (VECTOR) {
          Vec16<DT> v;
          v.u = ld16<false>(wr);
#pragma unroll
          for (int j = 0; j < V; ++j) wv[j] = to_f32<DT>(v.e[j]);
        } else {
          wv[0] = to_f32<DT>(wr[0]);
        }
#pragma unroll
        for (int m = 0; m < MB; ++m) {
          const float xv = xs[m * kc + kk];
#pragma unroll
          for (int j = 0; j < V; ++j) acc[m][j] = fmaf(xv, wv[j], acc[m][j]);
        }
      }
    }
    // combine the phases in phase order, MH batch rows at a time: every (row,
    // column) sum reads its np partials with eight loads in flight and adds
    // them in order
    const int ncols = std::min(cgw, cg_n - cbase) * V;
    const int rs = cgw * V;  // LDS row stride
#pragma unroll
    for (int h0 = 0; h0 < MB; h0 += MH) {
      if (h0 >= mcnt) break;
      if (active)
#pragma unroll
        for (int m = 0; m < MH; ++m)
#pragma unroll
          for (int j = 0; j < V; ++j) red[(ph * MH + m) * rs + c_in * V + j] = acc[h0 + m][j];
      __syncthreads();
      const int hc = std::min(MH, mcnt - h0);
      for (int q = tid; q < hc * ncols; q += 256) {
        const int m = q / ncols, col = q - m * ncols;
        const float *r = red + m * rs + col;
        float s = 0.f;
        int p = 0;
        for (; p + 8 <= np; p += 8) {
          float v[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) v[u] = r[(p + u) * MH * rs];
#pragma unroll
          for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; p < np; ++p) s += r[p * MH * rs];
        prow[(h0 + m) * N + cbase * V + col] = s;
      }
      __syncthreads();
    }
  }
}

// y[m0 + i] = RNE(sum over the rows of the partial matrix [rows][cols]):
// 16 columns per workgroup, 16 row phases per column (phase p sums rows p,
// p + 16, ... in order, eight loads in flight), phases combined in order.
// BIAS_ACT: then y = lrelu(y + bias[col % n]) rounded again, as the per-layer
// bias + leaky ReLU call does on the stored z.
template <int DT, bool BIAS_ACT = false>
__global__ __launch_bounds__(256) void fc_finalize_kernel(const float *__restrict__ part, int rows, int cols,
                                                          typename Store<DT>::T *y, const float *__restrict__ bias = nullptr,
                                                          int n = 1, float alpha = 0.f) {
  __shared__ float red[16][16];
  const int tid = threadIdx.x, cl = tid & 15, ph = tid >> 4;
  const int col = (int)blockIdx.x * 16 + cl;
  float s = 0.f;
  if (col < cols) {
    int r = ph;
    for (; r + 7 * 16 < rows; r += 8 * 16) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = part[(long long)(r + 16 * u) * cols + col];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; r < rows; r += 16) s += part[(long long)r * cols + col];
  }
  red[ph][cl] = s;
  __syncthreads();
  if (ph == 0 && col < cols) {
    float t = 0.f;
#pragma unroll
    for (int p = 0; p < 16; ++p) t += red[p][cl];
    if constexpr (BIAS_ACT) {
      const float u = to_f32<DT>(from_f32<DT>(t)) + bias[col % n];
      y[col] = from_f32<DT>(u > 0.f ? u : alpha * u);
    } else {
      y[col] = from_f32<DT>(t);
    }
  }
}

struct FwdPlan {
  int cgw, np, kc, blocks;
  bool vec;
};

FwdPlan plan_fwd(int K, int N, int V) {
  FwdPlan p{};
  p.vec = N % V == 0;
  const int cg_n = p.vec ? N / V : N;
  p.cgw = std::min(cg_n, 256);
  p.np = 256 / p.cgw;
  // about 512 workgroups, at most 512 rows each
  const long long target = ((long long)K + 511) / 512;
  long long u = std::max<long long>(1, (target + p.np - 1) / p.np);
  long long kc = std::min<long long>(u * p.np, 512);
  p.kc = (int)kc;
  p.blocks = (int)(((long long)K + kc - 1) / kc);
  return p;
}

template <int DT>
hipError_t fc_fwd_t(int M, int K, int N, const void *x, const void *w, void *y, void *ws, hipStream_t st) {
  using T = typename Store<DT>::T;
  const FwdPlan pl = plan_fwd(K, N, Store<DT>::VEC);
  float *part = (float *)ws;
  for (int m0 = 0; m0 < M; m0 += MB) {
    const int mcnt = std::min(MB, M - m0);
    if (pl.vec)
      hipLaunchKernelGGL((fc_fwd_kernel<DT, true>), dim3(pl.blocks), dim3(256), 0, st, (const T *)x, (const T *)w,
                         part, m0, mcnt, K, N, pl.cgw, pl.np, pl.kc);
    else
      hipLaunchKernelGGL((fc_fwd_kernel<DT, false>), dim3(pl.blocks), dim3(256), 0, st, (const T *)x, (const T *)w,
                         part, m0, mcnt, K, N, pl.cgw, pl.np, pl.kc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((fc_finalize_kernel<DT>), dim3((mcnt * N + 15) / 16), dim3(256), 0, st, part, pl.blocks,
                       mcnt * N, (T *)y + (size_t)m0 * N);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// ---- backward data --------------------------------------------------------
// G lanes per row (a power of two, G >= the column groups when they fit one
// wave); 256 / G rows per workgroup step.  When every lane owns at most one
// column group (RESIDENT), its dz values for all batch rows are loaded once
// and stay in registers across the rows it visits.
template <int DT, bool VECTOR, bool RESIDENT>
__global__ __launch_bounds__(256) void fc_bwd_data_kernel(const typename Store<DT>::T *__restrict__ dz,
                                                          const typename Store<DT>::T *__restrict__ w,
                                                          typename Store<DT>::T *__restrict__ dx, int m0, int mcnt,
                                                          int K, int N, int G) {
  constexpr int V = VECTOR ? Store<DT>::VEC : 1;
  const int tid = threadIdx.x;
  const int cg_n = N / V;
  const int gl = tid & (G - 1), rows_per = 256 / G;
  // one batch row's dz for this lane's column group
  auto load_dz = [&](int m, int cg, float *d) {
    const typename Store<DT>::T *dr = dz + (long long)(m0 + m) * N + (long long)cg * V;
    if constexpr (VECTOR) {
      Vec16<DT> g;
      g.u = ld16<false>(dr);
#pragma unroll
      for (int j = 0; j < V; ++j) d[j] = to_f32<DT>(g.e[j]);
    } else {
      d[0] = to_f32<DT>(dr[0]);
    }
  };
  auto load_w = [&](long long k, int cg, float *wv) {
    if constexpr (VECTOR) {
      Vec16<DT> v;
      v.u = ld16<false>(w + k * N + (long long)cg * V);
#pragma unroll
      for (int j = 0; j < V; ++j) wv[j] = to_f32<DT>(v.e[j]);
    } else {
      wv[0] = to_f32<DT>(w[k * N + cg]);
    }
  };
  float dzr[RESIDENT ? MB : 1][V];
  if constexpr (RESIDENT) {
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      if (m < mcnt && gl < cg_n) {
        load_dz(m, gl, dzr[m]);
      } else {
#pragma unroll
        for (int j = 0; j < V; ++j) dzr[m][j] = 0.f;
      }
    }
  }
  const long long kstep = (long long)gridDim.x * rows_per;
  long long k = (long long)blockIdx.x * rows_per + tid / G;
  if constexpr (RESIDENT) {
    // four rows per iteration, their W loads issued together
    for (; k + 3 * kstep < K; k += 4 * kstep) {
      float wv[4][V];
      if (gl < cg_n)
#pragma unroll
        for (int u = 0; u < 4; ++u) load_w(k + u * kstep, gl, wv[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        float acc[MB];
#pragma unroll
        for (int m = 0; m < MB; ++m) acc[m] = 0.f;
        if (gl < cg_n)
#pragma unroll
          for (int m = 0; m < MB; ++m)
#pragma unroll
            for (int j = 0; j < V; ++j) acc[m] = fmaf(dzr[m][j], wv[u][j], acc[m]);
        for (int off = G >> 1; off > 0; off >>= 1)
#pragma unroll
          for (int m = 0; m < MB; ++m) acc[m] += __shfl_xor(acc[m], off, 64);
#pragma unroll
        for (int m = 0; m < MB; ++m)
          if (m < mcnt && gl == m % G) dx[(long long)(m0 + m) * K + k + u * kstep] = from_f32<DT>(acc[m]);
      }
    }
  }
  for (; k < K; k += kstep) {
    float acc[MB];
#pragma unroll
    for (int m = 0; m < MB; ++m) acc[m] = 0.f;
    if constexpr (RESIDENT) {
      if (gl < cg_n) {
        float wv[V];
        load_w(k, gl, wv);
#pragma unroll
        for (int m = 0; m < MB; ++m)
#pragma unroll
          for (int j = 0; j < V; ++j) acc[m] = fmaf(dzr[m][j], wv[j], acc[m]);
      }
    } else {
      for (int cg = gl; cg < cg_n; cg += G) {
        float wv[V];
        load_w(k, cg, wv);
#pragma unroll
        for (int m = 0; m < MB; ++m) {
          if (m < mcnt) {
            float d[V];
            load_dz(m, cg, d);
#pragma unroll
            for (int j = 0; j < V; ++j) acc[m] = fmaf(d[j], wv[j], acc[m]);
          }
        }
      }
    }
    // butterfly over the G lanes of the row: every lane ends with the same sums
    for (int off = G >> 1; off > 0; off >>= 1)
#pragma unroll
      for (int m = 0; m < MB; ++m) acc[m] += __shfl_xor(acc[m], off, 64);
#pragma unroll
    for (int m = 0; m < MB; ++m)
      if (m < mcnt && gl == m % G) dx[(long long)(m0 + m) * K + k] = from_f32<DT>(acc[m]);
  }
}

template <int DT>
hipError_t fc_bwd_data_t(int M, int K, int N, const void *dz, const void *w, void *dx, hipStream_t st) {
  using T = typename Store<DT>::T;
  const bool vec = N % Store<DT>::VEC == 0;
  const int cg_n = vec ? N / Store<DT>::VEC : N;
  int G = 1;
  while (G < cg_n && G < 64) G <<= 1;
  const bool res = cg_n <= G;
  const int rows_per = 256 / G;
  // one row per thread for short matrices; about four per thread for long
  // ones when dz is register-resident
  const long long want = ((long long)K + rows_per - 1) / rows_per;
  const int blocks = (int)std::min<long long>(res ? std::max(std::min<long long>(want, 1024), (want + 3) / 4) : want,
                                              4096);
  for (int m0 = 0; m0 < M; m0 += MB) {
    const int mcnt = std::min(MB, M - m0);
#define CF_FC_BWD_DATA(VEC_, RES_)                                                                                \
  hipLaunchKernelGGL((fc_bwd_data_kernel<DT, VEC_, RES_>), dim3(blocks), dim3(256), 0, st, (const T *)dz,            \
                     (const T *)w, (T *)dx, m0, mcnt, K, N, G)
    if (vec && res)
      CF_FC_BWD_DATA(true, true);
    else if (vec)
      CF_FC_BWD_DATA(true, false);
    else if (res)
      CF_FC_BWD_DATA(false, true);
    else
      CF_FC_BWD_DATA(false, false);
#undef CF_FC_BWD_DATA
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// ---- backward weights ------------------------------------------------------
// dW[k][4 c .. 4 c + 3] = sum over m = 0 .. M-1 of x[m][k] dz[m][4 c ..]
template <int DT, bool VECTOR>
__global__ __launch_bounds__(256) void fc_bwd_weight_kernel(const typename Store<DT>::T *__restrict__ x,
                                                            const typename Store<DT>::T *__restrict__ dz,
                                                            float *__restrict__ dw, int M, int K, int N,
                                                            long long items) {
  constexpr int V = VECTOR ? 4 : 1;
  const int gq = N / V;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < items; i += (long long)gridDim.x * 256) {
    const long long k = i / gq;
    const int c = (int)(i - k * gq) * V;
    float acc[V];
#pragma unroll
    for (int j = 0; j < V; ++j) acc[j] = 0.f;
    for (int m = 0; m < M; ++m) {
      const float xv = to_f32<DT>(x[(long long)m * K + k]);
#pragma unroll
      for (int j = 0; j < V; ++j) acc[j] = fmaf(xv, to_f32<DT>(dz[(long long)m * N + c + j]), acc[j]);
    }
    if constexpr (VECTOR)
      *reinterpret_cast<float4 *>(dw + k * N + c) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    else
      dw[k * N + c] = acc[0];
  }
}

// Blocked form for N % 4 == 0: thread = (8 consecutive rows kb .. kb+7,
// column quad c .. c+3).  Per batch row one load of 4 dz values and one
// 16-byte load of x[m][kb .. kb+7] (bf16; two for fp32) when K % 8 == 0,
// else guarded element loads; 32 outputs summed over m in order.
template <int DT, bool XVEC>
__global__ __launch_bounds__(256) void fc_bwd_weight_blk_kernel(const typename Store<DT>::T *__restrict__ x,
                                                                const typename Store<DT>::T *__restrict__ dz,
                                                                float *__restrict__ dw, int M, int K, int N,
                                                                long long items) {
  const int gq = N / 4;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < items; i += (long long)gridDim.x * 256) {
    const long long kb = (i / gq) * 8;
    const int c = (int)(i - (i / gq) * gq) * 4;
    const int kn = (int)std::min<long long>(8, K - kb);
    float acc[8][4];
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[r][j] = 0.f;
    for (int m = 0; m < M; ++m) {
      float d[4];
      const typename Store<DT>::T *dr = dz + (long long)m * N + c;
      if constexpr (DT == DT_BF16) {
        const uint2 u = *reinterpret_cast<const uint2 *>(dr);
        d[0] = __uint_as_float(u.x << 16); d[1] = __uint_as_float(u.x & 0xffff0000u);
        d[2] = __uint_as_float(u.y << 16); d[3] = __uint_as_float(u.y & 0xffff0000u);
      } else {
        const float4 f = *reinterpret_cast<const float4 *>(dr);
        d[0] = f.x; d[1] = f.y; d[2] = f.z; d[3] = f.w;
      }
      float xv[8];
      const typename Store<DT>::T *xr = x + (long long)m * K + kb;
      if constexpr (XVEC) {
        if constexpr (DT == DT_BF16) {
          Vec16<DT_BF16> v;
          v.u = ld16<false>(xr);
#pragma unroll
          for (int r = 0; r < 8; ++r) xv[r] = bf2f(v.e[r]);
        } else {
          const float4 a = *reinterpret_cast<const float4 *>(xr);
          const float4 b = *reinterpret_cast<const float4 *>(xr + 4);
          xv[0] = a.x; xv[1] = a.y; xv[2] = a.z; xv[3] = a.w;
          xv[4] = b.x; xv[5] = b.y; xv[6] = b.z; xv[7] = b.w;
        }
      } else {
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          xv[r] = 0.f;
          if (r < kn) xv[r] = to_f32<DT>(xr[r]);
        }
      }
#pragma unroll
      for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[r][j] = fmaf(xv[r], d[j], acc[r][j]);
    }
#pragma unroll
    for (int r = 0; r < 8; ++r)
      if (r < kn) *reinterpret_cast<float4 *>(dw + (kb + r) * N + c) = make_float4(acc[r][0], acc[r][1], acc[r][2], acc[r][3]);
  }
}

template <int DT>
hipError_t fc_bwd_weight_t(int M, int K, int N, const void *x, const void *dz, float *dw, hipStream_t st) {
  using T = typename Store<DT>::T;
  if (N % 4 == 0) {
    const long long items = ((long long)K + 7) / 8 * (N / 4);
    const int blocks = (int)std::min<long long>((items + 255) / 256, 256LL * 64);
    if (K % 8 == 0)
      hipLaunchKernelGGL((fc_bwd_weight_blk_kernel<DT, true>), dim3(blocks), dim3(256), 0, st, (const T *)x,
                         (const T *)dz, dw, M, K, N, items);
    else
      hipLaunchKernelGGL((fc_bwd_weight_blk_kernel<DT, false>), dim3(blocks), dim3(256), 0, st, (const T *)x,
                         (const T *)dz, dw, M, K, N, items);
    return hipGetLastError();
  }
  const long long items = (long long)K * N;
  const int blocks = (int)std::min<long long>((items + 255) / 256, 256LL * 64);
  hipLaunchKernelGGL((fc_bwd_weight_kernel<DT, false>), dim3(blocks), dim3(256), 0, st, (const T *)x, (const T *)dz,
                     dw, M, K, N, items);
  return hipGetLastError();
}

// ---- loss ------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(256) void mse_loss_kernel(const typename Store<DT>::T *__restrict__ p,
                                                       const float *__restrict__ t, float *__restrict__ loss,
                                                       typename Store<DT>::T *__restrict__ dp, long long n,
                                                       float inv) {
  __shared__ float red[256];
  const int tid = threadIdx.x;
  float s = 0.f;
  for (long long i = tid; i < n; i += 256) {
    const float e = to_f32<DT>(p[i]) - t[i];
    s = fmaf(e, e, s);
    if (dp) dp[i] = from_f32<DT>(2.f * e * inv);
  }
  red[tid] = s;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (tid < h) red[tid] += red[tid + h];
    __syncthreads();
  }
  if (tid == 0) loss[0] = red[0] * inv;
}

// ---- the whole head in four launches ----------------------------------------
// (1) fc_fwd_kernel: the first layer's split-K partial rows (as cf_fc_fwd);
// (2) fc_finalize_kernel<BIAS_ACT>: their column sums with bias and leaky ReLU;
// (3) fc_head_tail_kernel, one workgroup: every later layer forward from LDS,
//     the loss, every later layer backward, and the first layer's leaky-ReLU
//     backward (dz1, db1);
// (4) fc_head_bwd1_kernel: the first layer's dW and dx in one pass over W.
// The layers after the first are a few thousand weights (the network's 128 ->
// 64 -> 3): their weights and activations live in LDS.  Rounding points are
// those of the per-layer calls (z and y rounded to the dtype, dz rounded, db
// summing the unrounded products), and the first layer's y, dW and dx are the
// per-layer kernels' sums in the same order.

constexpr int HEAD_MAX_L = 4;    // layers
constexpr int HEAD_MAX_W = 512;  // width of every layer's output
constexpr int HEAD_ACT = 8192;   // batch rows x (sum of the output widths), fp32 in LDS
constexpr int HEAD_WT = 16384;   // weights after the first layer, rows padded by one (fp32 in LDS)

struct HeadParams {
  int m, L;  // batch rows, layers
  int dims[HEAD_MAX_L + 1];
  float alpha, inv;  // inv = 1 / (m * dims[L])
  const void *w[HEAD_MAX_L];
  const float *b[HEAD_MAX_L];
  const float *target;
  void *y[HEAD_MAX_L];
  void *dz[HEAD_MAX_L];
  void *dx[HEAD_MAX_L];
  float *dw[HEAD_MAX_L];
  float *db[HEAD_MAX_L];
  float *loss;
};

template <int DT>
__global__ __launch_bounds__(1024) void fc_head_tail_kernel(const HeadParams p) {
  using T = typename Store<DT>::T;
  __shared__ float wl[HEAD_WT];         // layer i >= 1: [K][N + 1]
  __shared__ float ys[HEAD_ACT];        // layer i: y [m][N] (fp32 values of the stored dtype)
  __shared__ float gb[8 * HEAD_MAX_W];  // gradient of the current layer's output
  __shared__ float zb[8 * HEAD_MAX_W];  // dz of the current layer (rounded)
  __shared__ float red[1024];
  __shared__ float bl[HEAD_MAX_L * HEAD_MAX_W];  // biases of layers 1 .. L-1
  const int tid = threadIdx.x, m = p.m, L = p.L;
  const float alpha = p.alpha;

  // Everything the workgroup reads from global memory, in one round: the
  // weights of layers 1 .. L-1 (16-byte loads), their biases, the target (in
  // zb until the loss) and layer 0's y (written by the finalize kernel).
  {
    constexpr int EV = 16 / sizeof(T);
    int off = 0;
    for (int i = 1; i < L; ++i) {
      const int K = p.dims[i], N = p.dims[i + 1], KN = K * N, nv = KN / EV;
      const T *w = (const T *)p.w[i];
      for (int v = tid; v < nv; v += 1024) {
        Vec16<DT> u;
        u.u = ld16<false>(w + (long long)v * EV);
#pragma unroll
        for (int e = 0; e < EV; ++e) {
          const int q = v * EV + e, k = q / N, j = q - k * N;
          wl[off + k * (N + 1) + j] = to_f32<DT>(u.e[e]);
        }
      }
      for (int q = nv * EV + tid; q < KN; q += 1024) {
        const int k = q / N, j = q - k * N;
        wl[off + k * (N + 1) + j] = to_f32<DT>(w[q]);
      }
      for (int j = tid; j < N; j += 1024) bl[(i - 1) * HEAD_MAX_W + j] = p.b[i][j];
      off += K * (N + 1);
    }
    for (int o = tid; o < m * p.dims[L]; o += 1024) zb[o] = p.target[o];
    for (int o = tid; o < m * p.dims[1]; o += 1024) ys[o] = to_f32<DT>(((const T *)p.y[0])[o]);
  }
  __syncthreads();
  // layers 1 .. L-1 forward: z = y_prev W (k ascending), rounded; y = lrelu(z + b)
  int yo = 0, wo = 0;
  for (int i = 1; i < L; ++i) {
    const int K = p.dims[i], N = p.dims[i + 1];
    const int yin = yo, yout = yo + m * K;
    for (int o = tid; o < m * N; o += 1024) {
      const int mm = o / N, j = o - mm * N;
      float acc = 0.f;
#pragma unroll 16
      for (int k = 0; k < K; ++k) acc = fmaf(ys[yin + mm * K + k], wl[wo + k * (N + 1) + j], acc);
      const T z = from_f32<DT>(acc);
      const float u = to_f32<DT>(z) + bl[(i - 1) * HEAD_MAX_W + j];
      const T y = from_f32<DT>(u > 0.f ? u : alpha * u);
      ((T *)p.y[i])[o] = y;
      ys[yout + o] = to_f32<DT>(y);
    }
    yo = yout;
    wo += K * (N + 1);
    __syncthreads();
  }
  // loss = sum e^2 / (m n), dL/dy = 2 e / (m n) rounded to the dtype
  {
    const int n = m * p.dims[L];
    float s = 0.f;
    for (int o = tid; o < n; o += 1024) {
      const float e = ys[yo + o] - zb[o];
      s = fmaf(e, e, s);
      gb[o] = to_f32<DT>(from_f32<DT>(2.f * e * p.inv));
    }
    red[tid] = s;
    __syncthreads();  // also: the target in zb is read
    for (int h = 512; h > 0; h >>= 1) {
      if (tid < h) red[tid] += red[tid + h];
      __syncthreads();
    }
    if (tid == 0) p.loss[0] = red[0] * p.inv;
  }
  // backward, layer L-1 down to 0
  for (int i = L - 1; i >= 0; --i) {
    const int N = p.dims[i + 1];
    // dz = g * slope(y), rounded; db = sum over the batch rows of the unrounded products
    for (int o = tid; o < m * N; o += 1024) {
      const float d = gb[o] * (ys[yo + o] > 0.f ? 1.f : alpha);
      const T dzv = from_f32<DT>(d);
      ((T *)p.dz[i])[o] = dzv;
      zb[o] = to_f32<DT>(dzv);
    }
    for (int j = tid; j < N; j += 1024) {
      float s = 0.f;
#pragma unroll 8
      for (int mm = 0; mm < m; ++mm) s += gb[mm * N + j] * (ys[yo + mm * N + j] > 0.f ? 1.f : alpha);
      p.db[i][j] = s;
    }
    __syncthreads();
    if (i == 0) break;
    const int K = p.dims[i];
    const int yin = yo - m * K;
    wo -= K * (N + 1);
    // dW[k][j] = sum over the batch rows (ascending) of y_prev[mm][k] dz[mm][j]
    for (int e = tid; e < K * N; e += 1024) {
      const int k = e / N, j = e - k * N;
      float acc = 0.f;
#pragma unroll 8
      for (int mm = 0; mm < m; ++mm) acc = fmaf(ys[yin + mm * K + k], zb[mm * N + j], acc);
      p.dw[i][e] = acc;
    }
    // dx[mm][k] = sum over j (ascending) of dz[mm][j] W[k][j], rounded: the next g
    for (int o = tid; o < m * K; o += 1024) {
      const int mm = o / K, k = o - mm * K;
      float acc = 0.f;
#pragma unroll 16
      for (int j = 0; j < N; ++j) acc = fmaf(zb[mm * N + j], wl[wo + k * (N + 1) + j], acc);
      const T v = from_f32<DT>(acc);
      ((T *)p.dx[i])[o] = v;
      gb[o] = to_f32<DT>(v);
    }
    yo = yin;
    __syncthreads();
  }
}

// First layer backward: lane gl of a G-lane group owns columns [V gl, V gl + V)
// of dz (resident in registers for all batch rows); a group walks blocks of
// eight rows k of W.  dx[mm][k]: the lane's V products in column order, then
// an xor butterfly over the group (the order of fc_bwd_data_kernel); dW[k][c]:
// the batch rows in ascending order (that of fc_bwd_weight_blk_kernel).
template <int DT, int G>
__global__ __launch_bounds__(256) void fc_head_bwd1_kernel(const typename Store<DT>::T *__restrict__ x,
                                                           const typename Store<DT>::T *__restrict__ dz,
                                                           const typename Store<DT>::T *__restrict__ w,
                                                           float *__restrict__ dw, typename Store<DT>::T *__restrict__ dx,
                                                           int M, int K, int N) {
  using T = typename Store<DT>::T;
  constexpr int V = Store<DT>::VEC;
  constexpr int XV = 16 / sizeof(T);  // elements of a 16-byte load
  const int tid = threadIdx.x, gl = tid & (G - 1);
  constexpr int GROUPS = 256 / G;
  float dzr[MB][V];
#pragma unroll
  for (int mm = 0; mm < MB; ++mm) {
    if (mm < M) {
      Vec16<DT> g;
      g.u = ld16<false>(dz + (long long)mm * N + gl * V);
#pragma unroll
      for (int j = 0; j < V; ++j) dzr[mm][j] = to_f32<DT>(g.e[j]);
    } else {
#pragma unroll
      for (int j = 0; j < V; ++j) dzr[mm][j] = 0.f;
    }
  }
  const int nblk = K / 8;
  for (int kb = (int)blockIdx.x * GROUPS + tid / G; kb < nblk; kb += (int)gridDim.x * GROUPS) {
    const long long k0 = (long long)kb * 8;
    // x[mm][k0 .. k0 + 7] for every batch row
    float xv[MB][8];
#pragma unroll
    for (int mm = 0; mm < MB; ++mm) {
      if (mm < M) {
#pragma unroll
        for (int h = 0; h < 8 / XV; ++h) {
          Vec16<DT> v;
          v.u = ld16<false>(x + (long long)mm * K + k0 + h * XV);
#pragma unroll
          for (int e = 0; e < XV; ++e) xv[mm][h * XV + e] = to_f32<DT>(v.e[e]);
        }
      } else {
#pragma unroll
        for (int r = 0; r < 8; ++r) xv[mm][r] = 0.f;
      }
    }
    float dxo[8];  // lane mm < M: dx[mm][k0 + r]
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const long long k = k0 + r;
      Vec16<DT> wv;
      wv.u = ld16<false>(w + k * N + gl * V);
      float wf[V];
#pragma unroll
      for (int j = 0; j < V; ++j) wf[j] = to_f32<DT>(wv.e[j]);
      // dW row k, this lane's columns
      float a[V];
#pragma unroll
      for (int j = 0; j < V; ++j) a[j] = 0.f;
#pragma unroll
      for (int mm = 0; mm < MB; ++mm)
        if (mm < M)
#pragma unroll
          for (int j = 0; j < V; ++j) a[j] = fmaf(xv[mm][r], dzr[mm][j], a[j]);
#pragma unroll
      for (int j = 0; j < V; j += 4)
        *reinterpret_cast<float4 *>(dw + k * N + gl * V + j) = make_float4(a[j], a[j + 1], a[j + 2], a[j + 3]);
      // dx column k
      float acc[MB];
#pragma unroll
      for (int mm = 0; mm < MB; ++mm) {
        acc[mm] = 0.f;
#pragma unroll
        for (int j = 0; j < V; ++j) acc[mm] = fmaf(dzr[mm][j], wf[j], acc[mm]);
      }
#pragma unroll
      for (int off = G >> 1; off > 0; off >>= 1)
#pragma unroll
        for (int mm = 0; mm < MB; ++mm) acc[mm] += __shfl_xor(acc[mm], off, 64);
      dxo[r] = acc[0];
#pragma unroll
      for (int mm = 1; mm < MB; ++mm)
        if (gl == mm) dxo[r] = acc[mm];
    }
    if (gl < M) {
      Vec16<DT> o;
#pragma unroll
      for (int h = 0; h < 8 / XV; ++h) {
#pragma unroll
        for (int e = 0; e < XV; ++e) o.e[e] = from_f32<DT>(dxo[h * XV + e]);
        *reinterpret_cast<uint4 *>(dx + (long long)gl * K + k0 + h * XV) = o.u;
      }
    }
  }
}

}  // namespace

size_t fc_fwd_workspace(int M, int K, int N) {
  if (M <= 0 || K <= 0 || N <= 0) return 0;
  const FwdPlan a = plan_fwd(K, N, 8), b = plan_fwd(K, N, 4);
  const int blocks = std::max(a.blocks, b.blocks);
  return (size_t)blocks * MB * N * sizeof(float);
}

hipError_t launch_fc_fwd(int M, int K, int N, int dtype, const void *x, const void *w, void *y, void *ws,
                         hipStream_t st) {
  return dtype == DT_BF16 ? fc_fwd_t<DT_BF16>(M, K, N, x, w, y, ws, st)
                          : fc_fwd_t<DT_F32>(M, K, N, x, w, y, ws, st);
}

hipError_t launch_fc_bwd_data(int M, int K, int N, int dtype, const void *dz, const void *w, void *dx,
                              hipStream_t st) {
  return dtype == DT_BF16 ? fc_bwd_data_t<DT_BF16>(M, K, N, dz, w, dx, st)
                          : fc_bwd_data_t<DT_F32>(M, K, N, dz, w, dx, st);
}

hipError_t launch_fc_bwd_weight(int M, int K, int N, int dtype, const void *x, const void *dz, float *dw,
                                hipStream_t st) {
  return dtype == DT_BF16 ? fc_bwd_weight_t<DT_BF16>(M, K, N, x, dz, dw, st)
                          : fc_bwd_weight_t<DT_F32>(M, K, N, x, dz, dw, st);
}

bool fc_head_supported(int M, int L, const int *dims, int dtype) {
  if (L < 2 || L > HEAD_MAX_L || M < 1 || M > MB) return false;
  const int V = dtype == DT_BF16 ? Store<DT_BF16>::VEC : Store<DT_F32>::VEC;
  const long long K0 = dims[0], N1 = dims[1];
  if (K0 < 8 || K0 % 8 != 0 || K0 >= (1LL << 31) || N1 % V != 0) return false;
  const long long g = N1 / V;  // lanes per row of the first layer's backward: a power of two, 8 .. 64
  if (g < 8 || g > 64 || (g & (g - 1)) != 0 || K0 * N1 >= (1LL << 40)) return false;
  long long act = 0, wts = 0;
  for (int i = 1; i <= L; ++i) {
    if (dims[i] < 1 || dims[i] > HEAD_MAX_W) return false;
    act += (long long)M * dims[i];
    if (i < L) wts += (long long)dims[i] * (dims[i + 1] + 1);
  }
  return act <= HEAD_ACT && wts <= HEAD_WT;
}

size_t fc_head_workspace(int M, int L, const int *dims) { return fc_fwd_workspace(M, dims[0], dims[1]); }

hipError_t launch_fc_head(int M, int L, const int *dims, int dtype, const void *x, const void *const *w,
                          const float *const *b, float alpha, const float *target, void *const *y, void *const *dz,
                          void *const *dx, float *const *dw, float *const *db, float *loss, void *ws,
                          hipStream_t st) {
  const int K0 = dims[0], N1 = dims[1];
  const int V = dtype == DT_BF16 ? Store<DT_BF16>::VEC : Store<DT_F32>::VEC;
  const FwdPlan pl = plan_fwd(K0, N1, V);
  float *part = (float *)ws;
  HeadParams hp{};
  hp.m = M; hp.L = L;
  for (int i = 0; i <= L; ++i) hp.dims[i] = dims[i];
  hp.alpha = alpha;
  hp.inv = (float)(1.0 / ((double)M * dims[L]));
  for (int i = 0; i < L; ++i) {
    hp.w[i] = w[i]; hp.b[i] = b[i]; hp.y[i] = y[i]; hp.dz[i] = dz[i]; hp.dx[i] = dx[i];
    hp.dw[i] = dw[i]; hp.db[i] = db[i];
  }
  hp.target = target;
  hp.loss = loss;
  const int G = N1 / V;
  const int blocks = std::min((K0 / 8 + 256 / G - 1) / (256 / G), 2 * kNumCUs);
#define CF_HEAD_LAUNCH(DTV, TT)                                                                                    \
  {                                                                                                                \
    hipLaunchKernelGGL((fc_fwd_kernel<DTV, true>), dim3(pl.blocks), dim3(256), 0, st, (const TT *)x,              \
                       (const TT *)w[0], part, 0, M, K0, N1, pl.cgw, pl.np, pl.kc);                                \
    hipError_t e = hipGetLastError();                                                                              \
    if (e != hipSuccess) return e;                                                                                 \
    hipLaunchKernelGGL((fc_finalize_kernel<DTV, true>), dim3((M * N1 + 15) / 16), dim3(256), 0, st, part,          \
                       pl.blocks, M * N1, (TT *)y[0], b[0], N1, alpha);                                            \
    if ((e = hipGetLastError()) != hipSuccess) return e;                                                           \
    hipLaunchKernelGGL((fc_head_tail_kernel<DTV>), dim3(1), dim3(1024), 0, st, hp);                               \
    if ((e = hipGetLastError()) != hipSuccess) return e;                                                           \
    switch (G) {                                                                                                   \
      case 8: hipLaunchKernelGGL((fc_head_bwd1_kernel<DTV, 8>), dim3(blocks), dim3(256), 0, st, (const TT *)x,     \
                                 (const TT *)dz[0], (const TT *)w[0], dw[0], (TT *)dx[0], M, K0, N1); break;       \
      case 16: hipLaunchKernelGGL((fc_head_bwd1_kernel<DTV, 16>), dim3(blocks), dim3(256), 0, st, (const TT *)x,   \
                                  (const TT *)dz[0], (const TT *)w[0], dw[0], (TT *)dx[0], M, K0, N1); break;      \
      case 32: hipLaunchKernelGGL((fc_head_bwd1_kernel<DTV, 32>), dim3(blocks), dim3(256), 0, st, (const TT *)x,   \
                                  (const TT *)dz[0], (const TT *)w[0], dw[0], (TT *)dx[0], M, K0, N1); break;      \
      default: hipLaunchKernelGGL((fc_head_bwd1_kernel<DTV, 64>), dim3(blocks), dim3(256), 0, st, (const TT *)x,   \
                                  (const TT *)dz[0], (const TT *)w[0], dw[0], (TT *)dx[0], M, K0, N1); break;      \
    }                                                                                                              \
    return hipGetLastError();                                                                                      \
  }
  if (dtype == DT_BF16) CF_HEAD_LAUNCH(DT_BF16, uint16_t)
  CF_HEAD_LAUNCH(DT_F32, float)
#undef CF_HEAD_LAUNCH
}

hipError_t launch_mse_loss(long long n, int dtype, const void *p, const float *t, float *loss, void *dp,
                           float inv, hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(mse_loss_kernel<DT_BF16>, dim3(1), dim3(256), 0, st, (const uint16_t *)p, t, loss,
                       (uint16_t *)dp, n, inv);
  else
    hipLaunchKernelGGL(mse_loss_kernel<DT_F32>, dim3(1), dim3(256), 0, st, (const float *)p, t, loss, (float *)dp,
                       n, inv);
  return hipGetLastError();
}

}  // namespace cf
