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
template <int DT>
__global__ __launch_bounds__(256) void fc_finalize_kernel(const float *__restrict__ part, int rows, int cols,
                                                          typename Store<DT>::T *y) {
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
    y[col] = from_f32<DT>(t);
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
