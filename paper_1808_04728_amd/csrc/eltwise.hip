// eltwise.hip -- bias + leaky ReLU forward / backward for gfx950.
//
// Section III-A: every convolution layer is followed by a leaky ReLU; the
// paper runs it as separate, OpenMP-threaded TensorFlow element-wise ops and
// notes their load imbalance (Section V-B).  Here both directions are single
// HBM-bound passes with 16-byte vector access:
//   forward   y = lrelu(z + b)                               (read z, write y)
//   backward  dz = dy * (y > 0 ? 1 : alpha), db = sum dz      (read dy, y; write dz)
// The bias gradient is reduced without atomics: each workgroup owns a fixed
// contiguous voxel range, threads own (voxel phase, channel group) pairs and
// keep fp32 partial sums in registers, the workgroup combines its phases in
// LDS in phase order and writes one partial row; a second kernel sums the
// rows in workgroup order.

#include "cf_common.h"
#include "cf_kernels.h"
#include "fastdiv.h"

#include <algorithm>

namespace cf {
namespace {

__device__ __forceinline__ float lrelu(float u, float alpha) { return u > 0.f ? u : alpha * u; }

template <int DT, bool VECTOR>
__global__ __launch_bounds__(256) void bias_lrelu_fwd_kernel(const typename Store<DT>::T *z,
                                                             const float *__restrict__ bias,
                                                             float alpha,
                                                             typename Store<DT>::T *y,
                                                             long long nelem, int c) {
  using T = typename Store<DT>::T;
  constexpr int V = VECTOR ? Store<DT>::VEC : 1;
  const long long nv = nelem / V;
  const long long stride = (long long)gridDim.x * 256;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < nv; i += stride) {
    const int c0 = (int)((i * V) % c);
    if constexpr (VECTOR) {
      Vec16<DT> v;
      v.u = reinterpret_cast<const uint4 *>(z)[i];
#pragma unroll
      for (int j = 0; j < V; ++j)
        v.e[j] = from_f32<DT>(lrelu(to_f32<DT>(v.e[j]) + bias[c0 + j], alpha));
      reinterpret_cast<uint4 *>(y)[i] = v.u;
    } else {
      y[i] = from_f32<DT>(lrelu(to_f32<DT>(z[i]) + bias[c0], alpha));
    }
  }
}

// 32-bit form of the vector forward pass (every element offset below 2^31):
// the channel group of item i is i mod c/V by a launch-time divisor instead of
// a 64-bit remainder
template <int DT, bool NT>
__global__ __launch_bounds__(256) void bias_lrelu_fwd32_kernel(const typename Store<DT>::T *z,
                                                               const float *__restrict__ bias, float alpha,
                                                               typename Store<DT>::T *y, int nv, FastDiv fcg) {
  constexpr int V = Store<DT>::VEC;
  const int i = (int)blockIdx.x * 256 + threadIdx.x;
  if (i >= nv) return;
  const int c0 = (i - fdiv(i, fcg) * (int)fcg.div) * V;
  Vec16<DT> v;
  v.u = ld16<NT>(z + (long long)V * i);
#pragma unroll
  for (int j = 0; j < V; ++j) v.e[j] = from_f32<DT>(lrelu(to_f32<DT>(v.e[j]) + bias[c0 + j], alpha));
  st16<NT>(y + (long long)V * i, v.u);
}

// Thread layout of the backward kernel: CG channel groups of V channels,
// PH = max(1, 256 / CG) voxel phases.
template <int DT, bool VECTOR, bool WITH_DB>
__global__ __launch_bounds__(256) void bias_lrelu_bwd_kernel(const typename Store<DT>::T *dy,
                                                             const typename Store<DT>::T *__restrict__ y,
                                                             float alpha,
                                                             typename Store<DT>::T *dz,
                                                             float *__restrict__ part,
                                                             long long nvox, int c, long long vpb) {
  using T = typename Store<DT>::T;
  constexpr int V = VECTOR ? Store<DT>::VEC : 1;
  __shared__ float red[2048];  // phases * c <= 256 * V, and c <= 2048 (checked by the host)
  const int cg_n = c / V;
  const int ph_n = cg_n >= 256 ? 1 : 256 / cg_n;
  const int tid = threadIdx.x;
  const long long v0 = (long long)blockIdx.x * vpb;
  const long long v1 = v0 + vpb < nvox ? v0 + vpb : nvox;
  const int ph = tid / (cg_n >= 256 ? 256 : cg_n);
  // every (phase, group) pair this thread owns
  for (int cg = (cg_n >= 256 ? tid : tid % cg_n); ph < ph_n && cg < cg_n; cg += 256) {
    float s[V];
#pragma unroll
    for (int j = 0; j < V; ++j) s[j] = 0.f;
    long long v = v0 + ph;
    if constexpr (VECTOR) {
      // four voxels per step (eight loads in flight), summed in voxel order as below
      for (; v + 3LL * ph_n < v1; v += 4LL * ph_n) {
        Vec16<DT> g[4], o[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const long long e = (v + (long long)u * ph_n) * c + (long long)cg * V;
          g[u].u = *reinterpret_cast<const uint4 *>(dy + e);
          o[u].u = *reinterpret_cast<const uint4 *>(y + e);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int j = 0; j < V; ++j) {
            float d = to_f32<DT>(g[u].e[j]) * (to_f32<DT>(o[u].e[j]) > 0.f ? 1.f : alpha);
            s[j] += d;
            g[u].e[j] = from_f32<DT>(d);
          }
#pragma unroll
        for (int u = 0; u < 4; ++u)
          *reinterpret_cast<uint4 *>(dz + (v + (long long)u * ph_n) * c + (long long)cg * V) = g[u].u;
      }
    }
    for (; v < v1; v += ph_n) {
      const long long e = v * c + (long long)cg * V;
      if constexpr (VECTOR) {
        Vec16<DT> g, o;
        g.u = *reinterpret_cast<const uint4 *>(dy + e);
        o.u = *reinterpret_cast<const uint4 *>(y + e);
#pragma unroll
        for (int j = 0; j < V; ++j) {
          float d = to_f32<DT>(g.e[j]) * (to_f32<DT>(o.e[j]) > 0.f ? 1.f : alpha);
          s[j] += d;
          g.e[j] = from_f32<DT>(d);
        }
        *reinterpret_cast<uint4 *>(dz + e) = g.u;
      } else {
        float d = to_f32<DT>(dy[e]) * (to_f32<DT>(y[e]) > 0.f ? 1.f : alpha);
        s[0] += d;
        dz[e] = from_f32<DT>(d);
      }
    }
    if constexpr (WITH_DB) {
#pragma unroll
      for (int j = 0; j < V; ++j) {
        if (cg_n >= 256) red[cg * V + j] = s[j];  // a single phase
        else red[ph * c + cg * V + j] = s[j];
      }
    }
    if (cg_n < 256) break;
  }
  if constexpr (WITH_DB) {
    __syncthreads();
    for (int ch = tid; ch < c; ch += 256) {
      float acc = 0.f;
      for (int k = 0; k < ph_n; ++k) acc += red[k * c + ch];
      part[(long long)blockIdx.x * c + ch] = acc;
    }
  }
}

// One pass over whole 16-byte vectors with 32-bit offsets, for c / V a power
// of two up to 64 and c <= 256: workgroup b takes the chunks of U * 256
// consecutive vectors starting at (b + i * gridDim) * U * 256, thread t the
// vectors t, t + 256, ... of each chunk (all of channel group t % (c / V),
// since c / V divides 256), its U loads of a chunk issued together.  The
// bias-gradient partial of the workgroup: each thread sums its vectors in
// order, a fixed butterfly over the lanes of a wave that share a channel
// group, then the four waves as (w0 + w1) + (w2 + w3).  Looping over chunks
// keeps the number of workgroups, and so of partial rows to sum, small.
template <int DT, bool WITH_DB, int U, bool NT>
__global__ __launch_bounds__(256) void bias_lrelu_bwd_vec_kernel(const typename Store<DT>::T *__restrict__ dy,
                                                                 const typename Store<DT>::T *__restrict__ y,
                                                                 float alpha, typename Store<DT>::T *__restrict__ dz,
                                                                 float *__restrict__ part, int nv, int cg_n, int c) {
  constexpr int V = Store<DT>::VEC;
  __shared__ float red[4 * 256];
  const int tid = threadIdx.x;
  float s[V];
#pragma unroll
  for (int j = 0; j < V; ++j) s[j] = 0.f;
  for (int k0 = (int)blockIdx.x * (256 * U) + tid; k0 < nv; k0 += (int)gridDim.x * (256 * U)) {
    Vec16<DT> g[U], o[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (k0 + 256 * u < nv) {
        g[u].u = ld16<NT>(dy + V * (k0 + 256 * u));
        o[u].u = ld16<NT>(y + V * (k0 + 256 * u));
      }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (k0 + 256 * u < nv) {
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const float d = to_f32<DT>(g[u].e[j]) * (to_f32<DT>(o[u].e[j]) > 0.f ? 1.f : alpha);
          s[j] += d;
          g[u].e[j] = from_f32<DT>(d);
        }
        st16<NT>(dz + V * (k0 + 256 * u), g[u].u);
      }
  }
  if constexpr (WITH_DB) {
    for (int off = cg_n; off < 64; off <<= 1)
#pragma unroll
      for (int j = 0; j < V; ++j) s[j] += __shfl_xor(s[j], off, 64);
    const int lane = tid & 63, wave = tid >> 6;
    if (lane < cg_n)
#pragma unroll
      for (int j = 0; j < V; ++j) red[wave * 256 + lane * V + j] = s[j];
    __syncthreads();
    if (tid < c)
      part[(long long)blockIdx.x * c + tid] = (red[tid] + red[256 + tid]) + (red[512 + tid] + red[768 + tid]);
  }
}

// Pooled layer's dz in one pass, the adjoints of the 2^3 pool and of the
// leaky ReLU composed (Section III-C: pooling is a constant-weight
// convolution; Section III-A: leaky ReLU after the convolution):
//   dz[v, c] = g[pool(v), c] / 8 * (mask bit (v, c) ? 1 : alpha),
// zero where no complete window covers v; db[c] = sum_v dz[v, c] from the
// unrounded fp32 values, in the fixed order of bias_lrelu_bwd_vec_kernel.
// Item k is the k-th 16-byte vector of dz (NDHWC): voxel k / cg_n, channel
// group k % cg_n; its mask bits are bits V k .. V k + V - 1.
template <int DT, bool WITH_DB>
__global__ __launch_bounds__(256) void pool_lrelu_bwd_kernel(const typename Store<DT>::T *__restrict__ g,
                                                             const uint8_t *__restrict__ mask, float alpha,
                                                             typename Store<DT>::T *__restrict__ dz,
                                                             float *__restrict__ part, int nv, int cg_n, int c,
                                                             FastDiv fcg, FastDiv fw, FastDiv fh, FastDiv fd,
                                                             int pd, int ph, int pw) {
  constexpr int V = Store<DT>::VEC;
  __shared__ float red[4 * 256];
  const int tid = threadIdx.x;
  const float a1 = 0.125f, a0 = 0.125f * alpha;
  float s[V];
#pragma unroll
  for (int j = 0; j < V; ++j) s[j] = 0.f;
  for (int k = (int)blockIdx.x * 256 + tid; k < nv; k += (int)gridDim.x * 256) {
    const int vox = fdiv(k, fcg), cg = k - vox * (int)fcg.div;
    const int t1 = fdiv(vox, fw), t2 = fdiv(t1, fh), n = fdiv(t2, fd);
    const int x_ = vox - t1 * (int)fw.div, y_ = t1 - t2 * (int)fh.div, z_ = t2 - n * (int)fd.div;
    const int px = x_ >> 1, py = y_ >> 1, pz = z_ >> 1;
    Vec16<DT> v;
    if (pz < pd && py < ph && px < pw) {
      v.u = ld16<false>(g + (((n * pd + pz) * ph + py) * pw + px) * c + V * cg);
      uint32_t bits = mask[(V * k) >> 3];
      if constexpr (V == 4) bits >>= 4 * (k & 1);
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const float d = to_f32<DT>(v.e[j]) * (((bits >> j) & 1u) ? a1 : a0);
        s[j] += d;
        v.e[j] = from_f32<DT>(d);
      }
    } else {
      v.u = make_uint4(0, 0, 0, 0);
    }
    st16<false>(dz + V * k, v.u);
  }
  if constexpr (WITH_DB) {
    for (int off = cg_n; off < 64; off <<= 1)
#pragma unroll
      for (int j = 0; j < V; ++j) s[j] += __shfl_xor(s[j], off, 64);
    const int lane = tid & 63, wave = tid >> 6;
    if (lane < cg_n)
#pragma unroll
      for (int j = 0; j < V; ++j) red[wave * 256 + lane * V + j] = s[j];
    __syncthreads();
    if (tid < c)
      part[(long long)blockIdx.x * c + tid] = (red[tid] + red[256 + tid]) + (red[512 + tid] + red[768 + tid]);
  }
}

__global__ __launch_bounds__(256) void fill_zero_kernel(float *out, long long n) {
  long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) out[i] = 0.f;
}

struct BwdPlan {
  long long vpb;  // general kernel: voxels per workgroup
  int blocks;
  int unroll;     // vector kernel: vectors per thread (0: the general kernel)
};

// V = elements per 16-byte vector of the dtype
BwdPlan plan_bwd(long long nvox, int c, int V) {
  BwdPlan p{};
  const int cg_n = c / V;
  if (c % V == 0 && (cg_n & (cg_n - 1)) == 0 && cg_n <= 64 && c <= 256 && nvox * c < (1LL << 31)) {
    const long long nv = nvox * cg_n;
    // large tensors: four vectors per thread and chunk, at most 1024 workgroups
    p.unroll = nv >= (1LL << 20) ? 4 : 1;
    p.blocks = (int)((nv + 256LL * p.unroll - 1) / (256LL * p.unroll));
    if (p.unroll == 4) p.blocks = std::min(p.blocks, 1024);
    return p;
  }
  long long vpb = std::max<long long>(64, (nvox + 2047) / 2048);
  p.vpb = vpb;
  p.blocks = (int)((nvox + vpb - 1) / vpb);
  return p;
}

template <int DT>
hipError_t fwd_t(long long nvox, int c, const void *z, const float *bias, float alpha, void *y,
                 hipStream_t st) {
  using T = typename Store<DT>::T;
  const long long nelem = nvox * c;
  const bool vec = c % Store<DT>::VEC == 0;
  const long long items = vec ? nelem / Store<DT>::VEC : nelem;
  if (vec && nelem < (1LL << 31)) {
    if (nelem * (long long)sizeof(T) >= kStreamBytes)
      hipLaunchKernelGGL((bias_lrelu_fwd32_kernel<DT, true>), dim3((unsigned)((items + 255) / 256)), dim3(256), 0,
                         st, (const T *)z, bias, alpha, (T *)y, (int)items, make_fastdiv(c / Store<DT>::VEC));
    else
      hipLaunchKernelGGL((bias_lrelu_fwd32_kernel<DT, false>), dim3((unsigned)((items + 255) / 256)), dim3(256), 0,
                         st, (const T *)z, bias, alpha, (T *)y, (int)items, make_fastdiv(c / Store<DT>::VEC));
    return hipGetLastError();
  }
  const int blocks = (int)std::min<long long>((items + 255) / 256, 256LL * 64);
  if (vec)
    hipLaunchKernelGGL((bias_lrelu_fwd_kernel<DT, true>), dim3(blocks), dim3(256), 0, st,
                       (const T *)z, bias, alpha, (T *)y, nelem, c);
  else
    hipLaunchKernelGGL((bias_lrelu_fwd_kernel<DT, false>), dim3(blocks), dim3(256), 0, st,
                       (const T *)z, bias, alpha, (T *)y, nelem, c);
  return hipGetLastError();
}

template <int DT, bool WITH_DB>
hipError_t bwd_t(long long nvox, int c, const void *dy, const void *y, float alpha, void *dz,
                 float *db, void *ws, hipStream_t st) {
  using T = typename Store<DT>::T;
  const BwdPlan pl = plan_bwd(nvox, c, Store<DT>::VEC);
  const bool vec = c % Store<DT>::VEC == 0;
  float *part = (float *)ws;
  if (pl.unroll) {
    const int nv = (int)(nvox * c / Store<DT>::VEC), cg_n = c / Store<DT>::VEC;
    if (nvox * c * (long long)sizeof(T) >= kStreamBytes)
      hipLaunchKernelGGL((bias_lrelu_bwd_vec_kernel<DT, WITH_DB, 4, true>), dim3(pl.blocks), dim3(256), 0, st,
                         (const T *)dy, (const T *)y, alpha, (T *)dz, part, nv, cg_n, c);
    else if (pl.unroll == 4)
      hipLaunchKernelGGL((bias_lrelu_bwd_vec_kernel<DT, WITH_DB, 4, false>), dim3(pl.blocks), dim3(256), 0, st,
                         (const T *)dy, (const T *)y, alpha, (T *)dz, part, nv, cg_n, c);
    else
      hipLaunchKernelGGL((bias_lrelu_bwd_vec_kernel<DT, WITH_DB, 1, false>), dim3(pl.blocks), dim3(256), 0, st,
                         (const T *)dy, (const T *)y, alpha, (T *)dz, part, nv, cg_n, c);
  } else if (vec)
    hipLaunchKernelGGL((bias_lrelu_bwd_kernel<DT, true, WITH_DB>), dim3(pl.blocks), dim3(256), 0, st,
                       (const T *)dy, (const T *)y, alpha, (T *)dz, part, nvox, c, pl.vpb);
  else
    hipLaunchKernelGGL((bias_lrelu_bwd_kernel<DT, false, WITH_DB>), dim3(pl.blocks), dim3(256), 0, st,
                       (const T *)dy, (const T *)y, alpha, (T *)dz, part, nvox, c, pl.vpb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !WITH_DB) return e;
  return launch_sum_rows(part, db, pl.blocks, c, st);
}

}  // namespace

hipError_t launch_bias_lrelu_fwd(int64_t nvox, int c, int dtype, const void *z, const float *bias,
                                 float alpha, void *y, hipStream_t st) {
  if (nvox == 0) return hipSuccess;
  return dtype == DT_BF16 ? fwd_t<DT_BF16>(nvox, c, z, bias, alpha, y, st)
                          : fwd_t<DT_F32>(nvox, c, z, bias, alpha, y, st);
}

size_t bias_lrelu_bwd_workspace(int64_t nvox, int c) {
  if (nvox <= 0) return 0;
  // the larger of the two dtypes' plans (the workspace query takes no dtype)
  const int blocks = std::max(plan_bwd(nvox, c, 8).blocks, plan_bwd(nvox, c, 4).blocks);
  return (size_t)blocks * c * sizeof(float);
}

hipError_t launch_bias_lrelu_bwd(int64_t nvox, int c, int dtype, const void *dy, const void *y,
                                 float alpha, void *dz, float *db, void *ws, hipStream_t st) {
  if (nvox == 0) {
    return db ? launch_fill_zero(db, c, st) : hipSuccess;
  }
  if (dtype == DT_BF16)
    return db ? bwd_t<DT_BF16, true>(nvox, c, dy, y, alpha, dz, db, ws, st)
              : bwd_t<DT_BF16, false>(nvox, c, dy, y, alpha, dz, db, ws, st);
  return db ? bwd_t<DT_F32, true>(nvox, c, dy, y, alpha, dz, db, ws, st)
            : bwd_t<DT_F32, false>(nvox, c, dy, y, alpha, dz, db, ws, st);
}

// workgroups of the pooled dz pass: at most 1024, each a whole number of
// 256-vector rounds (the thread -> channel-group map is fixed, see above)
static int pool_lrelu_blocks(long long nvox, int c, int V) {
  const long long nv = nvox * (c / V);
  return (int)std::min<long long>((nv + 255) / 256, 1024);
}

bool pool_lrelu_bwd_supported(long long nvox, int c, int dtype) {
  const int V = dtype == DT_BF16 ? 8 : 4;
  const int cg_n = c / V;
  return c % V == 0 && (cg_n & (cg_n - 1)) == 0 && cg_n <= 64 && c <= 256 && nvox * c < (1LL << 31);
}

size_t pool_lrelu_bwd_workspace(int64_t nvox, int c) {
  if (nvox <= 0) return 0;
  return (size_t)std::max(pool_lrelu_blocks(nvox, c, 8), pool_lrelu_blocks(nvox, c, 4)) * c * sizeof(float);
}

template <int DT>
static hipError_t pool_lrelu_t(int n, int d, int h, int w, int c, const void *g, const uint8_t *mask, float alpha,
                               void *dz, float *db, void *ws, hipStream_t st) {
  using T = typename Store<DT>::T;
  constexpr int V = Store<DT>::VEC;
  const long long nvox = (long long)n * d * h * w;
  const int cg_n = c / V, nv = (int)(nvox * cg_n);
  const int blocks = pool_lrelu_blocks(nvox, c, V);
  float *part = (float *)ws;
  if (db)
    hipLaunchKernelGGL((pool_lrelu_bwd_kernel<DT, true>), dim3(blocks), dim3(256), 0, st, (const T *)g, mask, alpha,
                       (T *)dz, part, nv, cg_n, c, make_fastdiv(cg_n), make_fastdiv(w), make_fastdiv(h),
                       make_fastdiv(d), d / 2, h / 2, w / 2);
  else
    hipLaunchKernelGGL((pool_lrelu_bwd_kernel<DT, false>), dim3(blocks), dim3(256), 0, st, (const T *)g, mask,
                       alpha, (T *)dz, part, nv, cg_n, c, make_fastdiv(cg_n), make_fastdiv(w), make_fastdiv(h),
                       make_fastdiv(d), d / 2, h / 2, w / 2);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !db) return e;
  return launch_sum_rows(part, db, blocks, c, st);
}

hipError_t launch_pool_lrelu_bwd(int n, int d, int h, int w, int c, int dtype, const void *g, const void *mask,
                                 float alpha, void *dz, float *db, void *ws, hipStream_t st) {
  if ((long long)n * d * h * w == 0) return db ? launch_fill_zero(db, c, st) : hipSuccess;
  return dtype == DT_BF16 ? pool_lrelu_t<DT_BF16>(n, d, h, w, c, g, (const uint8_t *)mask, alpha, dz, db, ws, st)
                          : pool_lrelu_t<DT_F32>(n, d, h, w, c, g, (const uint8_t *)mask, alpha, dz, db, ws, st);
}

hipError_t launch_fill_zero(float *out, long long n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, out, n);
  return hipGetLastError();
}

}  // namespace cf
