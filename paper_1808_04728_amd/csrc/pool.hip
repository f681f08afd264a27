// pool.hip -- 3D average pooling forward / backward for gfx950.
//
// Section III-C: average pooling is a per-channel convolution whose weights
// are all 1/KS^3, and it is bandwidth-bound; Section III-A gives the stride
// (2,2,2).  With non-overlapping windows (k == s) every input voxel belongs
// to at most one window, so both directions are single coalesced passes:
//   forward   one thread per (output voxel, 16-byte channel group): k^3
//             vector loads, fp32 sum, one rounding on store;
//   backward  one thread per (input voxel, channel group): dy = dp / k^3 of
//             the covering window, or 0 outside every window (odd tails).
// 2^3 windows over whole 16-byte channel vectors take the vector kernels
// below (32-bit indices with launch-time divisors: a 64-bit division per
// item made the passes ALU-bound); anything else the general kernels.

#include "cf_common.h"
#include "cf_kernels.h"
#include "fastdiv.h"

#include <algorithm>

namespace cf {
namespace {

template <int DT, bool VECTOR>
__global__ __launch_bounds__(256) void avgpool_fwd_kernel(const typename Store<DT>::T *__restrict__ y,
                                                          typename Store<DT>::T *__restrict__ p,
                                                          int d, int h, int w, int c, int k,
                                                          int od, int oh, int ow, long long items) {
  using T = typename Store<DT>::T;
  constexpr int V = VECTOR ? Store<DT>::VEC : 1;
  const int cg_n = c / V;
  const float scale = 1.f / (float)(k * k * k);
  const long long stride = (long long)gridDim.x * 256;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < items; i += stride) {
    long long t = i;
    const int cg = (int)(t % cg_n); t /= cg_n;
    const int x_ = (int)(t % ow); t /= ow;
    const int y_ = (int)(t % oh); t /= oh;
    const int z_ = (int)(t % od);
    const int n = (int)(t / od);
    float s[V];
#pragma unroll
    for (int j = 0; j < V; ++j) s[j] = 0.f;
    for (int a = 0; a < k; ++a)
      for (int b = 0; b < k; ++b)
        for (int e = 0; e < k; ++e) {
          const long long off =
              ((((long long)n * d + z_ * k + a) * h + y_ * k + b) * w + x_ * k + e) * c + cg * V;
          if constexpr (VECTOR) {
            Vec16<DT> v;
            v.u = *reinterpret_cast<const uint4 *>(y + off);
#pragma unroll
            for (int j = 0; j < V; ++j) s[j] += to_f32<DT>(v.e[j]);
          } else {
            s[0] += to_f32<DT>(y[off]);
          }
        }
    const long long ooff = i * V;  // output is dense NDHWC in the same order
    if constexpr (VECTOR) {
      Vec16<DT> v;
#pragma unroll
      for (int j = 0; j < V; ++j) v.e[j] = from_f32<DT>(s[j] * scale);
      *reinterpret_cast<uint4 *>(p + ooff) = v.u;
    } else {
      p[ooff] = from_f32<DT>(s[0] * scale);
    }
  }
}

template <int DT, bool VECTOR>
__global__ __launch_bounds__(256) void avgpool_bwd_kernel(const typename Store<DT>::T *__restrict__ dp,
                                                          typename Store<DT>::T *__restrict__ dy,
                                                          int d, int h, int w, int c, int k,
                                                          int od, int oh, int ow, long long items) {
  using T = typename Store<DT>::T;
  constexpr int V = VECTOR ? Store<DT>::VEC : 1;
  const int cg_n = c / V;
  const float scale = 1.f / (float)(k * k * k);
  const long long stride = (long long)gridDim.x * 256;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < items; i += stride) {
    long long t = i;
    const int cg = (int)(t % cg_n); t /= cg_n;
    const int x_ = (int)(t % w); t /= w;
    const int y_ = (int)(t % h); t /= h;
    const int z_ = (int)(t % d);
    const int n = (int)(t / d);
    const int pz = z_ / k, py = y_ / k, px = x_ / k;
    const bool cov = pz < od && py < oh && px < ow;
    const long long poff = ((((long long)n * od + pz) * oh + py) * ow + px) * c + cg * V;
    if constexpr (VECTOR) {
      Vec16<DT> v;
      if (cov) {
        v.u = *reinterpret_cast<const uint4 *>(dp + poff);
#pragma unroll
        for (int j = 0; j < V; ++j) v.e[j] = from_f32<DT>(to_f32<DT>(v.e[j]) * scale);
      } else {
        v.u = make_uint4(0, 0, 0, 0);
      }
      *reinterpret_cast<uint4 *>(dy + i * V) = v.u;
    } else {
      dy[i] = cov ? from_f32<DT>(to_f32<DT>(dp[poff]) * scale) : from_f32<DT>(0.f);
    }
  }
}

// 2^3 windows with whole 16-byte vectors and every offset below 2^31 (the
// bf16 and fp32 fast paths).  Forward: one thread per (pooled voxel, vector),
// its eight loads issued together.  Backward: one thread per (batch, pooled
// plane, pooled row, vector of an input row): it loads the covering pooled
// vector once and stores it, scaled by 1/8, into the four input rows of the
// window, so every store instruction of a wave writes a contiguous 1 KiB;
// the planes, rows and columns that no window covers (odd extents) get
// zeros.  Items are decoded with launch-time divisors.
template <int DT, bool NT>
__global__ __launch_bounds__(256) void avgpool2_fwd_vec_kernel(const typename Store<DT>::T *__restrict__ y,
                                                               typename Store<DT>::T *__restrict__ p, int d, int h,
                                                               int w, int c, FastDiv fcg, FastDiv fow, FastDiv foh,
                                                               FastDiv fod, int items) {
  constexpr int V = Store<DT>::VEC;
  const int i = (int)blockIdx.x * 256 + threadIdx.x;
  if (i >= items) return;
  const int t1 = fdiv(i, fcg), t2 = fdiv(t1, fow), t3 = fdiv(t2, foh), n = fdiv(t3, fod);
  const int cg = i - t1 * (int)fcg.div, x_ = t1 - t2 * (int)fow.div, y_ = t2 - t3 * (int)foh.div;
  const int z_ = t3 - n * (int)fod.div;
  const int base = (((n * d + 2 * z_) * h + 2 * y_) * w + 2 * x_) * c + V * cg;
  Vec16<DT> v[8];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int e = 0; e < 2; ++e)
        v[4 * a + 2 * b + e].u = ld16<NT>(y + base + ((a * h + b) * w + e) * c);
  float sum[V];
#pragma unroll
  for (int j = 0; j < V; ++j) sum[j] = 0.f;
#pragma unroll
  for (int u = 0; u < 8; ++u)
#pragma unroll
    for (int j = 0; j < V; ++j) sum[j] += to_f32<DT>(v[u].e[j]);
  Vec16<DT> o;
#pragma unroll
  for (int j = 0; j < V; ++j) o.e[j] = from_f32<DT>(sum[j] * 0.125f);
  st16<NT>(p + V * i, o.u);  // output is dense NDHWC in item order
}

template <int DT, bool NT>
__global__ __launch_bounds__(256) void avgpool2_bwd_vec_kernel(const typename Store<DT>::T *__restrict__ dp,
                                                               typename Store<DT>::T *__restrict__ dy, int d, int h,
                                                               int w, int c, int od, int oh, int ow, FastDiv frow,
                                                               FastDiv fhc, FastDiv fdc, FastDiv fcg, int items) {
  constexpr int V = Store<DT>::VEC;
  const int i = (int)blockIdx.x * 256 + threadIdx.x;
  if (i >= items) return;
  // frow = vectors per input row, fhc / fdc = pooled rows / planes including an uncovered last one
  const int t = fdiv(i, frow), t2 = fdiv(t, fhc), n = fdiv(t2, fdc);
  const int j = i - t * (int)frow.div, py = t - t2 * (int)fhc.div, pz = t2 - n * (int)fdc.div;
  const int xv = fdiv(j, fcg), cg = j - xv * (int)fcg.div, px = xv >> 1;
  Vec16<DT> v;
  if (pz < od && py < oh && px < ow) {
    v.u = ld16<NT>(dp + (((n * od + pz) * oh + py) * ow + px) * c + V * cg);
#pragma unroll
    for (int k = 0; k < V; ++k) v.e[k] = from_f32<DT>(to_f32<DT>(v.e[k]) * 0.125f);
  } else {
    v.u = make_uint4(0, 0, 0, 0);
  }
  const int base = ((n * d + 2 * pz) * h + 2 * py) * w * c + V * j;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
      if (2 * pz + a < d && 2 * py + b < h) st16<NT>(dy + base + (a * h + b) * w * c, v.u);
}

template <int DT, bool BWD>
hipError_t pool_t(int n, int d, int h, int w, int c, int k, const void *src, void *dst,
                  hipStream_t st) {
  using T = typename Store<DT>::T;
  const int od = (d - k) / k + 1, oh = (h - k) / k + 1, ow = (w - k) / k + 1;
  const bool vec = c % Store<DT>::VEC == 0;
  const int V = vec ? Store<DT>::VEC : 1;
  const long long vox = BWD ? (long long)n * d * h * w : (long long)n * od * oh * ow;
  const long long items = vox * (c / V);
  if (items == 0) return hipSuccess;
  // 2^3 windows, whole 16-byte vectors, offsets below 2^31: the vector kernels
  const long long elems = (long long)n * d * h * w * c;
  if (k == 2 && vec && elems < (1LL << 31)) {
    const int cgn = c / V;
    const bool nt = elems * (long long)sizeof(T) >= kStreamBytes;
    if (BWD) {
      const int dc = (d + 1) / 2, hc = (h + 1) / 2;
      const long long its = (long long)n * dc * hc * w * cgn;
      hipLaunchKernelGGL((nt ? avgpool2_bwd_vec_kernel<DT, true> : avgpool2_bwd_vec_kernel<DT, false>),
                         dim3((int)((its + 255) / 256)), dim3(256), 0, st,
                         (const T *)src, (T *)dst, d, h, w, c, od, oh, ow, make_fastdiv(w * cgn), make_fastdiv(hc),
                         make_fastdiv(dc), make_fastdiv(cgn), (int)its);
    } else {
      hipLaunchKernelGGL((nt ? avgpool2_fwd_vec_kernel<DT, true> : avgpool2_fwd_vec_kernel<DT, false>),
                         dim3((int)((items + 255) / 256)), dim3(256), 0, st,
                         (const T *)src, (T *)dst, d, h, w, c, make_fastdiv(cgn), make_fastdiv(ow), make_fastdiv(oh),
                         make_fastdiv(od), (int)items);
    }
    return hipGetLastError();
  }
  const int blocks = (int)std::min<long long>((items + 255) / 256, 256LL * 64);
  if (BWD) {
    if (vec)
      hipLaunchKernelGGL((avgpool_bwd_kernel<DT, true>), dim3(blocks), dim3(256), 0, st,
                         (const T *)src, (T *)dst, d, h, w, c, k, od, oh, ow, items);
    else
      hipLaunchKernelGGL((avgpool_bwd_kernel<DT, false>), dim3(blocks), dim3(256), 0, st,
                         (const T *)src, (T *)dst, d, h, w, c, k, od, oh, ow, items);
  } else {
    if (vec)
      hipLaunchKernelGGL((avgpool_fwd_kernel<DT, true>), dim3(blocks), dim3(256), 0, st,
                         (const T *)src, (T *)dst, d, h, w, c, k, od, oh, ow, items);
    else
      hipLaunchKernelGGL((avgpool_fwd_kernel<DT, false>), dim3(blocks), dim3(256), 0, st,
                         (const T *)src, (T *)dst, d, h, w, c, k, od, oh, ow, items);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_avgpool_fwd(int n, int d, int h, int w, int c, int k, int dtype, const void *y,
                              void *p, hipStream_t st) {
  return dtype == DT_BF16 ? pool_t<DT_BF16, false>(n, d, h, w, c, k, y, p, st)
                          : pool_t<DT_F32, false>(n, d, h, w, c, k, y, p, st);
}

hipError_t launch_avgpool_bwd(int n, int d, int h, int w, int c, int k, int dtype, const void *dp,
                              void *dy, hipStream_t st) {
  return dtype == DT_BF16 ? pool_t<DT_BF16, true>(n, d, h, w, c, k, dp, dy, st)
                          : pool_t<DT_F32, true>(n, d, h, w, c, k, dp, dy, st);
}

}  // namespace cf
