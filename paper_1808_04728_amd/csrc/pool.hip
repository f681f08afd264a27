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
// The backward pass decodes its items with launch-time divisors in 32-bit
// arithmetic when every index fits (a 64-bit division per input item made it
// ALU-bound); larger tensors take the 64-bit kernel.

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

// 32-bit backward: fc = c / V and fw, fh, fd = the input extents; every element
// offset is below 2^31.  (A 32-bit forward measured no faster than the kernel
// above: its decode is per pooled voxel, eight times fewer items.)
template <int DT>
__global__ __launch_bounds__(256) void avgpool2_bwd32_kernel(const uint16_t *__restrict__ dp, uint16_t *__restrict__ dy,
                                                             int c, int od, int oh, int ow, FastDiv fc, FastDiv fw,
                                                             FastDiv fh, FastDiv fd, int items) {
  const int i = (int)blockIdx.x * 256 + threadIdx.x;
  if (i >= items) return;
  const int t1 = fdiv(i, fc), t2 = fdiv(t1, fw), t3 = fdiv(t2, fh), n = fdiv(t3, fd);
  const int cg = i - t1 * (int)fc.div, x_ = t1 - t2 * (int)fw.div, y_ = t2 - t3 * (int)fh.div;
  const int z_ = t3 - n * (int)fd.div;
  const int pz = z_ >> 1, py = y_ >> 1, px = x_ >> 1;
  Vec16<DT_BF16> v;
  if (pz < od && py < oh && px < ow) {
    v.u = *reinterpret_cast<const uint4 *>(dp + (((n * od + pz) * oh + py) * ow + px) * c + 8 * cg);
#pragma unroll
    for (int j = 0; j < 8; ++j) v.e[j] = f2bf(bf2f(v.e[j]) * 0.125f);
  } else {
    v.u = make_uint4(0, 0, 0, 0);
  }
  *reinterpret_cast<uint4 *>(dy + 8 * i) = v.u;
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
  // bf16 backward, 2^3 windows, whole 16-byte channel groups, offsets below 2^31
  const long long elems = (long long)n * d * h * w * c;
  if constexpr (DT == DT_BF16 && BWD) {
    if (k == 2 && vec && elems < (1LL << 31)) {
      hipLaunchKernelGGL(avgpool2_bwd32_kernel<DT>, dim3((int)((items + 255) / 256)), dim3(256), 0, st,
                         (const uint16_t *)src, (uint16_t *)dst, c, od, oh, ow, make_fastdiv(c / 8),
                         make_fastdiv(w), make_fastdiv(h), make_fastdiv(d), (int)items);
      return hipGetLastError();
    }
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
