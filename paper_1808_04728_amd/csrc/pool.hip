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

#include "cf_common.h"
#include "cf_kernels.h"

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
