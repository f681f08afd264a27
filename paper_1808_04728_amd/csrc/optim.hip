// optim.hip -- the parameter update of CosmoFlow's training step (Section
// III-B): Adam on a gradient rescaled per parameter group by LARC's clipped
// local rate, with a global rate on a linear (power 1) decay.
//
// Two launches, both HBM-bound streaming passes over flat fp32 arrays:
//   norms   every workgroup owns one chunk of one group and writes the fp64
//           sums of squares of v and g over it (a fixed-order tree);
//   update  every workgroup first sums its group's chunk partials in the
//           same fixed order (so all chunks of a group see the same bits),
//           forms eta_t, the trust ratio eta* and its clip eta+, then
//           updates v, m, s of its chunk in one pass (and writes a bf16
//           copy of v when asked).
// Scalars and the per-element update are computed in fp64 and rounded once
// on the fp32 stores: the pass is bound by HBM and launch latency, so the
// wider arithmetic costs nothing measurable.
//
// A group's chunk is kChunk << shift elements (one 16-byte vector per
// thread and array when shift = 0), with the smallest shift that leaves at
// most 256 chunks, so the second pass re-reads at most 256 partial pairs
// per workgroup (one per thread).

#include "cf_common.h"
#include "cf_kernels.h"

namespace cf {
namespace {

constexpr int kThreads = 256;
constexpr long long kChunk = 4 * kThreads;

__device__ __forceinline__ int find_group(const OptGroups &G, int b) {
  // last l with chunk0[l] <= b; groups without chunks are never returned,
  // since the following group starts at the same chunk
  int lo = 0, hi = G.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (G.chunk0[mid] <= b) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Sum of two doubles over the workgroup, in a fixed order: butterfly within
// each wave, then the four wave results as (w0 + w1) + (w2 + w3).
__device__ __forceinline__ void block_sum2(double &a, double &b, double *red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    a += __shfl_xor(a, o, 64);
    b += __shfl_xor(b, o, 64);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[2 * wave] = a;
    red[2 * wave + 1] = b;
  }
  __syncthreads();
  a = (red[0] + red[2]) + (red[4] + red[6]);
  b = (red[1] + red[3]) + (red[5] + red[7]);
}

__global__ __launch_bounds__(kThreads) void adam_norms_kernel(OptGroups G, const float *__restrict__ v,
                                                              const float *__restrict__ g,
                                                              double *__restrict__ part) {
  __shared__ double red[8];
  const int b = blockIdx.x;
  const int l = find_group(G, b);
  const long long span = kChunk << G.shift[l];
  const long long beg = G.off[l] + (long long)(b - G.chunk0[l]) * span;
  const long long end = min(beg + span, G.off[l + 1]);
  double vv = 0.0, gg = 0.0;
  for (long long e = beg + 4LL * threadIdx.x; e < end; e += 4LL * kThreads) {
    if (e + 4 <= end) {
      const float4 a = *reinterpret_cast<const float4 *>(v + e);
      const float4 c = *reinterpret_cast<const float4 *>(g + e);
      vv += (double)a.x * a.x + (double)a.y * a.y + (double)a.z * a.z + (double)a.w * a.w;
      gg += (double)c.x * c.x + (double)c.y * c.y + (double)c.z * c.z + (double)c.w * c.w;
    } else {
      for (long long i = e; i < end; ++i) {
        vv += (double)v[i] * v[i];
        gg += (double)g[i] * g[i];
      }
    }
  }
  block_sum2(vv, gg, red);
  if (threadIdx.x == 0) {
    part[2 * b] = vv;
    part[2 * b + 1] = gg;
  }
}

__device__ __forceinline__ void adam_one(double gi, float &vi, float &mi, float &si, double dag, double b1,
                                         double b2, double a_k, double eps) {
  const double gs = dag * gi;
  const double m = b1 * (double)mi + (1.0 - b1) * gs;
  const double s = b2 * (double)si + (1.0 - b2) * gs * gs;
  const double v = (double)vi - a_k * m / (sqrt(s) + eps);
  mi = (float)m;
  si = (float)s;
  vi = (float)v;
}

__global__ __launch_bounds__(kThreads) void adam_update_kernel(OptGroups G, OptHparams hp, long long t,
                                                               float *__restrict__ v, const float *__restrict__ g,
                                                               float *__restrict__ m, float *__restrict__ s,
                                                               uint16_t *__restrict__ v16,
                                                               const double *__restrict__ part) {
  __shared__ double red[8];
  const int b = blockIdx.x;
  const int l = find_group(G, b);
  // the group's squared norms: one partial pair per thread (at most 256 chunks)
  const int c0 = G.chunk0[l], nc = G.chunk0[l + 1] - c0;
  double vv = 0.0, gg = 0.0;
  if ((int)threadIdx.x < nc) {
    vv = part[2 * (c0 + threadIdx.x)];
    gg = part[2 * (c0 + threadIdx.x) + 1];
  }
  block_sum2(vv, gg, red);
  // global rate (linear decay, clamped after t_decay) and Adam's step size
  // with both bias corrections; Adam counts updates from 1
  const double tc = (double)(t < hp.t_decay ? t : hp.t_decay);
  const double eta_t = (hp.eta0 - hp.eta_min) * (1.0 - tc / (double)hp.t_decay) + hp.eta_min;
  const double k = (double)(t + 1);
  const double a_k = eta_t * sqrt(1.0 - pow(hp.beta2, k)) / (1.0 - pow(hp.beta1, k));
  // LARC: trust ratio from the layer norms, fallback when either is zero, clip
  const double vn = sqrt(vv), gn = sqrt(gg);
  const double star = (vn != 0.0 && gn != 0.0) ? hp.coef * vn / gn : hp.fallback;
  const double dag = star < hp.clip ? star : hp.clip;

  const long long span = kChunk << G.shift[l];
  const long long beg = G.off[l] + (long long)(b - c0) * span;
  const long long end = min(beg + span, G.off[l + 1]);
  for (long long e = beg + 4LL * threadIdx.x; e < end; e += 4LL * kThreads) {
    if (e + 4 <= end) {
      float4 vq = *reinterpret_cast<const float4 *>(v + e);
      const float4 gq = *reinterpret_cast<const float4 *>(g + e);
      float4 mq = *reinterpret_cast<const float4 *>(m + e);
      float4 sq = *reinterpret_cast<const float4 *>(s + e);
      adam_one(gq.x, vq.x, mq.x, sq.x, dag, hp.beta1, hp.beta2, a_k, hp.eps_hat);
      adam_one(gq.y, vq.y, mq.y, sq.y, dag, hp.beta1, hp.beta2, a_k, hp.eps_hat);
      adam_one(gq.z, vq.z, mq.z, sq.z, dag, hp.beta1, hp.beta2, a_k, hp.eps_hat);
      adam_one(gq.w, vq.w, mq.w, sq.w, dag, hp.beta1, hp.beta2, a_k, hp.eps_hat);
      *reinterpret_cast<float4 *>(v + e) = vq;
      *reinterpret_cast<float4 *>(m + e) = mq;
      *reinterpret_cast<float4 *>(s + e) = sq;
      if (v16) {
        uint2 o;
        o.x = f2bf2(vq.x, vq.y);
        o.y = f2bf2(vq.z, vq.w);
        *reinterpret_cast<uint2 *>(v16 + e) = o;
      }
    } else {
      for (long long i = e; i < end; ++i) {
        float vi = v[i], mi = m[i], si = s[i];
        adam_one(g[i], vi, mi, si, dag, hp.beta1, hp.beta2, a_k, hp.eps_hat);
        v[i] = vi;
        m[i] = mi;
        s[i] = si;
        if (v16) v16[i] = f2bf(vi);
      }
    }
  }
}

}  // namespace

int plan_opt_groups(int n, const long long *off, OptGroups *G) {
  G->n = n;
  int chunks = 0;
  for (int l = 0; l < n; ++l) {
    const long long len = off[l + 1] - off[l];
    int sh = 0;
    while ((len + (kChunk << sh) - 1) / (kChunk << sh) > 256) ++sh;
    G->off[l] = off[l];
    G->shift[l] = sh;
    G->chunk0[l] = chunks;
    chunks += (int)((len + (kChunk << sh) - 1) / (kChunk << sh));
  }
  G->off[n] = off[n];
  G->chunk0[n] = chunks;
  return chunks;
}

hipError_t launch_adam_larc(const OptGroups &G, int chunks, const OptHparams &hp, long long t, float *v,
                            const float *g, float *m, float *s, uint16_t *v16, double *part, hipStream_t st) {
  if (chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(adam_norms_kernel, dim3(chunks), dim3(kThreads), 0, st, G, (const float *)v, g, part);
  hipLaunchKernelGGL(adam_update_kernel, dim3(chunks), dim3(kThreads), 0, st, G, hp, t, v, g, m, s, v16,
                     (const double *)part);
  return hipGetLastError();
}

}  // namespace cf
