// reduce.hip -- deterministic column sums of per-workgroup partials (gfx950).
//
// Split reductions (weight gradient slices, bias-gradient workgroup rows)
// leave a [rows][cols] fp32 matrix of partials; out[c] = sum_r part[r][c].
// Every such sum in the library goes through one kernel that takes a batch of
// independent jobs (one launch for all the gradient sums of a training step
// when the caller defers them).  A workgroup owns consecutive columns of one
// job and splits each column's rows over PH phases (thread (phase, col): rows
// phase, phase + PH, ..., summed in ascending order with independent loads in
// flight); the phases are then combined by a fixed binary tree in LDS.  PH is
// a function of (rows, cols) only, and a thread that owns four columns (16-byte
// loads, for wide aligned matrices) sums each of them in exactly that order,
// so the result bits depend on (rows, cols) and the data alone: bitwise
// reproducible, and identical whether a job runs alone or in a batch.

#include "cf_common.h"
#include "cf_kernels.h"

namespace cf {
namespace {

constexpr int MAX_JOBS = 16;

struct RedJob {
  const float *part;
  float *out;
  int rows, cols;
  int ph;      // phases (power of two, <= 64)
  int vec4;    // a thread owns four consecutive columns
  int block0;  // first workgroup of the job
};

struct RedBatch {
  int n;
  RedJob job[MAX_JOBS];
};

__global__ __launch_bounds__(256) void sum_batch_kernel(const RedBatch b) {
  __shared__ float4 red[256];
  int j = 0;
  while (j + 1 < b.n && (int)blockIdx.x >= b.job[j + 1].block0) ++j;
  const RedJob &J = b.job[j];
  const int tid = threadIdx.x, PH = J.ph, CPB = 256 / PH;
  const int cl = tid % CPB, ph = tid / CPB;
  const int c = ((int)blockIdx.x - J.block0) * CPB + cl;  // column (or column quad)
  const int rows = J.rows;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  if (J.vec4) {
    const int cols4 = J.cols >> 2;
    const float4 *part = reinterpret_cast<const float4 *>(J.part);
    if (c < cols4) {
      int r = ph;
      // four independent loads per iteration, added in row order
      for (; r + 3 * PH < rows; r += 4 * PH) {
        const float4 a0 = part[(long long)r * cols4 + c];
        const float4 a1 = part[(long long)(r + PH) * cols4 + c];
        const float4 a2 = part[(long long)(r + 2 * PH) * cols4 + c];
        const float4 a3 = part[(long long)(r + 3 * PH) * cols4 + c];
        s.x += a0.x; s.y += a0.y; s.z += a0.z; s.w += a0.w;
        s.x += a1.x; s.y += a1.y; s.z += a1.z; s.w += a1.w;
        s.x += a2.x; s.y += a2.y; s.z += a2.z; s.w += a2.w;
        s.x += a3.x; s.y += a3.y; s.z += a3.z; s.w += a3.w;
      }
      for (; r < rows; r += PH) {
        const float4 a = part[(long long)r * cols4 + c];
        s.x += a.x; s.y += a.y; s.z += a.z; s.w += a.w;
      }
    }
  } else {
    const int cols = J.cols;
    const float *part = J.part;
    if (c < cols) {
      int r = ph;
      for (; r + 3 * PH < rows; r += 4 * PH) {
        const float a0 = part[(long long)r * cols + c];
        const float a1 = part[(long long)(r + PH) * cols + c];
        const float a2 = part[(long long)(r + 2 * PH) * cols + c];
        const float a3 = part[(long long)(r + 3 * PH) * cols + c];
        s.x += a0;
        s.x += a1;
        s.x += a2;
        s.x += a3;
      }
      for (; r < rows; r += PH) s.x += part[(long long)r * cols + c];
    }
  }
  red[tid] = s;
  __syncthreads();
  for (int st = PH / 2; st > 0; st /= 2) {
    if (ph < st) {
      const float4 o = red[tid + st * CPB];
      float4 m = red[tid];
      m.x += o.x; m.y += o.y; m.z += o.z; m.w += o.w;
      red[tid] = m;
    }
    __syncthreads();
  }
  if (ph == 0) {
    if (J.vec4) {
      if (c < (J.cols >> 2)) reinterpret_cast<float4 *>(J.out)[c] = red[tid];
    } else if (c < J.cols) {
      J.out[c] = red[tid].x;
    }
  }
}

thread_local SumCollector *g_collector = nullptr;

}  // namespace

void set_sum_collector(SumCollector *c) { g_collector = c; }

hipError_t launch_sum_batch(const SumJob *jobs, int n, hipStream_t st) {
  for (int b0 = 0; b0 < n; b0 += MAX_JOBS) {
    RedBatch b{};
    int blocks = 0;
    for (int i = b0; i < n && b.n < MAX_JOBS; ++i) {
      const SumJob &s = jobs[i];
      if (s.cols <= 0) continue;
      RedJob &J = b.job[b.n++];
      J.part = s.part;
      J.out = s.out;
      J.rows = s.rows;
      J.cols = s.cols;
      // phases: each thread sums ~4 rows of a narrow matrix (few workgroups: the
      // serial chain is the latency), ~64 of a wide one (fewer, longer row
      // segments per workgroup: measured fastest on the stack's partials); at
      // most 64 phases
      const int per = s.cols < 256 ? 4 : 64;
      int ph = 1;
      while (ph < 64 && (long long)ph * per < s.rows) ph *= 2;
      J.ph = ph;
      J.vec4 = (s.cols % 4 == 0 && s.cols >= 256 && ((uintptr_t)s.part & 15) == 0 && ((uintptr_t)s.out & 15) == 0);
      const int units = J.vec4 ? s.cols / 4 : s.cols;
      const int cpb = 256 / ph;
      J.block0 = blocks;
      blocks += (units + cpb - 1) / cpb;
    }
    if (b.n == 0) continue;
    hipLaunchKernelGGL(sum_batch_kernel, dim3(blocks), dim3(256), 0, st, b);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_sum_rows(const float *part, float *out, int rows, int cols, hipStream_t st) {
  if (cols <= 0) return hipSuccess;
  if (g_collector) {  // deferred: the caller reduces later, batched with other jobs
    if (g_collector->n >= SumCollector::CAP) return hipErrorInvalidValue;
    g_collector->job[g_collector->n++] = SumJob{part, out, rows, cols};
    return hipSuccess;
  }
  const SumJob j{part, out, rows, cols};
  return launch_sum_batch(&j, 1, st);
}

}  // namespace cf
