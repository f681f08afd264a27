// reduce.hip -- deterministic column sums of per-workgroup partials (gfx950).
//
// Split reductions (weight gradient slices, bias-gradient workgroup rows)
// leave a [rows][cols] fp32 matrix of partials; out[c] = sum_r part[r][c].
// A workgroup owns CPB consecutive columns and splits the rows of each
// column over PH phases (thread (phase, col): rows phase, phase + PH, ...,
// summed in ascending order with independent loads in flight); the phases
// are then combined by a fixed binary tree in LDS.  The summation order is a
// function of (rows, cols) only, so results are bitwise reproducible, and
// consecutive threads read consecutive columns (coalesced).

#include "cf_common.h"
#include "cf_kernels.h"

namespace cf {
namespace {

template <int PH>
__global__ __launch_bounds__(256) void sum_rows_kernel(const float *__restrict__ part, float *__restrict__ out,
                                                       int rows, int cols) {
  constexpr int CPB = 256 / PH;
  __shared__ float red[256];
  const int tid = threadIdx.x;
  const int cl = tid % CPB, ph = tid / CPB;
  const int c = blockIdx.x * CPB + cl;
  float s = 0.f;
  if (c < cols) {
    int r = ph;
    // four independent loads per iteration, added in row order
    for (; r + 3 * PH < rows; r += 4 * PH) {
      float a0 = part[(long long)r * cols + c];
      float a1 = part[(long long)(r + PH) * cols + c];
      float a2 = part[(long long)(r + 2 * PH) * cols + c];
      float a3 = part[(long long)(r + 3 * PH) * cols + c];
      s += a0;
      s += a1;
      s += a2;
      s += a3;
    }
    for (; r < rows; r += PH) s += part[(long long)r * cols + c];
  }
  red[tid] = s;
  __syncthreads();
#pragma unroll
  for (int st = PH / 2; st > 0; st /= 2) {
    if (ph < st) red[tid] += red[tid + st * CPB];
    __syncthreads();
  }
  if (ph == 0 && c < cols) out[c] = red[tid];
}

// 16-byte variant (cols % 4 == 0, 16-byte aligned rows): thread (phase, q)
// owns four consecutive columns, CQ = 256 / PH quads per workgroup, so a wave
// reads row segments of 16 * CQ bytes with float4 loads.
template <int PH>
__global__ __launch_bounds__(256) void sum_rows4_kernel(const float4 *__restrict__ part, float4 *__restrict__ out,
                                                        int rows, int cols4) {
  constexpr int CQ = 256 / PH;
  __shared__ float4 red[256];
  const int tid = threadIdx.x;
  const int cq = tid % CQ, ph = tid / CQ;
  const int c = blockIdx.x * CQ + cq;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  if (c < cols4) {
    int r = ph;
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
  red[tid] = s;
  __syncthreads();
#pragma unroll
  for (int st = PH / 2; st > 0; st /= 2) {
    if (ph < st) {
      const float4 o = red[tid + st * CQ];
      float4 m = red[tid];
      m.x += o.x; m.y += o.y; m.z += o.z; m.w += o.w;
      red[tid] = m;
    }
    __syncthreads();
  }
  if (ph == 0 && c < cols4) out[c] = red[tid];
}

template <int PH>
hipError_t launch_ph4(const float *part, float *out, int rows, int cols, hipStream_t st) {
  constexpr int CQ = 256 / PH;
  const int cols4 = cols / 4;
  hipLaunchKernelGGL((sum_rows4_kernel<PH>), dim3((cols4 + CQ - 1) / CQ), dim3(256), 0, st,
                     reinterpret_cast<const float4 *>(part), reinterpret_cast<float4 *>(out), rows, cols4);
  return hipGetLastError();
}

template <int PH>
hipError_t launch_ph(const float *part, float *out, int rows, int cols, hipStream_t st) {
  constexpr int CPB = 256 / PH;
  hipLaunchKernelGGL((sum_rows_kernel<PH>), dim3((cols + CPB - 1) / CPB), dim3(256), 0, st, part, out, rows, cols);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sum_rows(const float *part, float *out, int rows, int cols, hipStream_t st) {
  if (cols <= 0) return hipSuccess;
  // wide, 16-byte aligned: float4 columns; phases so that a thread sums ~32 rows,
  // at least 16 (256-byte row segments per wave) once rows are many
  if (cols % 4 == 0 && ((uintptr_t)part & 15) == 0 && ((uintptr_t)out & 15) == 0 && cols >= 256) {
    int ph = 1;
    while (ph < 64 && (long long)ph * 32 < rows) ph *= 2;
    switch (ph) {
      case 1: return launch_ph4<1>(part, out, rows, cols, st);
      case 2: return launch_ph4<2>(part, out, rows, cols, st);
      case 4: return launch_ph4<4>(part, out, rows, cols, st);
      case 8: return launch_ph4<8>(part, out, rows, cols, st);
      case 16: return launch_ph4<16>(part, out, rows, cols, st);
      case 32: return launch_ph4<32>(part, out, rows, cols, st);
      default: return launch_ph4<64>(part, out, rows, cols, st);
    }
  }
  // enough phases that each thread sums at most ~16 rows (~4 when the matrix is
  // narrow: few workgroups, so the serial chain per thread is the latency)
  const int per = cols < 256 ? 4 : 16;
  int ph = 1;
  while (ph < 256 && (long long)ph * per < rows) ph *= 2;
  switch (ph) {
    case 1: return launch_ph<1>(part, out, rows, cols, st);
    case 2: return launch_ph<2>(part, out, rows, cols, st);
    case 4: return launch_ph<4>(part, out, rows, cols, st);
    case 8: return launch_ph<8>(part, out, rows, cols, st);
    case 16: return launch_ph<16>(part, out, rows, cols, st);
    case 32: return launch_ph<32>(part, out, rows, cols, st);
    case 64: return launch_ph<64>(part, out, rows, cols, st);
    case 128: return launch_ph<128>(part, out, rows, cols, st);
    default: return launch_ph<256>(part, out, rows, cols, st);
  }
}

}  // namespace cf
