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

template <int PH>
hipError_t launch_ph(const float *part, float *out, int rows, int cols, hipStream_t st) {
  constexpr int CPB = 256 / PH;
  hipLaunchKernelGGL((sum_rows_kernel<PH>), dim3((cols + CPB - 1) / CPB), dim3(256), 0, st, part, out, rows, cols);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sum_rows(const float *part, float *out, int rows, int cols, hipStream_t st) {
  if (cols <= 0) return hipSuccess;
  // enough phases that each thread sums at most ~16 rows
  int ph = 1;
  while (ph < 256 && (long long)ph * 16 < rows) ph *= 2;
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
