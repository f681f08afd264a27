// conv_smallc_pair.hip -- bf16 first-layer forward with the fused pooling
// epilogue, built on voxel-pair windows (gfx950).
//
// The first CosmoFlow layer (Section III-A) convolves the one-channel density
// cube with 3^3 taps into 16 channels, followed by bias, leaky ReLU and the
// 2^3 average pool.  With one input channel the im2col row of an output voxel
// is 27 scattered values; assembling it element by element from LDS costs
// more issue slots than the MFMAs it feeds.  Here the contraction is arranged
// so that every operand fragment is a run of four consecutive input voxels:
//
//   v_mfma_f32_32x32x16_bf16:  D (32 x 32) += A (32 x 16) . B (16 x 32)
//   A row m     = a pair of neighbouring output voxels (w0, w0 + 1), w0 even,
//                 of one (d, h) line;
//   A K slots   = for two (kd, kh) kernel rows, the four input voxels
//                 w0 - p .. w0 - p + 3 (p = leading pad): one 8-byte LDS read
//                 per kernel row;
//   B column n  = (output voxel w0 + e, channel co), n = 16 e + co;
//   B[(row, s), (e, co)] = W[kd, kh, s - e, co] / 8 when 0 <= s - e <= 2,
//                 else 0: a banded copy of the weights, so one window serves
//                 both voxels of the pair.
// Three MFMAs take the nine (kd, kh) rows and a tenth row for the bias (A = 1,
// B = the bias split into two bf16 parts, as the other first-layer kernel
// does), i.e. 64 output voxels x 16 channels.  The 1/8 of the average pool is
// a power of two folded into B, so every partial sum is the unscaled one
// times 1/8 exactly and the epilogue is
//     mask bit = u > 0,   pooled = sum over the window of (u > 0 ? u : alpha u),
// the sum taken as ((1 + alpha) sum u + (1 - alpha) sum |u|) / 2.
//
// Row order m = 8a + 4hb + c, c = 2 dd + hh, pair P = 2a + hb (voxels
// w0 = 2P, 2P + 1 of a 16-voxel segment): the accumulator layout (lane =
// column, registers = rows 8a + 4 (lane / 32) + c) then gives each lane the
// four (dd, hh) values of one e of four pairs, and
//   * the ballot of one register is the 16-bit mask words of four
//     consecutive voxels, bit co of voxel 4a + lane / 16, exactly the mask
//     tensor's layout;
//   * the pooling window's other half (the other e) sits 16 lanes away: one
//     v_permlane16_swap and one add finish two windows at once.
//
// A workgroup stages the zero-padded input halo of a 4 x 8 x 128 output tile
// in LDS once (each row shifted so that every window starts on a 4-byte
// boundary); each wave then computes two (d, h) pair rows of 128 voxels.
// Inputs with an infinite or NaN voxel can spread it one voxel further along
// w than the convolution itself (the banded zeros of B multiply it).

#include "cf_common.h"
#include "cf_kernels.h"

// v_writelane_b32 through the compiler (it places the wait states between the
// compare that writes a ballot and the move that reads it)
__device__ int cf_lane_write(int v, int lane, int old) __asm("llvm.amdgcn.writelane.i32");

namespace cf {
namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2a4_t __attribute__((ext_vector_type(2), aligned(4)));

constexpr int TDP = 2, THP = 4;             // pair rows per tile (d, h)
constexpr int TD = 2 * TDP, TH = 2 * THP;   // output tile (voxels)
constexpr int TW = 128;                     // output voxels per tile along w
constexpr int NSET = TW / 16;               // 16-voxel segments per pair row
constexpr int HD = TD + 2, HH = TH + 2;     // halo rows
constexpr int NR = HD * HH;
constexpr int NVR = (TW + 2 + 7) / 8;       // 16-byte vectors staged per row
constexpr int RP = 320;                     // row pitch (bytes): +16 banks per h, +32 per d
static_assert(NVR * 16 <= RP, "row pitch");
static_assert((HH * RP / 4) % 64 == 32 && (RP / 4) % 64 == 16, "bank layout of the four (dd, hh) rows");

__device__ __forceinline__ float swap_add(float x, float y) {
  // rows of 16 lanes: x's odd rows trade places with y's even rows
  const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, x), __builtin_bit_cast(uint32_t, y),
                                                  false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}

__global__ __launch_bounds__(256) void l1_pair_fwd_kernel(const uint16_t *__restrict__ x,
                                                          const uint16_t *__restrict__ w,
                                                          const float *__restrict__ bias, float alpha,
                                                          uint16_t *__restrict__ out, uint16_t *__restrict__ mask16,
                                                          SmallcParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char halo[NR * RP];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tiles_w = (p.ow + TW - 1) / TW, tiles_h = (p.oh + TH - 1) / TH;
  int t = blockIdx.x;
  const int tw = t % tiles_w; t /= tiles_w;
  const int th = t % tiles_h; t /= tiles_h;
  const int td = t;
  const int n = blockIdx.y;
  const int od0 = td * TD, oh0 = th * TH, ow0 = tw * TW;

  // ---- halo: slot j of row (a, b) holds input (od0 - pd + a, oh0 - ph + b, ow0 - pw + j)
  {
    const int sh = p.pw;  // 0, 1 or 2: the staged row starts sh voxels before a 16-byte chunk
    for (int e = tid; e < NR * NVR; e += 256) {
      const int v = e % NVR, r = e / NVR;
      const int a = r / HH, b = r % HH;
      const int id = od0 - p.pd + a, ih = oh0 - p.ph + b;
      const bool rowok = (unsigned)id < (unsigned)p.d && (unsigned)ih < (unsigned)p.h;
      const int cb = ow0 + 8 * v;  // the chunk's first input column (chunks lie wholly inside or outside)
      const uint16_t *xr = x + (((long long)n * p.d + (rowok ? id : 0)) * p.h + (rowok ? ih : 0)) * p.w;
      uint4 c = make_uint4(0, 0, 0, 0);
      uint32_t pv = 0;  // input columns cb - 2, cb - 1
      if (rowok && cb + 8 <= p.w) c = *reinterpret_cast<const uint4 *>(xr + cb);
      if (rowok && cb >= 2 && cb <= p.w) pv = *reinterpret_cast<const uint32_t *>(xr + cb - 2);
      uint4 o;
      if (sh == 0) {
        o = c;
      } else if (sh == 1) {
        o.x = __builtin_amdgcn_alignbyte(c.x, pv, 2);
        o.y = __builtin_amdgcn_alignbyte(c.y, c.x, 2);
        o.z = __builtin_amdgcn_alignbyte(c.z, c.y, 2);
        o.w = __builtin_amdgcn_alignbyte(c.w, c.z, 2);
      } else {
        o = make_uint4(pv, c.x, c.y, c.z);
      }
      *reinterpret_cast<uint4 *>(halo + r * RP + 16 * v) = o;
    }
  }

  // ---- B fragments (banded weights / 8, bias row), lane = column n, K half kh2
  const int n32 = lane & 31, kh2 = lane >> 5;
  const int e = n32 >> 4, co = n32 & 15;
  bf16x8_t bfr[3];
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    uint16_t vals[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int sg = 4 * j + 2 * kh2 + (q >> 2), s = q & 3;
      float v = 0.f;
      if (sg < 9) {
        const int kw = s - e;
        if (kw >= 0 && kw <= 2) v = bf2f(w[(sg * 3 + kw) * 16 + co]) * 0.125f;
      } else if (sg == 9 && s < 2) {
        const float b = bias[co];
        const float hi = bf2f(f2bf(b));
        v = (s == 0 ? hi : bf2f(f2bf(b - hi))) * 0.125f;
      }
      vals[q] = f2bf(v);  // exact: a bf16 value times a power of two
    }
    Vec16<DT_BF16> pk;
#pragma unroll
    for (int q = 0; q < 8; ++q) pk.e[q] = vals[q];
    bfr[j] = __builtin_bit_cast(bf16x8_t, pk.u);
  }

  // ---- A read addresses: lane row m = 8a + 4hb + c (pair P = 2a + hb, voxel
  // (dd, hh) = c), K half kh2 -> kernel rows sg = 4j + 2 kh2 + tt
  const int m = lane & 31;
  const int am = m >> 3, hbm = (m >> 2) & 1, cm = m & 3;
  const int Pm = 2 * am + hbm;
  int aaddr[5];
#pragma unroll
  for (int k = 0; k < 5; ++k) {
    const int j = k >> 1, tt = k & 1;
    int sg = 4 * j + 2 * kh2 + tt;
    if (sg > 8) sg = 8;  // rows 10, 11 meet zero B columns: any finite input will do
    const int kd = sg / 3, khh = sg % 3;
    aaddr[k] = ((cm >> 1) + kd) * HH * RP + ((cm & 1) + khh) * RP + 4 * Pm;
  }
  const uint32_t ONES = 0x3f803f80u;  // two bf16 1.0: the bias row's A slots

  const float c1 = 0.5f * (1.f + alpha), c2 = 0.5f * (1.f - alpha);
  const int pooled_w0 = ow0 >> 1;
  const int rho = lane >> 4;
  const int Pst = ((rho & 1) << 1) | (rho >> 1);  // pair whose pooled value this lane stores
  __syncthreads();

  for (int pr = wave; pr < TDP * THP; pr += 4) {
    const int pdi = pr / THP, phi = pr % THP;
    const int d0 = od0 + 2 * pdi, h0 = oh0 + 2 * phi;
    if (d0 >= p.od || h0 >= p.oh) continue;  // od, oh even: both rows of the pair exist
    const unsigned char *hb = halo + (2 * pdi * HH + 2 * phi) * RP;
    uint32_t mw[4] = {0u, 0u, 0u, 0u};  // mask row c: dword k = voxels ow0 + 2k, ow0 + 2k + 1
    uint16_t *const prow = out + (((long long)n * p.pod + (d0 >> 1)) * p.poh + (h0 >> 1)) * p.pow_ * 16;
#pragma unroll
    for (int s = 0; s < NSET; ++s) {
      if (ow0 + 16 * s >= p.ow) break;
      u32x2a4_t r[5];
#pragma unroll
      for (int k = 0; k < 5; ++k) r[k] = *reinterpret_cast<const u32x2a4_t *>(hb + aaddr[k] + 32 * s);
      f32x16_t acc = {};
#pragma unroll
      for (int j = 0; j < 3; ++j) {
        u32x4_t av;
        if (j < 2) {
          av = u32x4_t{r[2 * j].x, r[2 * j].y, r[2 * j + 1].x, r[2 * j + 1].y};
        } else {
          av = u32x4_t{r[4].x, r[4].y, ONES, ONES};
        }
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, av), bfr[j], acc, 0, 0, 0);
      }
      // sum of lrelu(u) = c1 * sum(u) + c2 * sum(|u|): the compare feeds only the
      // ballot, and |u| is an operand modifier
      float S[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        float su = 0.f, sa = 0.f;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const float u = acc[4 * a + c];
          const uint64_t bal = __builtin_amdgcn_ballot_w64(u > 0.f);
          mw[c] = cf_lane_write((int)(uint32_t)bal, 8 * s + 2 * a, (int)mw[c]);
          mw[c] = cf_lane_write((int)(uint32_t)(bal >> 32), 8 * s + 2 * a + 1, (int)mw[c]);
          su = c == 0 ? u : su + u;
          sa = c == 0 ? fabsf(u) : sa + fabsf(u);
        }
        S[a] = fmaf(c1, su, c2 * sa);
      }
      const float r01 = swap_add(S[0], S[1]);
      const float r23 = swap_add(S[2], S[3]);
      const uint32_t pk = f2bf2(r01, r23);
      const int pw_ = pooled_w0 + 8 * s + Pst;
      if (pw_ < p.pow_) prow[pw_ * 16 + co] = (uint16_t)(pk & 0xffffu);
      if (pw_ + 4 < p.pow_) prow[(pw_ + 4) * 16 + co] = (uint16_t)(pk >> 16);
    }
    // mask rows (d0 + dd, h0 + hh), c = 2 dd + hh: lane k stores voxels ow0 + 2k, + 1
    if (ow0 + 2 * lane < p.ow) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const long long vrow = (((long long)n * p.od + d0 + (c >> 1)) * p.oh + h0 + (c & 1)) * p.ow;
        *reinterpret_cast<uint32_t *>(mask16 + vrow + ow0 + 2 * lane) = mw[c];
      }
    }
  }
}

}  // namespace

bool l1pair_supported(const ConvShape &s) {
  if (s.dtype != DT_BF16 || s.ci != 1 || s.co != 16) return false;
  if (s.kd != 3 || s.kh != 3 || s.kw != 3 || s.sd != 1 || s.sh != 1 || s.sw != 1) return false;
  if (s.pd < 0 || s.pd > 2 || s.ph < 0 || s.ph > 2 || s.pw < 0 || s.pw > 2) return false;
  if (s.od % 2 || s.oh % 2 || s.ow % 2 || s.od < 2 || s.oh < 2 || s.ow < 2) return false;
  if (s.w % 8) return false;
  const char *e = getenv("CF_L1PAIR");
  return !(e && e[0] == '0');
}

hipError_t launch_l1pair_fwd(const ConvShape &s, const void *x, const void *w, const float *bias, float alpha,
                             void *out, uint16_t *mask, hipStream_t st) {
  SmallcParams p{};
  p.n = s.n; p.d = s.d; p.h = s.h; p.w = s.w; p.ci = s.ci; p.co = s.co;
  p.kd = s.kd; p.kh = s.kh; p.kw = s.kw; p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.od = s.od; p.oh = s.oh; p.ow = s.ow;
  p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
  const long long tiles = (long long)((p.ow + TW - 1) / TW) * ((p.oh + TH - 1) / TH) * ((p.od + TD - 1) / TD);
  if (tiles > 0x7fffffffLL || p.n > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(l1_pair_fwd_kernel, dim3((unsigned)tiles, p.n), dim3(256), 0, st, (const uint16_t *)x,
                     (const uint16_t *)w, bias, alpha, (uint16_t *)out, mask, p);
  return hipGetLastError();
}

}  // namespace cf
