// conv_smallc.hip -- first-layer convolution (few input channels) for gfx950.
//
// The first CosmoFlow layer convolves a single-channel density cube
// (Section III-A; 1 -> 16 channels, 3^3 taps).  With C_in * k^3 <= 128 the
// whole reduction fits in a handful of MFMA K-steps, so each 16-voxel x
// 16-channel MFMA tile needs its im2col row only once: a workgroup stages the
// zero-padded input halo of a 4x8x32-voxel output tile in LDS, and every lane
// gathers its 8 (bf16) or 1 (fp32) K-values of the im2col row straight from
// the halo with precomputed tap offsets.  Weights stay in registers for the
// whole tile.
//
// The 16 rows of one MFMA tile are a 2x2x4 (d,h,w) voxel brick, so the MFMA
// output layout (lane group q holds rows 4q..4q+3) puts each lane's four
// values on one w-row of the brick: the 2^3 average pool is two in-lane adds
// plus two cross-lane adds, and the fused epilogue
//     u = acc + bias,  y = lrelu(u),  mask bit = (u > 0),  p = pool(y)
// writes only the pooled output and the 1-bit slope mask (the forward layer's
// full-resolution activation never reaches HBM).  The unfused variant stores z.

#include "cf_common.h"
#include "cf_kernels.h"

#include <type_traits>

namespace cf {
namespace {

constexpr int TD = 4, TH = 8, TW = 32;       // output tile (voxels)
constexpr int NBLK = (TD / 2) * (TH / 2) * (TW / 4);  // 64 MFMA bricks of 2x2x4
constexpr int KMAXE = 4;                      // kernel extent limit per dimension
constexpr int HALO_MAX = (TD + KMAXE - 1) * (TH + KMAXE - 1) * (TW + KMAXE - 1);

template <int DT, int CIN, int NF, int KE, bool FUSED>
__global__ __launch_bounds__(256) void conv_smallc_fwd_kernel(
    const typename Store<DT>::T *__restrict__ x, const typename Store<DT>::T *__restrict__ w,
    const float *__restrict__ bias, float alpha, typename Store<DT>::T *__restrict__ out,
    uint16_t *__restrict__ mask16, SmallcParams p) {
  using T = typename Store<DT>::T;
  constexpr int COUT = 16 * NF;
  constexpr bool BF = DT == DT_BF16;
  constexpr int KPER = BF ? 32 : 4;  // K per MFMA
  __shared__ __attribute__((aligned(16))) T halo[HALO_MAX * CIN];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tiles_w = (p.ow + TW - 1) / TW, tiles_h = (p.oh + TH - 1) / TH;
  int t = blockIdx.x;
  const int tw = t % tiles_w; t /= tiles_w;
  const int th = t % tiles_h; t /= tiles_h;
  const int td = t;
  const int n = blockIdx.y;
  const int od0 = td * TD, oh0 = th * TH, ow0 = tw * TW;
  // cubic kernel of extent KE: every halo / tap index below divides by constants
  constexpr int HD = TD + KE - 1, HH = TH + KE - 1, HW = TW + KE - 1;
  constexpr int K = KE * KE * KE * CIN;
  constexpr int ksteps = (K + KPER - 1) / KPER;

  // ---- stage the zero-padded input halo ------------------------------------
  constexpr int helems = HD * HH * HW * CIN;
  for (int e = tid; e < helems; e += 256) {
    int c = e % CIN;
    int v = e / CIN;
    int a = v / (HH * HW), b = (v / HW) % HH, cc = v % HW;
    int id = od0 - p.pd + a, ih = oh0 - p.ph + b, iw = ow0 - p.pw + cc;
    T val = from_f32<DT>(0.f);
    if ((unsigned)id < (unsigned)p.d && (unsigned)ih < (unsigned)p.h && (unsigned)iw < (unsigned)p.w)
      val = x[((((long long)n * p.d + id) * p.h + ih) * p.w + iw) * CIN + c];
    halo[e] = val;
  }

  // ---- per-lane constants: im2col tap offsets and the weight fragments ------
  const int r = lane & 15, q = lane >> 4;
  // brick row r -> voxel (dd, hh, ww) inside the 2x2x4 brick
  const int m_off = (((r >> 3) * HH + ((r >> 2) & 1)) * HW + (r & 3)) * CIN;
  constexpr int KS_MAX = ksteps;
  constexpr int JPER = BF ? 8 : 1;  // K-values per lane per MFMA
  int toff[KS_MAX][JPER];
#pragma unroll
  for (int ks = 0; ks < KS_MAX; ++ks)
#pragma unroll
    for (int j = 0; j < JPER; ++j) {
      int kg = ks * KPER + (BF ? 8 * q + j : q);
      int off = 0;
      if (kg < K) {
        int tap = kg / CIN, c = kg % CIN;
        int a = tap / (KE * KE), b = (tap / KE) % KE, cc = tap % KE;
        off = ((a * HH + b) * HW + cc) * CIN + c;
      }
      toff[ks][j] = off;
    }
  using AFrag = typename std::conditional<BF, bf16x8_t, float>::type;
  AFrag bw[KS_MAX][NF];
#pragma unroll
  for (int ks = 0; ks < KS_MAX; ++ks)
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      if constexpr (BF) {
        Vec16<DT_BF16> v;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          int kg = ks * 32 + 8 * q + j;
          v.e[j] = kg < K ? w[(long long)kg * COUT + 16 * f + r] : (uint16_t)0;
        }
        bw[ks][f] = __builtin_bit_cast(bf16x8_t, v.u);
      } else {
        int kg = ks * 4 + q;
        bw[ks][f] = kg < K ? (float)w[(long long)kg * COUT + 16 * f + r] : 0.f;
      }
    }
  float bz[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) bz[f] = FUSED ? bias[16 * f + r] : 0.f;
  __syncthreads();

  // ---- 64 bricks per tile, 16 per wave --------------------------------------
  for (int bi = wave; bi < NBLK; bi += 4) {
    const int bd = bi / ((TH / 2) * (TW / 4)), bh = (bi / (TW / 4)) % (TH / 2), bwi = bi % (TW / 4);
    const int base = ((2 * bd * HH + 2 * bh) * HW + 4 * bwi) * CIN + m_off;
    f32x4_t acc[NF];
#pragma unroll
    for (int f = 0; f < NF; ++f) acc[f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS_MAX; ++ks) {
      if (ks >= ksteps) break;
      AFrag a;
      if constexpr (BF) {
        Vec16<DT_BF16> v;
#pragma unroll
        for (int j = 0; j < 8; ++j) v.e[j] = halo[base + toff[ks][j]];
        a = __builtin_bit_cast(bf16x8_t, v.u);
      } else {
        a = halo[base + toff[ks][0]];
      }
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        if constexpr (BF)
          acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bw[ks][f], acc[f], 0, 0, 0);
        else
          acc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bw[ks][f], acc[f], 0, 0, 0);
      }
    }
    // this lane's outputs: brick rows 4q+j = voxel (dd, hh) = (q>>1, q&1), ww = j
    const int vd = od0 + 2 * bd + (q >> 1), vh = oh0 + 2 * bh + (q & 1), vw0 = ow0 + 4 * bwi;
    const bool row_ok = vd < p.od && vh < p.oh;
    const long long vrow = (((long long)n * p.od + vd) * p.oh + vh) * p.ow;
    if constexpr (!FUSED) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (!row_ok || vw0 + j >= p.ow) continue;
#pragma unroll
        for (int f = 0; f < NF; ++f) out[(vrow + vw0 + j) * COUT + 16 * f + r] = from_f32<DT>(acc[f][j]);
      }
    } else {
      const int pd_ = (od0 + 2 * bd) >> 1, ph_ = (oh0 + 2 * bh) >> 1, pw0 = vw0 >> 1;
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        float y[4];
        unsigned long long bal[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float u = acc[f][j] + bz[f];
          y[j] = u > 0.f ? u : alpha * u;
          bal[j] = __ballot(u > 0.f);
        }
        // mask: lanes 16q + j (j < 4) store the 16 channel bits of voxel (q, j)
        if (r < 4 && row_ok && vw0 + r < p.ow) {
          unsigned long long b = r == 0 ? bal[0] : r == 1 ? bal[1] : r == 2 ? bal[2] : bal[3];
          mask16[(vrow + vw0 + r) * NF + f] = (uint16_t)((b >> (16 * q)) & 0xffffu);
        }
        float s0 = y[0] + y[1], s1 = y[2] + y[3];
        s0 += __shfl_xor(s0, 16);
        s1 += __shfl_xor(s1, 16);
        s0 += __shfl_xor(s0, 32);
        s1 += __shfl_xor(s1, 32);
        if (q < 2 && pd_ < p.pod && ph_ < p.poh && pw0 + q < p.pow_) {
          float s = q == 0 ? s0 : s1;
          long long pv = (((long long)n * p.pod + pd_) * p.poh + ph_) * p.pow_ + pw0 + q;
          out[pv * COUT + 16 * f + r] = from_f32<DT>(s * 0.125f);
        }
      }
    }
  }
}

template <int DT, int CIN, int NF, int KE, bool FUSED>
hipError_t launch_t(const SmallcParams &p, const void *x, const void *w, const float *bias, float alpha,
                    void *out, uint16_t *mask, hipStream_t st) {
  using T = typename Store<DT>::T;
  if constexpr (KE * KE * KE * CIN > (DT == DT_BF16 ? 128 : 32)) {
    return hipErrorInvalidValue;  // not instantiated: the reduction is too long for this kernel
  } else {
  const int tiles = ((p.ow + TW - 1) / TW) * ((p.oh + TH - 1) / TH) * ((p.od + TD - 1) / TD);
  hipLaunchKernelGGL((conv_smallc_fwd_kernel<DT, CIN, NF, KE, FUSED>), dim3(tiles, p.n), dim3(256), 0, st,
                     (const T *)x, (const T *)w, bias, alpha, (T *)out, mask, p);
  return hipGetLastError();
  }
}

template <int DT, bool FUSED>
hipError_t dispatch(const SmallcParams &p, const void *x, const void *w, const float *bias, float alpha,
                    void *out, uint16_t *mask, hipStream_t st) {
  const int nf = p.co / 16;
#define CF_SMALLC_CASE(CI, NFV, KEV) \
  if (p.ci == CI && nf == NFV && p.kd == KEV) return launch_t<DT, CI, NFV, KEV, FUSED>(p, x, w, bias, alpha, out, mask, st);
#define CF_SMALLC_KE(KEV) \
  CF_SMALLC_CASE(1, 1, KEV) CF_SMALLC_CASE(1, 2, KEV) CF_SMALLC_CASE(2, 1, KEV) CF_SMALLC_CASE(4, 1, KEV) \
  CF_SMALLC_CASE(4, 2, KEV)
  CF_SMALLC_KE(2) CF_SMALLC_KE(3) CF_SMALLC_KE(4)
#undef CF_SMALLC_KE
#undef CF_SMALLC_CASE
  return hipErrorInvalidValue;
}

}  // namespace

bool smallc_supported(const ConvShape &s, bool fused) {
  if (s.sd != 1 || s.sh != 1 || s.sw != 1) return false;
  if (s.kd != s.kh || s.kd != s.kw || s.kd < 2 || s.kd > KMAXE) return false;  // cubic 2^3..4^3
  const int nf = s.co / 16;
  if (s.co % 16 != 0) return false;
  const bool shape_ok = (s.ci == 1 && (nf == 1 || nf == 2)) || (s.ci == 2 && nf == 1) ||
                        (s.ci == 4 && (nf == 1 || nf == 2));
  if (!shape_ok) return false;
  const int K = s.kd * s.kh * s.kw * s.ci;
  if (K > (s.dtype == DT_BF16 ? 128 : 32)) return false;
  if (fused && (s.oh < 2 || s.od < 2 || s.ow < 2)) return false;
  return true;
}

hipError_t launch_conv_fwd_smallc(const ConvShape &s, const void *x, const void *w, const float *bias,
                                  float alpha, void *out, uint16_t *mask, bool fused, hipStream_t st) {
  SmallcParams p{};
  p.n = s.n; p.d = s.d; p.h = s.h; p.w = s.w; p.ci = s.ci; p.co = s.co;
  p.kd = s.kd; p.kh = s.kh; p.kw = s.kw; p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.od = s.od; p.oh = s.oh; p.ow = s.ow;
  p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
  if (s.dtype == DT_BF16)
    return fused ? dispatch<DT_BF16, true>(p, x, w, bias, alpha, out, mask, st)
                 : dispatch<DT_BF16, false>(p, x, w, bias, alpha, out, mask, st);
  return fused ? dispatch<DT_F32, true>(p, x, w, bias, alpha, out, mask, st)
               : dispatch<DT_F32, false>(p, x, w, bias, alpha, out, mask, st);
}

}  // namespace cf
