// conv_smallc.hip -- first-layer convolution (few input channels) for gfx950.
//
// The first CosmoFlow layer convolves a single-channel density cube
// (Section III-A; 1 -> 16 channels, 3^3 taps).  With C_in * k^3 <= 128 the
// whole reduction fits in a handful of MFMA K-steps, so each 16-voxel x
// 16-channel MFMA tile needs its im2col row only once: a workgroup stages the
// zero-padded input halo of a 4x8x64-voxel output tile in LDS, and every lane
// gathers its 8 (bf16) or 1 (fp32) K-values of the im2col row straight from
// the halo with precomputed tap offsets.  Weights stay in registers for the
// whole tile.
//
// Voxel order inside an MFMA tile: row r = 4q + j is voxel
// (h = 2 ph + (j >> 1), w = 8 pw + 2q + (j & 1)) of one d-plane, and two
// tiles (d = 2 pd, 2 pd + 1) are computed together.  The MFMA output layout
// (lane group q holds rows 4q .. 4q+3 of one channel) then places the whole
// 2x2x2 pooling window of pooled voxel (pd, ph, 4 pw + q) in one lane, so the
// fused epilogue
//     u = acc + bias,  y = lrelu(u),  mask bit = (u > 0),  p = mean of 8 y
// is in-lane arithmetic: one coalesced 128-byte store per tile pair for the
// pooled output and four 16-byte stores for the 1-bit slope mask.  The
// full-resolution activation never reaches HBM.  The unfused variant stores z.

#include "cf_common.h"
#include "cf_kernels.h"

#include <type_traits>

namespace cf {
namespace {

constexpr int TD = 4, TH = 8, TW = 64;                   // output tile (voxels)
constexpr int NPAIR = (TD / 2) * (TH / 2) * (TW / 8);    // 64 tile pairs of 2 x (2x2x8) voxels
constexpr int KMAXE = 4;                                  // kernel extent limit per dimension

template <int DT, int CIN, int NF, int KE, bool FUSED>
__global__ __launch_bounds__(256) void conv_smallc_fwd_kernel(
    const typename Store<DT>::T *__restrict__ x, const typename Store<DT>::T *__restrict__ w,
    const float *__restrict__ bias, float alpha, typename Store<DT>::T *__restrict__ out,
    uint16_t *__restrict__ mask16, SmallcParams p) {
  using T = typename Store<DT>::T;
  constexpr int COUT = 16 * NF;
  constexpr bool BF = DT == DT_BF16;
  constexpr int KPER = BF ? 32 : 4;  // K per MFMA
  // cubic kernel of extent KE: every halo / tap index below divides by constants
  constexpr int HD = TD + KE - 1, HH = TH + KE - 1, HW = TW + KE - 1;
  constexpr int K = KE * KE * KE * CIN;
  constexpr int KS = (K + KPER - 1) / KPER;
  constexpr int JPER = BF ? 8 : 1;  // K-values per lane per MFMA
  constexpr int HALO = HD * HH * HW * CIN;
  __shared__ __attribute__((aligned(16))) T halo[HALO];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tiles_w = (p.ow + TW - 1) / TW, tiles_h = (p.oh + TH - 1) / TH;
  int t = blockIdx.x;
  const int tw = t % tiles_w; t /= tiles_w;
  const int th = t % tiles_h; t /= tiles_h;
  const int td = t;
  const int n = blockIdx.y;
  const int od0 = td * TD, oh0 = th * TH, ow0 = tw * TW;

  // ---- stage the zero-padded input halo: every load in flight before any store
  {
    constexpr int NL = (HALO + 255) / 256;
    T hv[NL];
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int e = tid + 256 * k;
      const int c = e % CIN;
      const int v = e / CIN;
      const int a = v / (HH * HW), b = (v / HW) % HH, cc = v % HW;
      const int id = od0 - p.pd + a, ih = oh0 - p.ph + b, iw = ow0 - p.pw + cc;
      T val = from_f32<DT>(0.f);
      if (e < HALO && (unsigned)id < (unsigned)p.d && (unsigned)ih < (unsigned)p.h && (unsigned)iw < (unsigned)p.w)
        val = x[((((long long)n * p.d + id) * p.h + ih) * p.w + iw) * CIN + c];
      hv[k] = val;
    }
#pragma unroll
    for (int k = 0; k < NL; ++k)
      if (tid + 256 * k < HALO) halo[tid + 256 * k] = hv[k];
  }

  // ---- per-lane constants: im2col tap offsets and the weight fragments ------
  const int r = lane & 15, q = lane >> 4;
  // A row r -> voxel (hh = (r&3)>>1, ww = r&1, w = 2 (r>>2) + ww) of a tile
  const int m_off = ((((r & 3) >> 1) * HW) + 2 * (r >> 2) + (r & 1)) * CIN;
  int toff[KS][JPER];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int j = 0; j < JPER; ++j) {
      const int kg = ks * KPER + (BF ? 8 * q + j : q);
      int off = 0;
      if (kg < K) {
        const int tap = kg / CIN, c = kg % CIN;
        const int a = tap / (KE * KE), b = (tap / KE) % KE, cc = tap % KE;
        off = ((a * HH + b) * HW + cc) * CIN + c;
      }
      toff[ks][j] = off;
    }
  using AFrag = typename std::conditional<BF, bf16x8_t, float>::type;
  AFrag bw[KS][NF];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      if constexpr (BF) {
        Vec16<DT_BF16> v;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int kg = ks * 32 + 8 * q + j;
          v.e[j] = kg < K ? w[(long long)kg * COUT + 16 * f + r] : (uint16_t)0;
        }
        bw[ks][f] = __builtin_bit_cast(bf16x8_t, v.u);
      } else {
        const int kg = ks * 4 + q;
        bw[ks][f] = kg < K ? (float)w[(long long)kg * COUT + 16 * f + r] : 0.f;
      }
    }
  float bz[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) bz[f] = FUSED ? bias[16 * f + r] : 0.f;
  __syncthreads();

  // ---- tile pairs: pooled voxels (pd, ph, pw .. pw+3) of this workgroup -----
  for (int pi = wave; pi < NPAIR; pi += 4) {
    const int bd = pi / ((TH / 2) * (TW / 8)), bh = (pi / (TW / 8)) % (TH / 2), bw8 = pi % (TW / 8);
    f32x4_t acc[2][NF];  // [dd][channel block]
#pragma unroll
    for (int dd = 0; dd < 2; ++dd) {
      const int base = (((2 * bd + dd) * HH + 2 * bh) * HW + 8 * bw8) * CIN + m_off;
#pragma unroll
      for (int f = 0; f < NF; ++f) acc[dd][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
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
            acc[dd][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bw[ks][f], acc[dd][f], 0, 0, 0);
          else
            acc[dd][f] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bw[ks][f], acc[dd][f], 0, 0, 0);
        }
      }
    }
    // this lane: channel 16f + r, rows 4q + j -> voxel (hh = j>>1, w = 8 bw8 + 2q + (j&1))
    const int vd0 = od0 + 2 * bd, vh0 = oh0 + 2 * bh, vw0 = ow0 + 8 * bw8;
    if constexpr (!FUSED) {
#pragma unroll
      for (int dd = 0; dd < 2; ++dd)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int vd = vd0 + dd, vh = vh0 + (j >> 1), vw = vw0 + 2 * q + (j & 1);
          if (vd >= p.od || vh >= p.oh || vw >= p.ow) continue;
          const long long vox = (((long long)n * p.od + vd) * p.oh + vh) * p.ow + vw;
#pragma unroll
          for (int f = 0; f < NF; ++f) out[vox * COUT + 16 * f + r] = from_f32<DT>(acc[dd][f][j]);
        }
    } else {
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        float s = 0.f;
        unsigned long long bal[2][4];
#pragma unroll
        for (int dd = 0; dd < 2; ++dd)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float u = acc[dd][f][j] + bz[f];
            bal[dd][j] = __ballot(u > 0.f);
            s += u > 0.f ? u : alpha * u;
          }
        // pooled voxel (pd, ph, pw + q): the whole window sits in this lane
        const int pd_ = vd0 >> 1, ph_ = vh0 >> 1, pw_ = (vw0 >> 1) + q;
        if (pd_ < p.pod && ph_ < p.poh && pw_ < p.pow_)
          out[((((long long)n * p.pod + pd_) * p.poh + ph_) * p.pow_ + pw_) * COUT + 16 * f + r] =
              from_f32<DT>(s * 0.125f);
        // slope mask: row (dd, hh) holds voxels w = vw0 .. vw0+7, 16 bits each;
        // lane 2 dd + hh (of the first four) writes those eight half-words
        if (lane < 4) {
          const int dd = lane >> 1, hh = lane & 1;
          const int vd = vd0 + dd, vh = vh0 + hh;
          if (vd < p.od && vh < p.oh) {
            const unsigned long long b0 = dd ? (hh ? bal[1][2] : bal[1][0]) : (hh ? bal[0][2] : bal[0][0]);
            const unsigned long long b1 = dd ? (hh ? bal[1][3] : bal[1][1]) : (hh ? bal[0][3] : bal[0][1]);
            uint16_t words[8];
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
              words[2 * qq] = (uint16_t)((b0 >> (16 * qq)) & 0xffffu);
              words[2 * qq + 1] = (uint16_t)((b1 >> (16 * qq)) & 0xffffu);
            }
            const long long vrow = (((long long)n * p.od + vd) * p.oh + vh) * p.ow;
            if (NF == 1 && vw0 + 8 <= p.ow && ((vrow + vw0) & 7) == 0) {
              uint4 pk;
              pk.x = words[0] | ((uint32_t)words[1] << 16);
              pk.y = words[2] | ((uint32_t)words[3] << 16);
              pk.z = words[4] | ((uint32_t)words[5] << 16);
              pk.w = words[6] | ((uint32_t)words[7] << 16);
              *reinterpret_cast<uint4 *>(mask16 + (vrow + vw0)) = pk;
            } else {
#pragma unroll
              for (int k = 0; k < 8; ++k)
                if (vw0 + k < p.ow) mask16[(vrow + vw0 + k) * NF + f] = words[k];
            }
          }
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
