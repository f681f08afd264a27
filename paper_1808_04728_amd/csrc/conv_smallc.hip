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
constexpr int KMAXE = 4;                                  // kernel extent limit per dimension

// Halo row staging: the staged w-window starts a whole 16-byte vector before
// the tile (covering the left padding) so that every row is a run of aligned
// 16-byte vectors, each entirely inside or entirely outside the input.
template <int DT, int CIN, int KE> struct HaloGeom {
  static constexpr int ES = DT == DT_BF16 ? 2 : 4;
  static constexpr int VV = 16 / (CIN * ES) > 0 ? 16 / (CIN * ES) : 1;  // voxels per 16-byte vector
  static constexpr int LEAD = (KE - 1 + VV - 1) / VV * VV;             // staged voxels left of the tile (>= pad)
  static constexpr int HD = TD + KE - 1, HH = TH + KE - 1;
  static constexpr int HWS = (LEAD + TW + KE - 1 + VV - 1) / VV * VV;  // staged row length (voxels)
  static constexpr int NVR = HWS / VV;                                 // 16-byte vectors per row
  static constexpr int ELEMS = HD * HH * HWS * CIN;
};

template <int DT, int CIN, int NF, int KE, bool FUSED>
__global__ __launch_bounds__(256) void conv_smallc_fwd_kernel(
    const typename Store<DT>::T *__restrict__ x, const typename Store<DT>::T *__restrict__ w,
    const float *__restrict__ bias, float alpha, typename Store<DT>::T *__restrict__ out,
    uint16_t *__restrict__ mask16, SmallcParams p) {
  using T = typename Store<DT>::T;
  using G = HaloGeom<DT, CIN, KE>;
  constexpr int COUT = 16 * NF;
  constexpr bool BF = DT == DT_BF16;
  constexpr int KPER = BF ? 32 : 4;  // K per MFMA
  constexpr int HH = G::HH, HWS = G::HWS;
  constexpr int K = KE * KE * KE * CIN;
  constexpr int KS = (K + KPER - 1) / KPER;
  constexpr int JPER = BF ? 8 : 1;  // K-values per lane per MFMA
  // Bias through the MFMA: with two spare K slots, slot K carries bf16(b) and
  // slot K + 1 the bf16 rounding of the remainder (b to ~16 significant bits),
  // both against A = 1.0, read from ONES_PLANES extra halo planes of ones that
  // sit HD planes after every voxel of the tile.
  constexpr bool BIAS_MFMA = FUSED && BF && (KS * 32 - K >= 2);
  constexpr int ONES = BIAS_MFMA ? TD * HH * HWS * CIN : 0;
  constexpr int ONES_OFF = G::HD * HH * HWS * CIN;  // element offset voxel -> its 1.0 slot
  __shared__ __attribute__((aligned(16))) T halo[G::ELEMS + ONES];
  // fused, 16 channels: raw slope ballots of one row of eight tile pairs per wave
  __shared__ __attribute__((aligned(16))) uint64_t bstage[4][(FUSED && NF == 1) ? 64 : 1];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tiles_w = (p.ow + TW - 1) / TW, tiles_h = (p.oh + TH - 1) / TH;
  int t = blockIdx.x;
  const int tw = t % tiles_w; t /= tiles_w;
  const int th = t % tiles_h; t /= tiles_h;
  const int td = t;
  const int n = blockIdx.y;
  const int od0 = td * TD, oh0 = th * TH, ow0 = tw * TW;
  // staged slot c of a halo row holds input column iw = ow0 - LEAD + c

  // ---- stage the zero-padded input halo: every load in flight before any store
  if (p.w % G::VV == 0) {
    constexpr int NV = G::HD * HH * G::NVR;
    constexpr int NL = (NV + 255) / 256;
    uint4 hv[NL];
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int e = tid + 256 * k;
      const int v = e % G::NVR, rb = e / G::NVR;
      const int a = rb / HH, b = rb % HH;
      const int id = od0 - p.pd + a, ih = oh0 - p.ph + b;
      const int iw0 = ow0 - G::LEAD + v * G::VV;  // a whole vector, inside or outside [0, w)
      uint4 val = make_uint4(0, 0, 0, 0);
      if (e < NV && (unsigned)id < (unsigned)p.d && (unsigned)ih < (unsigned)p.h && iw0 >= 0 && iw0 < p.w)
        val = *reinterpret_cast<const uint4 *>(x + ((((long long)n * p.d + id) * p.h + ih) * p.w + iw0) * CIN);
      hv[k] = val;
    }
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int e = tid + 256 * k;
      if (e < NV) *reinterpret_cast<uint4 *>(&halo[e * G::VV * CIN]) = hv[k];
    }
  } else {
    constexpr int NL = (G::ELEMS + 255) / 256;
    T hv[NL];
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int e = tid + 256 * k;
      const int c = e % CIN, v = e / CIN;
      const int cc = v % HWS, rb = v / HWS;
      const int a = rb / HH, b = rb % HH;
      const int id = od0 - p.pd + a, ih = oh0 - p.ph + b, iw = ow0 - G::LEAD + cc;
      T val = from_f32<DT>(0.f);
      if (e < G::ELEMS && (unsigned)id < (unsigned)p.d && (unsigned)ih < (unsigned)p.h && (unsigned)iw < (unsigned)p.w)
        val = x[((((long long)n * p.d + id) * p.h + ih) * p.w + iw) * CIN + c];
      hv[k] = val;
    }
#pragma unroll
    for (int k = 0; k < NL; ++k)
      if (tid + 256 * k < G::ELEMS) halo[tid + 256 * k] = hv[k];
  }

  if constexpr (BIAS_MFMA) {
    static_assert(G::ELEMS % 8 == 0 && ONES % 8 == 0, "16-byte fill");
    const uint4 one8 = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);
    for (int e = tid; e < ONES / 8; e += 256) *reinterpret_cast<uint4 *>(&halo[G::ELEMS + 8 * e]) = one8;
  }

  // ---- per-lane constants: im2col tap offsets and the weight fragments ------
  const int r = lane & 15, q = lane >> 4;
  // A row r -> voxel (hh = (r&3)>>1, w = 2 (r>>2) + (r&1)) of a tile
  const int m_off = ((((r & 3) >> 1) * HWS) + 2 * (r >> 2) + (r & 1)) * CIN;
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
        off = ((a * HH + b) * HWS + cc) * CIN + c;
      } else if (BIAS_MFMA && kg < K + 2) {
        off = ONES_OFF;
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
          uint16_t e = kg < K ? w[(long long)kg * COUT + 16 * f + r] : (uint16_t)0;
          if (BIAS_MFMA && kg >= K && kg < K + 2) {
            const float b = bias[16 * f + r];
            const uint16_t hi = f2bf(b);
            e = kg == K ? hi : f2bf(b - bf2f(hi));
          }
          v.e[j] = e;
        }
        bw[ks][f] = __builtin_bit_cast(bf16x8_t, v.u);
      } else {
        const int kg = ks * 4 + q;
        bw[ks][f] = kg < K ? (float)w[(long long)kg * COUT + 16 * f + r] : 0.f;
      }
    }
  float bz[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) bz[f] = FUSED && !BIAS_MFMA ? bias[16 * f + r] : 0.f;
  __syncthreads();

  // ---- rows (bd, bh) of eight tile pairs; pair bw8 = pooled voxels
  // (pd, ph, 4 bw8 .. 4 bw8 + 3) of the workgroup.  The lane's gather
  // addresses are formed once per row; every tile of the row reads the halo
  // at a compile-time byte offset from them.
  const unsigned char *hb = reinterpret_cast<const unsigned char *>(halo);
  for (int ri = wave; ri < (TD / 2) * (TH / 2); ri += 4) {
    const int bd = ri / (TH / 2), bh = ri % (TH / 2);
    const int row_base = ((2 * bd * HH + 2 * bh) * HWS + G::LEAD - p.pw) * CIN + m_off;
    int addr[KS][JPER];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int j = 0; j < JPER; ++j) addr[ks][j] = (row_base + toff[ks][j]) * (int)sizeof(T);
    const int vd0 = od0 + 2 * bd, vh0 = oh0 + 2 * bh;
#pragma unroll
    for (int bw8 = 0; bw8 < TW / 8; ++bw8) {
      f32x4_t acc[2][NF];  // [dd][channel block]
#pragma unroll
      for (int dd = 0; dd < 2; ++dd)
#pragma unroll
        for (int f = 0; f < NF; ++f) acc[dd][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int dd = 0; dd < 2; ++dd) {
        const int imm = ((dd * HH * HWS) + 8 * bw8) * CIN * (int)sizeof(T);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          AFrag a;
          if constexpr (BF) {
            // element by element (16-bit reads, packed in pairs by the compiler:
            // with SRAM ECC on, as on this part, a 16-bit read into half a
            // register does not keep the other half, so halves cannot be
            // loaded in place)
            typedef short v8i16_t __attribute__((ext_vector_type(8)));
            v8i16_t v;
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = *reinterpret_cast<const short *>(hb + addr[ks][j] + imm);
            a = __builtin_bit_cast(bf16x8_t, v);
          } else {
            a = *reinterpret_cast<const float *>(hb + addr[ks][0] + imm);
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
      const int vw0 = ow0 + 8 * bw8;
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
        const int pd_ = vd0 >> 1, ph_ = vh0 >> 1, pw_ = (vw0 >> 1) + q;
        const bool pin = pd_ < p.pod && ph_ < p.poh && pw_ < p.pow_;
        // pooled row of this lane's first pair; pair bw8 sits 4 bw8 pooled voxels on
        // (a compile-time offset from one row pointer)
        T *const prow = out + ((((long long)n * p.pod + pd_) * p.poh + ph_) * p.pow_ + (ow0 >> 1) + q) * COUT +
                        (long long)(4 * bw8 * COUT);
#pragma unroll
        for (int f = 0; f < NF; ++f) {
          float s = 0.f;
          uint64_t bal[2][4];
#pragma unroll
          for (int dd = 0; dd < 2; ++dd)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const float u = BIAS_MFMA ? acc[dd][f][j] : acc[dd][f][j] + bz[f];
              const bool pos = u > 0.f;
              bal[dd][j] = __ballot(pos);
              s = fmaf(pos ? 1.f : alpha, u, s);
            }
          // pooled voxel (pd, ph, pw + q): the whole window sits in this lane
          if (pin) prow[16 * f + r] = from_f32<DT>(s * 0.125f);
          if constexpr (NF == 1) {
            // the eight ballots of the pair go to LDS as they are (one lane writes);
            // the row's mask words are interleaved from them after the last pair
            // (moves the compiler places: it tracks the wait states between a
            // compare writing an SGPR pair and a vector instruction reading it)
            uint64_t bv[2][4];
#pragma unroll
            for (int dd = 0; dd < 2; ++dd)
#pragma unroll
              for (int j = 0; j < 4; ++j) bv[dd][j] = bal[dd][j];
            if (lane == 0) {
#pragma unroll
              for (int dd = 0; dd < 2; ++dd)
#pragma unroll
                for (int j = 0; j < 4; ++j) bstage[wave][bw8 * 8 + dd * 4 + j] = bv[dd][j];
            }
          } else {
            // general channel count: lanes 0..3 write mask row (dd, hh) as half-words
            if (lane < 4) {
              const int dd = lane >> 1, hh = lane & 1;
              const int vd = vd0 + dd, vh = vh0 + hh;
              if (vd < p.od && vh < p.oh) {
                const uint64_t b0 = dd ? (hh ? bal[1][2] : bal[1][0]) : (hh ? bal[0][2] : bal[0][0]);
                const uint64_t b1 = dd ? (hh ? bal[1][3] : bal[1][1]) : (hh ? bal[0][3] : bal[0][1]);
                const long long vrow = (((long long)n * p.od + vd) * p.oh + vh) * p.ow;
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                  const uint64_t bb = (k & 1) ? b1 : b0;
                  if (vw0 + k < p.ow) mask16[(vrow + vw0 + k) * NF + f] = (uint16_t)((bb >> (16 * (k >> 1))) & 0xffffu);
                }
              }
            }
          }
        }
      }
    }
    if constexpr (FUSED && NF == 1) {
      // lanes 0..31: the 16 bytes of mask row k = (dd, hh) = (lane & 3) for
      // voxels w = 8 b8 .. 8 b8 + 7, b8 = lane >> 2.  Ballot bit 16 q + c is
      // channel c of voxel w = 2q + parity, parity = which of the two ballots:
      // the row is the ballots' 16-bit words interleaved, even voxel first.
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      if (lane < 32) {
        const int k = lane & 3, b8 = lane >> 2;
        const uint64_t be = bstage[wave][b8 * 8 + (k >> 1) * 4 + 2 * (k & 1)];
        const uint64_t bo = bstage[wave][b8 * 8 + (k >> 1) * 4 + 2 * (k & 1) + 1];
        const uint32_t el = (uint32_t)be, eh = (uint32_t)(be >> 32), ol = (uint32_t)bo, oh = (uint32_t)(bo >> 32);
        uint4 mw;
        mw.x = __builtin_amdgcn_perm(ol, el, 0x05040100u);  // w0 | w1 << 16
        mw.y = __builtin_amdgcn_perm(ol, el, 0x07060302u);  // w2 | w3 << 16
        mw.z = __builtin_amdgcn_perm(oh, eh, 0x05040100u);
        mw.w = __builtin_amdgcn_perm(oh, eh, 0x07060302u);
        const int vd = vd0 + (k >> 1), vh = vh0 + (k & 1), vw = ow0 + 8 * b8;
        if (vd < p.od && vh < p.oh) {
          const long long vrow = (((long long)n * p.od + vd) * p.oh + vh) * p.ow;
          if (vw + 8 <= p.ow && ((vrow + vw) & 7) == 0) {
            *reinterpret_cast<uint4 *>(mask16 + (vrow + vw)) = mw;
          } else {
            const uint32_t words[4] = {mw.x, mw.y, mw.z, mw.w};
#pragma unroll
            for (int k2 = 0; k2 < 8; ++k2)
              if (vw + k2 < p.ow) mask16[vrow + vw + k2] = (uint16_t)((words[k2 >> 1] >> (16 * (k2 & 1))) & 0xffffu);
          }
        }
      }
      // the next row's ballots overwrite the stage only after every lane has read it
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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
