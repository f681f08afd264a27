// conv_c16_bwd.hip -- backward data of the 16 -> 32 channel stride-1 layer (gfx950, bf16).
//
// Backward data (Section III-C: propagate the output difference signal to
// the input) of a stride-1 layer is itself a stride-1 convolution of dz with
// the kernel flipped in every dimension and transposed in channels:
//     dx[i, ci] = sum_{t', co} dz[i - p' + t', co] * W[k-1-t', ci, co],
//     p' = k - 1 - pad_before.
// Per tap the reduction runs over the 32 output channels, which is exactly
// the K = 32 of v_mfma_f32_16x16x32_bf16:
//   A (16 x 32)  = 16 consecutive voxels along w x the 32 channels of dz,
//   B (32 x 16)  = W[tap][ci][co] read as [co][ci] -- 16 contiguous bytes per
//                  lane straight from the DHWIO tensor (no repacking),
//   D (16 x 16)  = 16 voxels x all 16 input channels.
// Persistent workgroups (two per CU) loop over 4x4x16-voxel tiles of dx; the zero-padded
// dz halo of the tile sits in LDS as [d][h][co/8][w][8 co] (a 256-byte
// contiguous run per quarter wave), each wave owns one d-row (4 h x 32 w) and
// reuses every A fragment for all k output rows it reaches.  The next tap's
// weight fragments are loaded into registers while the current ones are
// consumed; halo loads of one workgroup overlap the MFMAs of the other.
//
// Fused variant: dz is never stored.  It is rebuilt while staging the halo
// from the gradient of the pooled output and the forward slope mask,
//     dz[v, c] = dp[pool(v), c] / 8 * (mask(v, c) ? 1 : alpha),
// rounded to bf16 exactly as the unfused path stores it.

#include "cf_common.h"
#include "cf_kernels.h"

namespace cf {
namespace {

constexpr int TD = 4, TH = 4, TW = 16;  // 60 KB halo: two workgroups per CU
constexpr int WB = TW / 16;

template <int KE>
struct C16B {
  static constexpr int HD = TD + KE - 1, HH = TH + KE - 1, HW = TW + KE - 1;
  static constexpr int HALO_VEC = HD * HH * 4 * HW;  // 16-byte units: 8 of the 32 dz channels
  static constexpr int LDS_BYTES = HALO_VEC * 16;
  static constexpr int NPRE = (HALO_VEC + 255) / 256;
};

template <int KE, bool FUSED>
__global__ __launch_bounds__(256, 2) void c16_dgrad_kernel(const uint16_t *__restrict__ g,
                                                           const uint32_t *__restrict__ mask,
                                                           const uint16_t *__restrict__ w, float alpha,
                                                           uint16_t *__restrict__ dx, C16Params p) {
  using G = C16B<KE>;
  extern __shared__ __attribute__((aligned(16))) uint4 halo[];  // [HD][HH][4][HW]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, q = lane >> 4;
  const int pdp = KE - 1 - p.pd, php = KE - 1 - p.ph, pwp = KE - 1 - p.pw;  // flipped-kernel pads

  // here (d, h, w) is the dx extent and (od, oh, ow) the dz extent
  const int tiles_w = (p.w + TW - 1) / TW, tiles_h = (p.h + TH - 1) / TH, tiles_d = (p.d + TD - 1) / TD;
  const int tiles = p.n * tiles_d * tiles_h * tiles_w;
  const int nblk = gridDim.x;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, per_xcd_blocks = (nblk + 7) >> 3;
  const int per = (tiles + 7) >> 3;
  auto tile_of = [&](int i) { return xcd * per + i; };

  uint4 pre[G::NPRE];
  auto fetch = [&](int t) {
    int r = t;
    const int tw = r % tiles_w; r /= tiles_w;
    const int th = r % tiles_h; r /= tiles_h;
    const int td = r % tiles_d;
    const int n = r / tiles_d;
    const int i0d = td * TD - pdp, i0h = th * TH - php, i0w = tw * TW - pwp;
#pragma unroll
    for (int k = 0; k < G::NPRE; ++k) {
      const int e = tid + 256 * k;
      const int cq = e & 3;
      int v = e >> 2;
      const int hw = v % G::HW; v /= G::HW;
      const int hh = v % G::HH;
      const int hd = v / G::HH;
      const int sd = i0d + hd, sh = i0h + hh, sw = i0w + hw;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (e < G::HALO_VEC && (unsigned)sd < (unsigned)p.od && (unsigned)sh < (unsigned)p.oh &&
          (unsigned)sw < (unsigned)p.ow) {
        const long long vox = (((long long)n * p.od + sd) * p.oh + sh) * p.ow + sw;
        if constexpr (!FUSED) {
          val = *reinterpret_cast<const uint4 *>(g + vox * 32 + 8 * cq);
        } else {
          const int pd_ = sd >> 1, ph_ = sh >> 1, pw_ = sw >> 1;
          if (pd_ < p.pod && ph_ < p.poh && pw_ < p.pow_) {
            Vec16<DT_BF16> gv;
            gv.u = *reinterpret_cast<const uint4 *>(
                g + ((((long long)n * p.pod + pd_) * p.poh + ph_) * p.pow_ + pw_) * 32 + 8 * cq);
            const uint32_t bits = mask[vox] >> (8 * cq);
#pragma unroll
            for (int j = 0; j < 8; ++j)
              gv.e[j] = f2bf(bf2f(gv.e[j]) * 0.125f * (((bits >> j) & 1u) ? 1.f : alpha));
            val = gv.u;
          }
        }
      }
      pre[k] = val;
    }
  };

  for (int i = slot;; i += per_xcd_blocks) {
    const int t = tile_of(i);
    if (i >= per || t >= tiles) break;
    int r = t;
    const int tw = r % tiles_w; r /= tiles_w;
    const int th = r % tiles_h; r /= tiles_h;
    const int td = r % tiles_d;
    const int n = r / tiles_d;
    const int x0d = td * TD, x0h = th * TH, x0w = tw * TW;

    __syncthreads();
    fetch(t);  // all loads in flight at once; the other workgroup on the CU computes meanwhile
#pragma unroll
    for (int k = 0; k < G::NPRE; ++k) {
      const int e = tid + 256 * k;
      if (e >= G::HALO_VEC) continue;
      const int cq = e & 3;
      int v = e >> 2;
      const int hw = v % G::HW; v /= G::HW;
      const int hh = v % G::HH;
      const int hd = v / G::HH;
      halo[((hd * G::HH + hh) * 4 + cq) * G::HW + hw] = pre[k];
    }
    __syncthreads();

    f32x4_t acc[TH][WB];
#pragma unroll
    for (int a = 0; a < TH; ++a)
#pragma unroll
      for (int b = 0; b < WB; ++b) acc[a][b] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // weight fragment of flipped tap (kd', kh', kw'): W[k-1-kd'][k-1-kh'][k-1-kw'][ci = r16][8q .. 8q+7]
    auto wfrag = [&](int kd, int kh, int kw) {
      const int tap = ((KE - 1 - kd) * KE + (KE - 1 - kh)) * KE + (KE - 1 - kw);
      return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4 *>(w + ((long long)tap * 16 + r16) * 32 + 8 * q));
    };
    bf16x8_t bcur[KE], bnext[KE];
#pragma unroll
    for (int kh = 0; kh < KE; ++kh) bcur[kh] = wfrag(0, kh, 0);

    for (int kd = 0; kd < KE; ++kd) {
#pragma unroll 1
      for (int kw = 0; kw < KE; ++kw) {
        // prefetch the next (kd, kw) weight fragments (loop-carried, one step ahead)
        const int nkw = kw + 1 < KE ? kw + 1 : 0, nkd = kw + 1 < KE ? kd : kd + 1;
        if (nkd < KE) {
#pragma unroll
          for (int kh = 0; kh < KE; ++kh) bnext[kh] = wfrag(nkd, kh, nkw);
        }
        // all fragment reads of this (kd, kw) step are issued before its MFMAs
        bf16x8_t afr[TH + KE - 1][WB];
#pragma unroll
        for (int hi = 0; hi < TH + KE - 1; ++hi)
#pragma unroll
          for (int wb = 0; wb < WB; ++wb)
            afr[hi][wb] = __builtin_bit_cast(
                bf16x8_t, halo[(((wave + kd) * G::HH + hi) * 4 + q) * G::HW + wb * 16 + kw + r16]);
#pragma unroll
        for (int hi = 0; hi < TH + KE - 1; ++hi) {
#pragma unroll
          for (int wb = 0; wb < WB; ++wb) {
#pragma unroll
            for (int kh = 0; kh < KE; ++kh) {
              const int hrow = hi - kh;
              if (hrow >= 0 && hrow < TH)
                acc[hrow][wb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afr[hi][wb], bcur[kh], acc[hrow][wb], 0, 0, 0);
            }
          }
        }
#pragma unroll
        for (int kh = 0; kh < KE; ++kh) bcur[kh] = bnext[kh];
      }
    }

    // D: lane -> input channel r16, rows 4q + j -> voxel w within the 16-block
    const int vd = x0d + wave;
    if (vd < p.d) {
#pragma unroll
      for (int hh = 0; hh < TH; ++hh) {
        const int vh = x0h + hh;
        if (vh >= p.h) continue;
        const long long rowv = (((long long)n * p.d + vd) * p.h + vh) * p.w;
#pragma unroll
        for (int wb = 0; wb < WB; ++wb)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int vw = x0w + wb * 16 + 4 * q + j;
            if (vw < p.w) dx[(rowv + vw) * 16 + r16] = f2bf(acc[hh][wb][j]);
          }
      }
    }
  }
}

template <int KE, bool FUSED>
hipError_t launch_dgrad(const C16Params &p, const void *g, const uint32_t *mask, const void *w, float alpha,
                        void *dx, hipStream_t st) {
  using G = C16B<KE>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void *)c16_dgrad_kernel<KE, FUSED>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, G::LDS_BYTES);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess) hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  const long long tiles = (long long)p.n * ((p.d + TD - 1) / TD) * ((p.h + TH - 1) / TH) * ((p.w + TW - 1) / TW);
  int blocks = (int)std::min<long long>(tiles, 2LL * cus);
  blocks = std::max(8, (blocks + 7) / 8 * 8);
  hipLaunchKernelGGL((c16_dgrad_kernel<KE, FUSED>), dim3(blocks), dim3(256), G::LDS_BYTES, st, (const uint16_t *)g,
                     mask, (const uint16_t *)w, alpha, (uint16_t *)dx, p);
  return hipGetLastError();
}

}  // namespace

bool c16_bwd_supported(const ConvShape &s) { return c16_fwd_supported(s); }

hipError_t launch_conv_bwd_data_c16(const ConvShape &s, const void *g, const uint32_t *mask, const void *w,
                                    float alpha, void *dx, bool fused, hipStream_t st) {
  C16Params p{};
  p.n = s.n; p.d = s.d; p.h = s.h; p.w = s.w;
  p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.od = s.od; p.oh = s.oh; p.ow = s.ow;
  p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
#define CF_C16B_CASE(KEV)                                                                   \
  if (s.kd == KEV)                                                                          \
    return fused ? launch_dgrad<KEV, true>(p, g, mask, w, alpha, dx, st)                    \
                 : launch_dgrad<KEV, false>(p, g, mask, w, alpha, dx, st);
  CF_C16B_CASE(2) CF_C16B_CASE(3) CF_C16B_CASE(4)
#undef CF_C16B_CASE
  return hipErrorInvalidValue;
}

}  // namespace cf
