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
// A persistent workgroup of eight waves (two per SIMD) loops over 8x4x16-voxel
// tiles of dx; wave w owns d-plane w of the tile and reuses every A fragment
// for all k output rows it reaches.  The zero-padded dz halo of the tile sits
// in LDS as [d][h][co/8][w][8 co] (a 256-byte run per quarter wave).  The
// halo is staged by buffer -> LDS DMA; padding voxels get a byte offset past
// the buffer, which the hardware range check turns into zeros.  Weight
// fragments stream from global memory two (kd, kw) steps ahead, A fragments
// from LDS one step ahead.
//
// Fused variant: dz is never stored.  The tile's box of the pooled-output
// gradient and the slope-mask words of its halo voxels arrive by DMA in their
// own LDS areas, and the halo is built from them once per tile,
//     dz[v, c] = dp[pool(v), c] / 8 * (mask(v, c) ? 1 : alpha),
// rounded to bf16 exactly as the unfused path stores it.  A voxel outside dz,
// or off the pooling grid, maps to a pooled voxel outside dp, whose DMA slot
// is zero -- so no bounds test is needed there.  The next tile's DMA is issued
// as soon as the halo is built and overlaps the whole MFMA loop.

#include "cf_common.h"
#include "cf_kernels.h"

#include <algorithm>

namespace cf {
namespace {

constexpr int TD = 8, TH = 4, TW = 16;  // dx tile (voxels)
constexpr int NWAVE = 8;                // wave w owns d-plane w of the tile

template <int KE, bool FUSED>
struct C16B {
  static constexpr int HD = TD + KE - 1, HH = TH + KE - 1, HW = TW + KE - 1;
  static constexpr int HALO_VEC = HD * HH * 4 * HW;          // 16-byte slots: 8 of the 32 dz channels
  static constexpr int HALO_PAD = (HALO_VEC + 63) / 64 * 64;
  // fused staging: the pooled-gradient box covering the halo (either parity) and the mask words
  static constexpr int PD = HD / 2 + 1, PH = HH / 2 + 1, PW = HW / 2 + 1;
  static constexpr int DP_VEC = FUSED ? PD * PH * PW * 4 : 0;
  static constexpr int DP_PAD = (DP_VEC + 63) / 64 * 64;
  static constexpr int MK = FUSED ? HD * HH * HW : 0;          // 4-byte words
  static constexpr int MK_PAD = (MK + 63) / 64 * 64;
  static constexpr int LDS_BYTES = HALO_PAD * 16 + DP_PAD * 16 + MK_PAD * 4;
};

typedef __attribute__((address_space(3))) void lds_void_t;

template <int KE, bool FUSED>
__global__ __launch_bounds__(512, 1) void c16_dgrad_kernel(const uint16_t *__restrict__ g,
                                                           const uint32_t *__restrict__ mask,
                                                           const uint16_t *__restrict__ w, float alpha,
                                                           uint16_t *__restrict__ dx, C16Params p) {
  using G = C16B<KE, FUSED>;
  extern __shared__ __attribute__((aligned(16))) uint4 smem[];
  uint4 *halo = smem;                                             // [HD][HH][4][HW]
  uint4 *dpb = smem + G::HALO_PAD;                                // fused: [PD][PH][PW][4]
  uint32_t *mkw = reinterpret_cast<uint32_t *>(dpb + G::DP_PAD);  // fused: [HD][HH][HW]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, q = lane >> 4;
  const int pdp = KE - 1 - p.pd, php = KE - 1 - p.ph, pwp = KE - 1 - p.pw;  // flipped-kernel pads

  // here (d, h, w) is the dx extent and (od, oh, ow) the dz extent
  const int tiles_w = (p.w + TW - 1) / TW, tiles_h = (p.h + TH - 1) / TH, tiles_d = (p.d + TD - 1) / TD;
  const int tiles = p.n * tiles_d * tiles_h * tiles_w;
  const int nblk = gridDim.x;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, per_xcd_blocks = (nblk + 7) >> 3;
  const int per = (tiles + 7) >> 3;
  auto tile_of = [&](int i) { return xcd * per + i; };
  struct Org {
    int n, x0d, x0h, x0w;
  };
  auto origin = [&](int t) {
    Org o;
    int r = t;
    const int tw = r % tiles_w; r /= tiles_w;
    const int th = r % tiles_h; r /= tiles_h;
    const int td = r % tiles_d;
    o.n = r / tiles_d;
    o.x0d = td * TD; o.x0h = th * TH; o.x0w = tw * TW;
    return o;
  };

  // ---- DMA staging ---------------------------------------------------------
  const __amdgpu_buffer_rsrc_t grsrc = __builtin_amdgcn_make_buffer_rsrc((void *)g, (short)0, p.g_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t mrsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)mask, (short)0, FUSED ? p.m_bytes : 0, 0x00020000);
  auto issue = [&](int t) {
    const Org o = origin(t);
    const int s0d = o.x0d - pdp, s0h = o.x0h - php, s0w = o.x0w - pwp;  // halo origin in dz
    if constexpr (!FUSED) {
      // dz halo, slot s = ((hd * HH + hh) * 4 + cq) * HW + hw
      for (int c = wave; c < G::HALO_PAD / 64; c += NWAVE) {
        const int s = 64 * c + lane;
        const int hw = s % G::HW, t1 = s / G::HW;
        const int cq = t1 & 3, t2 = t1 >> 2;
        const int hh = t2 % G::HH, hd = t2 / G::HH;
        const int sd = s0d + hd, sh = s0h + hh, sw = s0w + hw;
        uint32_t off = 0x80000000u;
        if (s < G::HALO_VEC && (unsigned)sd < (unsigned)p.od && (unsigned)sh < (unsigned)p.oh &&
            (unsigned)sw < (unsigned)p.ow)
          off = (uint32_t)(((((o.n * p.od + sd) * p.oh + sh) * p.ow + sw) * 32 + 8 * cq) * 2);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(grsrc, (lds_void_t *)(halo + 64 * c), 16, off, 0, 0, 0);
      }
    } else {
      // pooled-gradient box [PD][PH][4][PW] (channel group before w: the halo
      // build then reads consecutive 16-byte slots) from pooled origin floor(s0 / 2)
      const int p0d = s0d >> 1, p0h = s0h >> 1, p0w = s0w >> 1;
      for (int c = wave; c < G::DP_PAD / 64; c += NWAVE) {
        const int s = 64 * c + lane;
        const int pw_ = s % G::PW, t1 = s / G::PW;
        const int cq = t1 & 3, t2 = t1 >> 2;
        const int ph_ = t2 % G::PH, pd_ = t2 / G::PH;
        const int gd = p0d + pd_, gh = p0h + ph_, gw = p0w + pw_;
        uint32_t off = 0x80000000u;
        if (s < G::DP_VEC && (unsigned)gd < (unsigned)p.pod && (unsigned)gh < (unsigned)p.poh &&
            (unsigned)gw < (unsigned)p.pow_)
          off = (uint32_t)(((((o.n * p.pod + gd) * p.poh + gh) * p.pow_ + gw) * 32 + 8 * cq) * 2);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(grsrc, (lds_void_t *)(dpb + 64 * c), 16, off, 0, 0, 0);
      }
      // slope-mask words of the halo voxels [HD][HH][HW]
      for (int c = wave; c < G::MK_PAD / 64; c += NWAVE) {
        const int s = 64 * c + lane;
        const int hw = s % G::HW, t1 = s / G::HW;
        const int hh = t1 % G::HH, hd = t1 / G::HH;
        const int sd = s0d + hd, sh = s0h + hh, sw = s0w + hw;
        uint32_t off = 0x80000000u;
        if (s < G::MK && (unsigned)sd < (unsigned)p.od && (unsigned)sh < (unsigned)p.oh && (unsigned)sw < (unsigned)p.ow)
          off = (uint32_t)((((o.n * p.od + sd) * p.oh + sh) * p.ow + sw) * 4);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(mrsrc, (lds_void_t *)(mkw + 64 * c), 4, off, 0, 0, 0);
      }
    }
  };

  // weight fragment of flipped tap (kd', kh', kw'): W[k-1-kd'][k-1-kh'][k-1-kw'][ci = r16][8q .. 8q+7],
  // a buffer load at the lane's byte offset plus a constant tap offset
  const __amdgpu_buffer_rsrc_t wrsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)w, (short)0, KE * KE * KE * 16 * 32 * 2, 0x00020000);
  const int wlane = (r16 * 32 + 8 * q) * 2;
  auto wfrag = [&](int kd, int kh, int kw) {
    const int tap = ((KE - 1 - kd) * KE + (KE - 1 - kh)) * KE + (KE - 1 - kw);
    typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(wrsrc, wlane, tap * 16 * 32 * 2, 0);
    return __builtin_bit_cast(bf16x8_t, v);
  };

  if (slot < per && tile_of(slot) < tiles) issue(tile_of(slot));

  for (int i = slot;; i += per_xcd_blocks) {
    const int t = tile_of(i);
    if (i >= per || t >= tiles) break;
    const Org o = origin(t);
    const int inext = i + per_xcd_blocks;
    const bool has_next = inext < per && tile_of(inext) < tiles;

    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this wave's DMA has landed
    __syncthreads();                     // ... and every other wave's
    if constexpr (FUSED) {
      // build the dz halo from the staged pooled gradient and mask words, one
      // pooling window (2x2x2 voxels x 8 channels) per item: the pooled vector
      // is converted once, every voxel of the window selects per channel
      const int s0d = o.x0d - pdp, s0h = o.x0h - php, s0w = o.x0w - pwp;
      const int p0d = s0d >> 1, p0h = s0h >> 1, p0w = s0w >> 1;
      const float a8 = 0.125f * alpha;
      for (int it = tid; it < G::DP_VEC; it += 64 * NWAVE) {
        const int pwl = it % G::PW, t1 = it / G::PW;
        const int cq = t1 & 3, t2 = t1 >> 2;
        const int phl = t2 % G::PH, pdl = t2 / G::PH;
        Vec16<DT_BF16> gv;
        gv.u = dpb[it];
        float g1[8], ga[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float gf = bf2f(gv.e[j]);
          g1[j] = gf * 0.125f;
          ga[j] = gf * a8;
        }
        // window voxels in halo coordinates
        const int hd0 = 2 * (p0d + pdl) - s0d, hh0 = 2 * (p0h + phl) - s0h, hw0 = 2 * (p0w + pwl) - s0w;
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const int hd = hd0 + (v >> 2), hh = hh0 + ((v >> 1) & 1), hw = hw0 + (v & 1);
          if ((unsigned)hd >= (unsigned)G::HD || (unsigned)hh >= (unsigned)G::HH || (unsigned)hw >= (unsigned)G::HW)
            continue;
          const uint32_t bits = mkw[(hd * G::HH + hh) * G::HW + hw] >> (8 * cq);
          Vec16<DT_BF16> dv;
#pragma unroll
          for (int j = 0; j < 8; ++j) dv.e[j] = f2bf(((bits >> j) & 1u) ? g1[j] : ga[j]);
          halo[((hd * G::HH + hh) * 4 + cq) * G::HW + hw] = dv.u;
        }
      }
      __syncthreads();
      if (has_next) issue(tile_of(inext));  // the staging areas are free: overlap the MFMA loop
    }

    // ---- MFMA: wave = d-plane; (kd, kw) steps, A one step and B two steps ahead
    f32x4_t acc[TH];
#pragma unroll
    for (int a = 0; a < TH; ++a) acc[a] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    constexpr int NSTEP = KE * KE;
    bf16x8_t bfr[3][KE];
    bf16x8_t afr[2][TH + KE - 1];
    auto load_b = [&](int st, bf16x8_t(&b)[KE]) {
#pragma unroll
      for (int kh = 0; kh < KE; ++kh) b[kh] = wfrag(st / KE, kh, st % KE);
    };
    // the wave's plane + the lane's (co group, voxel) part; every step adds a constant
    const uint4 *abase = halo + (wave * G::HH * 4 + q) * G::HW + r16;
    auto load_a = [&](int st, bf16x8_t(&a)[TH + KE - 1]) {
      const int kd = st / KE, kw = st % KE;
#pragma unroll
      for (int hi = 0; hi < TH + KE - 1; ++hi)
        a[hi] = __builtin_bit_cast(bf16x8_t, abase[(kd * G::HH + hi) * 4 * G::HW + kw]);
    };
    load_b(0, bfr[0]);
    if (NSTEP > 1) load_b(1, bfr[1]);
    load_a(0, afr[0]);
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) {
      if (st + 2 < NSTEP) load_b(st + 2, bfr[(st + 2) % 3]);
      if (st + 1 < NSTEP) load_a(st + 1, afr[(st + 1) & 1]);
#pragma unroll
      for (int hi = 0; hi < TH + KE - 1; ++hi)
#pragma unroll
        for (int kh = 0; kh < KE; ++kh) {
          const int hrow = hi - kh;
          if (hrow >= 0 && hrow < TH)
            acc[hrow] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afr[st & 1][hi], bfr[st % 3][kh], acc[hrow], 0, 0, 0);
        }
    }

    if constexpr (!FUSED) {
      __syncthreads();  // every wave is done with the halo
      if (has_next) issue(tile_of(inext));
    }

    // D: lane -> input channel r16, rows 4q + j -> voxel w within the 16-block
    const int vd = o.x0d + wave;
    if (vd < p.d) {
#pragma unroll
      for (int hh = 0; hh < TH; ++hh) {
        const int vh = o.x0h + hh;
        if (vh >= p.h) continue;
        const long long rowv = (((long long)o.n * p.d + vd) * p.h + vh) * p.w;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int vw = o.x0w + 4 * q + j;
          if (vw < p.w) dx[(rowv + vw) * 16 + r16] = f2bf(acc[hh][j]);
        }
      }
    }
  }
}

template <int KE, bool FUSED>
hipError_t launch_dgrad(const C16Params &p, const void *g, const uint32_t *mask, const void *w, float alpha,
                        void *dx, hipStream_t st) {
  using G = C16B<KE, FUSED>;
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
  int blocks = (int)std::min<long long>(tiles, cus);
  blocks = std::max(8, (blocks + 7) / 8 * 8);
  hipLaunchKernelGGL((c16_dgrad_kernel<KE, FUSED>), dim3(blocks), dim3(64 * NWAVE), G::LDS_BYTES, st,
                     (const uint16_t *)g, mask, (const uint16_t *)w, alpha, (uint16_t *)dx, p);
  return hipGetLastError();
}

}  // namespace

// 32-bit byte offsets into dz (unfused) or the pooled gradient and the mask (fused)
bool c16_bwd_supported(const ConvShape &s) {
  return c16_fwd_supported(s) && (long long)s.n * s.od * s.oh * s.ow * s.co * 2 < (1LL << 31);
}

hipError_t launch_conv_bwd_data_c16(const ConvShape &s, const void *g, const uint32_t *mask, const void *w,
                                    float alpha, void *dx, bool fused, hipStream_t st) {
  C16Params p{};
  p.n = s.n; p.d = s.d; p.h = s.h; p.w = s.w;
  p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.od = s.od; p.oh = s.oh; p.ow = s.ow;
  p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
  p.g_bytes = fused ? (int)((long long)s.n * p.pod * p.poh * p.pow_ * 32 * 2)
                    : (int)((long long)s.n * s.od * s.oh * s.ow * 32 * 2);
  p.m_bytes = (int)((long long)s.n * s.od * s.oh * s.ow * 4);
#define CF_C16B_CASE(KEV)                                                                   \
  if (s.kd == KEV)                                                                          \
    return fused ? launch_dgrad<KEV, true>(p, g, mask, w, alpha, dx, st)                    \
                 : launch_dgrad<KEV, false>(p, g, mask, w, alpha, dx, st);
  CF_C16B_CASE(2) CF_C16B_CASE(3) CF_C16B_CASE(4)
#undef CF_C16B_CASE
  return hipErrorInvalidValue;
}

}  // namespace cf
