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
//   B (32 x 16)  = W[tap][ci][co] read as [co][ci] (16 contiguous bytes per lane),
//   D (16 x 16)  = 16 voxels x all 16 input channels.
//
// Weights stay in registers.  A workgroup is four waves, one per SIMD, and
// two workgroups share a CU.  The taps are split into NS groups along kd
// (NS = 2 for the 4^3 kernel, whose 32 fragments per group fill 128 VGPRs;
// NS = 1 otherwise); every wave loads its group's B fragments once and keeps
// them for the whole persistent loop, so the MFMA loop issues no global loads
// at all.  A 4x4x16 dx tile is split into NWAVE / NS slots of WD planes; the
// two tap groups of a slot add their partial sums through LDS.
//
// The zero-padded dz halo of the tile sits in LDS as [co/8][d][h][w] x 16
// bytes, each channel-quarter plane padded to a multiple of 256 bytes.  An A
// fragment is then one ds_read_b128 whose 16-lane quarters each read 256
// contiguous bytes at the same offset modulo 256, which keeps every pair of
// consecutive 8-lane chunks on disjoint banks (no conflict cycles).  The halo
// arrives by buffer -> LDS DMA; a padding voxel gets a byte offset past the
// buffer, which the hardware range check turns into zeros.  Interior tiles
// add a per-tile base to offsets computed once per kernel.
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

constexpr int TD = 4, TH = 4, TW = 16;  // dx tile (voxels)
constexpr int NWAVE = 4;                // one wave per SIMD, two workgroups per CU

template <int KE, bool FUSED>
struct C16B {
  static constexpr int NS = KE == 4 ? 2 : 1;    // tap groups along kd
  static constexpr int KD0 = KE / NS;           // kd taps per group
  static constexpr int NSLOT = NWAVE / NS;      // spatial slots of a tile
  static constexpr int WD = TD / NSLOT;         // dx planes per slot
  static constexpr int HD = TD + KE - 1, HH = TH + KE - 1, HW = TW + KE - 1;
  static constexpr int HVOX = HD * HH * HW;
  static constexpr int PLANE = (HVOX + 15) / 16 * 16;  // 16-byte slots per channel quarter
  static constexpr int HALO = 4 * PLANE;                // a multiple of 64
  static constexpr int HCH = HALO / 64;                 // DMA instructions per tile
  // fused staging: pooled-gradient box [cq][pd][ph][pw] and mask words [hd][hh][hw]
  static constexpr int PD = HD / 2 + 1, PH = HH / 2 + 1, PW = HW / 2 + 1;
  static constexpr int GVOX = PD * PH * PW;
  static constexpr int GBOX = FUSED ? 4 * GVOX : 0;
  static constexpr int GCH = (GBOX + 63) / 64;
  static constexpr int MCH = FUSED ? (HVOX + 63) / 64 : 0;
  // partial sums handed between the tap groups: [slot][plane][row][lane] x 16 bytes
  static constexpr int RED = NS == 2 ? NSLOT * WD * TH * 64 : 0;
  static constexpr int OFF_G = HALO * 16;
  static constexpr int OFF_M = OFF_G + GCH * 64 * 16;
  static constexpr int END_M = OFF_M + MCH * 64 * 4;
  static constexpr int OFF_R = FUSED ? 0 : END_M;  // fused: partial sums reuse the halo
  static constexpr int LDS_BYTES = END_M > OFF_R + RED * 16 ? END_M : OFF_R + RED * 16;
  // DMA instructions per wave
  static constexpr int HK = (HCH + NWAVE - 1) / NWAVE;
  static constexpr int GK = (GCH + NWAVE - 1) / NWAVE;
  static constexpr int MK = (MCH + NWAVE - 1) / NWAVE;
  static_assert(RED * 16 <= HALO * 16 || !FUSED, "partial sums must fit in the halo");
  static_assert(2 * LDS_BYTES <= 160 * 1024, "two workgroups per CU");
};

typedef __attribute__((address_space(3))) void lds_void_t;
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
constexpr uint32_t OOB = 0x80000000u;  // a byte offset the range check always rejects

template <int KE, bool FUSED>
__global__ __launch_bounds__(256, 2) void c16_dgrad_kernel(const uint16_t *__restrict__ g,
                                                           const uint32_t *__restrict__ mask,
                                                           const uint16_t *__restrict__ w, float alpha,
                                                           uint16_t *__restrict__ dx, C16Params p) {
  using G = C16B<KE, FUSED>;
  __shared__ __attribute__((aligned(16))) uint4 smem[(G::LDS_BYTES + 15) / 16];
  unsigned char *lds = reinterpret_cast<unsigned char *>(smem);
  uint4 *halo = smem;                                            // [4][PLANE]
  uint4 *gbx = reinterpret_cast<uint4 *>(lds + G::OFF_G);        // fused: [4][PD][PH][PW]
  uint32_t *mkw = reinterpret_cast<uint32_t *>(lds + G::OFF_M);  // fused: [HD][HH][HW]
  f32x4_t *red = reinterpret_cast<f32x4_t *>(lds + G::OFF_R);    // two tap groups: partial sums
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, q = lane >> 4;
  const int slot = wave % G::NSLOT, grp = wave / G::NSLOT;
  const int pdp = KE - 1 - p.pd, php = KE - 1 - p.ph, pwp = KE - 1 - p.pw;  // flipped-kernel pads

  // here (d, h, w) is the dx extent and (od, oh, ow) the dz extent
  const int tiles_w = (p.w + TW - 1) / TW, tiles_h = (p.h + TH - 1) / TH, tiles_d = (p.d + TD - 1) / TD;
  const int tiles = p.n * tiles_d * tiles_h * tiles_w;
  const int xcd = blockIdx.x & 7, bslot = blockIdx.x >> 3, nb8 = gridDim.x >> 3;
  const int per = (tiles + 7) >> 3;  // contiguous tile range of one XCD
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
  // Per DMA slot, computed once: the tile-invariant part of its byte offset
  // (relative to the box origin) and its box coordinates packed as
  // x | y << 5 | z << 10 (x innermost; a padding slot gets z = 31, which no
  // validity mask covers).  A boundary tile tests the coordinates against
  // per-tile bitmasks of the valid x, y and z (one bit-field extract each).
  uint32_t hrel[G::HK > 0 ? G::HK : 1], hpk[G::HK > 0 ? G::HK : 1];
  uint32_t grel[G::GK > 0 ? G::GK : 1], gpk[G::GK > 0 ? G::GK : 1];
  uint32_t mrel[G::MK > 0 ? G::MK : 1], mpk[G::MK > 0 ? G::MK : 1];
  if constexpr (!FUSED) {
#pragma unroll
    for (int k = 0; k < G::HK; ++k) {
      const int s = 64 * (wave + NWAVE * k) + lane;
      const int cq = s / G::PLANE, v = s % G::PLANE;
      const int hw = v % G::HW, hh = (v / G::HW) % G::HH, hd = v / (G::HW * G::HH);
      const bool ok = s < G::HALO && v < G::HVOX;
      hrel[k] = (uint32_t)((((hd * p.oh + hh) * p.ow + hw) * 32 + 8 * cq) * 2);
      hpk[k] = ok ? (uint32_t)(hw | hh << 5 | hd << 10) : 31u << 10;
    }
  } else {
#pragma unroll
    for (int k = 0; k < G::GK; ++k) {
      const int s = 64 * (wave + NWAVE * k) + lane;
      const int cq = s / G::GVOX, v = s % G::GVOX;
      const int pw_ = v % G::PW, ph_ = (v / G::PW) % G::PH, pd_ = v / (G::PW * G::PH);
      grel[k] = (uint32_t)((((pd_ * p.poh + ph_) * p.pow_ + pw_) * 32 + 8 * cq) * 2);
      gpk[k] = s < G::GBOX ? (uint32_t)(pw_ | ph_ << 5 | pd_ << 10) : 31u << 10;
    }
#pragma unroll
    for (int k = 0; k < G::MK; ++k) {
      const int s = 64 * (wave + NWAVE * k) + lane;
      const int hw = s % G::HW, hh = (s / G::HW) % G::HH, hd = s / (G::HW * G::HH);
      mrel[k] = (uint32_t)(((hd * p.oh + hh) * p.ow + hw) * 4);
      mpk[k] = s < G::HVOX ? (uint32_t)(hw | hh << 5 | hd << 10) : 31u << 10;
    }
  }
  // bits [lo, hi) of the valid box coordinates along one dimension: 0 <= s0 + i < n
  auto vbits = [](int s0, int len, int n) {
    const int lo = s0 < 0 ? -s0 : 0, hi = n - s0 < len ? n - s0 : len;
    return hi > lo ? ((1u << hi) - 1u) & ~((1u << lo) - 1u) : 0u;
  };
  // one DMA instruction of a box: interior boxes add the base, boundary boxes
  // also test the slot's coordinates (opaque here, so that nothing derived from
  // them is hoisted out of the tile loop into registers)
  auto box_dma = [&](const __amdgpu_buffer_rsrc_t &rs, void *dst, int bytes, uint32_t rel, uint32_t pk, bool inside,
                     uint32_t base, uint32_t mx, uint32_t my, uint32_t mz) {
    uint32_t off = rel + base;
    if (!inside) {
      asm volatile("" : "+v"(pk));
      const uint32_t ok = __builtin_amdgcn_ubfe(mx, pk, 1) & __builtin_amdgcn_ubfe(my, pk >> 5, 1) &
                          __builtin_amdgcn_ubfe(mz, pk >> 10, 1);
      off = ok ? off : OOB;
    }
    if (bytes == 16)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t *)dst, 16, off, 0, 0, 0);
    else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t *)dst, 4, off, 0, 0, 0);
  };
  auto issue = [&](int t) {
    const Org o = origin(t);
    const int s0d = o.x0d - pdp, s0h = o.x0h - php, s0w = o.x0w - pwp;  // halo origin in dz (may be < 0)
    const bool inside = s0d >= 0 && s0h >= 0 && s0w >= 0 && s0d + G::HD <= p.od && s0h + G::HH <= p.oh &&
                        s0w + G::HW <= p.ow;
    const uint32_t vx = vbits(s0w, G::HW, p.ow), vy = vbits(s0h, G::HH, p.oh), vz = vbits(s0d, G::HD, p.od);
    const int hvox0 = ((o.n * p.od + s0d) * p.oh + s0h) * p.ow + s0w;  // dz voxel index of the origin
    if constexpr (!FUSED) {
#pragma unroll
      for (int k = 0; k < G::HK; ++k) {
        const int c = wave + NWAVE * k;
        if (c < G::HCH) box_dma(grsrc, halo + 64 * c, 16, hrel[k], hpk[k], inside, (uint32_t)hvox0 * 64u, vx, vy, vz);
      }
    } else {
      const int p0d = s0d >> 1, p0h = s0h >> 1, p0w = s0w >> 1;  // floor
      const bool pin = p0d >= 0 && p0h >= 0 && p0w >= 0 && p0d + G::PD <= p.pod && p0h + G::PH <= p.poh &&
                       p0w + G::PW <= p.pow_;
      const uint32_t px = vbits(p0w, G::PW, p.pow_), py = vbits(p0h, G::PH, p.poh), pz = vbits(p0d, G::PD, p.pod);
      const int pvox0 = ((o.n * p.pod + p0d) * p.poh + p0h) * p.pow_ + p0w;
#pragma unroll
      for (int k = 0; k < G::GK; ++k) {
        const int c = wave + NWAVE * k;
        if (c < G::GCH) box_dma(grsrc, gbx + 64 * c, 16, grel[k], gpk[k], pin, (uint32_t)pvox0 * 64u, px, py, pz);
      }
#pragma unroll
      for (int k = 0; k < G::MK; ++k) {
        const int c = wave + NWAVE * k;
        if (c < G::MCH) box_dma(mrsrc, mkw + 64 * c, 4, mrel[k], mpk[k], inside, (uint32_t)hvox0 * 4u, vx, vy, vz);
      }
    }
  };

  // ---- the wave's weight fragments, kept for the whole kernel ---------------
  // flipped tap (kd', kh', kw') with kd' = grp * KD0 + kdl:
  // W[k-1-kd'][k-1-kh'][k-1-kw'][ci = r16][co = 8q .. 8q+7]
  const __amdgpu_buffer_rsrc_t wrsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)w, (short)0, KE * KE * KE * 16 * 32 * 2, 0x00020000);
  const int wlane = (r16 * 32 + 8 * q) * 2;
  bf16x8_t bw[G::KD0][KE][KE];
#pragma unroll
  for (int kdl = 0; kdl < G::KD0; ++kdl)
#pragma unroll
    for (int kh = 0; kh < KE; ++kh)
#pragma unroll
      for (int kw = 0; kw < KE; ++kw) {
        const int kd = grp * G::KD0 + kdl;
        const int tap = ((KE - 1 - kd) * KE + (KE - 1 - kh)) * KE + (KE - 1 - kw);
        const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(wrsrc, wlane, tap * 16 * 32 * 2, 0);
        bw[kdl][kh][kw] = __builtin_bit_cast(bf16x8_t, v);
      }

  auto tile_at = [&](int i) { return xcd * per + bslot + i * nb8; };
  auto valid_at = [&](int i) { return bslot + i * nb8 < per && tile_at(i) < tiles; };
  if (valid_at(0)) issue(tile_at(0));

  for (int i = 0; valid_at(i); ++i) {
    const Org o = origin(tile_at(i));
    const bool has_next = valid_at(i + 1);

    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this wave's DMA (and the weights) have landed
    __syncthreads();                     // ... and every other wave's
    if constexpr (FUSED) {
      // build the dz halo from the staged pooled gradient and mask words, one
      // pooling window (2x2x2 voxels x 8 channels) per item: both candidate
      // values of the window are rounded once, every voxel selects per channel
      const int e0d = (o.x0d - pdp) & 1, e0h = (o.x0h - php) & 1, e0w = (o.x0w - pwp) & 1;
      const float a8 = 0.125f * alpha;
      for (int it = tid; it < G::GBOX; it += 64 * NWAVE) {
        const int cq = it / G::GVOX, v = it % G::GVOX;
        const int pwl = v % G::PW, phl = (v / G::PW) % G::PH, pdl = v / (G::PW * G::PH);
        const u32x4_t gv = __builtin_bit_cast(u32x4_t, gbx[it]);
        uint32_t one[4], slo[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float lo = __uint_as_float(gv[j] << 16), hi = __uint_as_float(gv[j] & 0xffff0000u);
          one[j] = (uint32_t)f2bf(lo * 0.125f) | ((uint32_t)f2bf(hi * 0.125f) << 16);
          slo[j] = (uint32_t)f2bf(lo * a8) | ((uint32_t)f2bf(hi * a8) << 16);
        }
        // the box starts at pooled voxel floor(s0 / 2), i.e. at halo index -(s0 & 1)
        const int hd0 = 2 * pdl - e0d, hh0 = 2 * phl - e0h, hw0 = 2 * pwl - e0w;
#pragma unroll
        for (int vv = 0; vv < 8; ++vv) {
          const int hd = hd0 + (vv >> 2), hh = hh0 + ((vv >> 1) & 1), hw = hw0 + (vv & 1);
          if ((unsigned)hd >= (unsigned)G::HD || (unsigned)hh >= (unsigned)G::HH || (unsigned)hw >= (unsigned)G::HW)
            continue;
          const int hv = (hd * G::HH + hh) * G::HW + hw;
          const uint32_t bits = mkw[hv] >> (8 * cq);
          u32x4_t dv;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            // all-ones halfword where the channel's slope bit is set
            const uint32_t mlo = (uint32_t)(((int)(bits << (31 - 2 * j))) >> 31) & 0x0000ffffu;
            const uint32_t mhi = (uint32_t)(((int)(bits << (30 - 2 * j))) >> 31) & 0xffff0000u;
            const uint32_t m = mlo | mhi;
            dv[j] = (one[j] & m) | (slo[j] & ~m);
          }
          halo[cq * G::PLANE + hv] = __builtin_bit_cast(uint4, dv);
        }
      }
      __syncthreads();
      if (has_next) issue(tile_at(i + 1));  // the staging areas are free: overlap the MFMA loop
    }

    // ---- MFMA: halo plane pl (relative to the wave's first), row r, w shift kw
    f32x4_t acc[G::WD][TH];
#pragma unroll
    for (int a = 0; a < G::WD; ++a)
#pragma unroll
      for (int b = 0; b < TH; ++b) acc[a][b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const uint4 *abase = halo + q * G::PLANE + (slot * G::WD + grp * G::KD0) * G::HH * G::HW + r16;
    // A fragments stream through a ring PF reads ahead of their MFMAs; the
    // interleaving strategy keeps several LDS reads in flight between MFMAs
    constexpr int NPL = G::WD + G::KD0 - 1, NR = TH + KE - 1, NA = KE * NPL * NR, PF = 3;
    auto aload = [&](int i) {
      const int kw = i / (NPL * NR), pl = (i / NR) % NPL, r = i % NR;
      return __builtin_bit_cast(bf16x8_t, abase[(pl * G::HH + r) * G::HW + kw]);
    };
    bf16x8_t ar[PF + 1];
    __builtin_amdgcn_iglp_opt(1);
#pragma unroll
    for (int i = 0; i < PF; ++i) ar[i] = aload(i);
#pragma unroll
    for (int kw = 0; kw < KE; ++kw)
#pragma unroll
      for (int pl = 0; pl < NPL; ++pl)
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          const int i = (kw * NPL + pl) * NR + r;
          if (i + PF < NA) {
            ar[(i + PF) % (PF + 1)] = aload(i + PF);
          }
#pragma unroll
          for (int od = 0; od < G::WD; ++od) {
            const int kdl = pl - od;
            if (kdl < 0 || kdl >= G::KD0) continue;
#pragma unroll
            for (int kh = 0; kh < KE; ++kh) {
              const int orow = r - kh;
              if (orow < 0 || orow >= TH) continue;
              acc[od][orow] =
                  __builtin_amdgcn_mfma_f32_16x16x32_bf16(ar[i % (PF + 1)], bw[kdl][kh][kw], acc[od][orow], 0, 0, 0);
            }
          }
        }

    __syncthreads();  // every wave is done with the halo
    if constexpr (!FUSED) {
      if (has_next) issue(tile_at(i + 1));
    }

    // ---- the two tap groups of a slot add their partial sums; group grp keeps plane grp
    f32x4_t res[TH];
    int pln = slot;
    if constexpr (G::NS == 2) {
      pln = slot * G::WD + grp;
#pragma unroll
      for (int r = 0; r < TH; ++r) {
        const f32x4_t other = grp ? acc[0][r] : acc[1][r];
        red[((slot * G::WD + (1 - grp)) * TH + r) * 64 + lane] = other;
      }
      __syncthreads();
#pragma unroll
      for (int r = 0; r < TH; ++r) {
        const f32x4_t mine = grp ? acc[1][r] : acc[0][r];
        res[r] = mine + red[((slot * G::WD + grp) * TH + r) * 64 + lane];
      }
    } else {
#pragma unroll
      for (int r = 0; r < TH; ++r) res[r] = acc[0][r];
    }

    // D: lane -> input channel r16, rows 4q + j -> voxel w within the 16-block
    const int vd = o.x0d + pln;
    if (vd < p.d) {
#pragma unroll
      for (int r = 0; r < TH; ++r) {
        const int vh = o.x0h + r;
        if (vh >= p.h) continue;
        const long long rowv = (((long long)o.n * p.d + vd) * p.h + vh) * p.w;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int vw = o.x0w + 4 * q + j;
          if (vw < p.w) dx[(rowv + vw) * 16 + r16] = f2bf(res[r][j]);
        }
      }
    }
  }
}

template <int KE, bool FUSED>
hipError_t launch_dgrad(const C16Params &p, const void *g, const uint32_t *mask, const void *w, float alpha,
                        void *dx, hipStream_t st) {
  const long long tiles = (long long)p.n * ((p.d + TD - 1) / TD) * ((p.h + TH - 1) / TH) * ((p.w + TW - 1) / TW);
  int blocks = (int)std::min<long long>(tiles, 2LL * kNumCUs);
  blocks = std::max(8, (blocks + 7) / 8 * 8);
  hipLaunchKernelGGL((c16_dgrad_kernel<KE, FUSED>), dim3(blocks), dim3(64 * NWAVE), 0, st,
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
