// conv_c16_wgrad.hip -- backward weights of the 16 -> 32 channel 4^3 stride-1 layer (gfx950, bf16).
//
// Backward weights (Section III-C) is a convolution with a long reduction
// over voxels and a small output: dW[t, ci, co] = sum_v x~[v + t, ci] dz[v, co].
// On v_mfma_f32_16x16x32_bf16 one instruction is one tap:
//   A (16 x 32) = 16 input channels x 32 consecutive voxels of the input halo
//                 shifted by the tap,
//   B (32 x 16) = the same 32 voxels of dz x 16 output channels,
//   D (16 x 16) += dW[tap][ci][co-block].
// Both operands need 8 consecutive voxels per lane while the tensors are
// channels-innermost (NDHWC).  The tiles are therefore kept in LDS in their
// natural layout and read with ds_read_b64_tr_b16, the gfx950 transposing
// LDS load: inside each 16-lane group, lane 4a+b receives element b of the
// 4-element rows addressed by lanes a, a+4, a+8, a+12.  Pointing lane r of
// the group at (voxel r/4 + 4t, channels 4(r%4) .. +3) and issuing t = 0, 1
// hands lane i channel i of 8 consecutive voxels -- any voxel offset, so the
// tap shift along w costs nothing.
//
// Work split: wave w owns the 16 taps with kd = w (all kh, kw, both 16-wide
// output-channel blocks: 32 accumulators); a persistent workgroup loops over
// 2x4x32-voxel dz tiles, staging the tile and its input halo in LDS, and in
// every (d-row, kw) step reuses one A fragment (input row h') for the k taps
// kh that reach dz rows h = h' - kh.  Each workgroup writes its fp32 partial
// dW once; a second kernel sums the partials in workgroup order.
//
// Fused variant: dz is rebuilt from the pooled-output gradient and the slope
// mask while staging (rounded to bf16 as the unfused path stores it), and the
// bias gradient is summed from the unrounded values in the same pass.  The
// tiles partition dz, so every element is built exactly once; when the caller
// asks for it, the staged dz is also written out (one 16-byte store per staged
// unit) for a following backward-data pass.

#include "cf_common.h"
#include "cf_kernels.h"

namespace cf {
namespace {

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;

constexpr int KE = 4;
constexpr int TD = 2, TH = 4, TW = 32;
constexpr int HD = TD + KE - 1, HH = TH + KE - 1, HW = TW + KE - 1;
constexpr int XH_VEC = HD * HH * HW * 2;    // 16-byte units of the input halo (16 ci = 2 units)
constexpr int DZ_VEC = TD * TH * TW * 4;    // 16-byte units of the dz tile (32 co = 4 units)
constexpr int DB_VEC = 256 * 2;             // fused: per-thread running bias sums (8 floats)
constexpr int NXC = (XH_VEC + 255) / 256, NZ = DZ_VEC / 256;  // DMA instructions per wave
constexpr int XH_PAD = NXC * 256;           // the last DMA instructions write padding slots
constexpr int LDS_BYTES = (XH_PAD + DZ_VEC + DB_VEC) * 16;
static_assert(DZ_VEC % 256 == 0, "dz staging");

// two transposing reads -> 8 consecutive voxels of one channel per lane
__device__ __forceinline__ bf16x8_t tr_frag(const uint16_t *lds, int e0, int e1) {
  const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(lds + e0));
  const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(lds + e1));
  typedef short v8i16_t __attribute__((ext_vector_type(8)));
  const v8i16_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}

template <bool FUSED>
__global__ __launch_bounds__(256, 2) void c16_wgrad_kernel(const uint16_t *__restrict__ x,
                                                           const uint16_t *__restrict__ g,
                                                           const uint32_t *__restrict__ mask, float alpha,
                                                           float *__restrict__ part_w, float *__restrict__ part_b,
                                                           uint16_t *__restrict__ dz_out, C16Params p) {
  __shared__ __attribute__((aligned(16))) uint4 smem[(LDS_BYTES + 15) / 16];
  uint4 *xh = smem;                 // [HD][HH][HW][2 x 8 ci]
  uint4 *dzt = smem + XH_PAD;       // [TD][TH][TW][4 x 8 co]
  const uint16_t *xh16 = reinterpret_cast<const uint16_t *>(xh);
  const uint16_t *dz16 = reinterpret_cast<const uint16_t *>(dzt);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, q = lane >> 4;
  // transposing-read row of this lane: voxel r16/4 (+4 for the second read), channel group r16%4
  const int trv = r16 >> 2, trc = 4 * (r16 & 3);

  const int tiles_w = (p.ow + TW - 1) / TW, tiles_h = (p.oh + TH - 1) / TH, tiles_d = (p.od + TD - 1) / TD;
  const int tiles = p.n * tiles_d * tiles_h * tiles_w;
  const int nblk = gridDim.x;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, per_xcd_blocks = (nblk + 7) >> 3;
  const int per = (tiles + 7) >> 3;

  f32x4_t acc[KE][KE][2];  // [kh][kw][co block]
#pragma unroll
  for (int a = 0; a < KE; ++a)
#pragma unroll
    for (int b = 0; b < KE; ++b)
#pragma unroll
      for (int c = 0; c < 2; ++c) acc[a][b][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // fused: running bias-gradient sums of this thread's 8 staged channels live in
  // LDS between tiles, so they hold no registers across the MFMA section
  float4 *dbl = reinterpret_cast<float4 *>(smem + XH_PAD + DZ_VEC) + 2 * tid;
  if constexpr (FUSED) {
    dbl[0] = make_float4(0.f, 0.f, 0.f, 0.f);
    dbl[1] = make_float4(0.f, 0.f, 0.f, 0.f);
  }

  // Input halo by buffer -> LDS DMA: per DMA slot e = 64 * (wave + 4k) + lane
  // (slot order = the [hd][hh][hw][half] layout), computed once: the byte
  // offset relative to the halo origin and the packed coordinates
  // hw | hh << 6 | hd << 9 (31 << 9 marks the padding slots past the halo).
  const __amdgpu_buffer_rsrc_t xrsrc = __builtin_amdgcn_make_buffer_rsrc((void *)x, (short)0, p.x_bytes, 0x00020000);
  typedef __attribute__((address_space(3))) void lds_void_t;
  uint32_t xrel[NXC], xpk[NXC];
#pragma unroll
  for (int k = 0; k < NXC; ++k) {
    const int e = 64 * (wave + 4 * k) + lane;
    const int hf = e & 1, v = e >> 1;
    const int hw = v % HW, hh = (v / HW) % HH, hd = v / (HW * HH);
    // padding slots: an offset past every buffer (the range check, which does
    // not include the scalar offset, returns zeros)
    xrel[k] = e < XH_VEC ? (uint32_t)((((hd * p.h + hh) * p.w + hw) * 16 + 8 * hf) * 2) : 0x80000000u;
    xpk[k] = e < XH_VEC ? (uint32_t)(hw | hh << 6 | hd << 9) : 31u << 9;
  }
  // unfused dz tile likewise: slot e = (voxel of the tile) * 4 + channel quarter
  const __amdgpu_buffer_rsrc_t grsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)g, (short)0, FUSED ? 0 : p.g_bytes, 0x00020000);
  uint32_t zrel[NZ], zpk[NZ];
#pragma unroll
  for (int k = 0; k < NZ; ++k) {
    const int e = 64 * (wave + 4 * k) + lane;
    const int cq = e & 3, v = e >> 2;
    const int lw = v % TW, lh = (v / TW) % TH, ld = v / (TW * TH);
    zrel[k] = (uint32_t)((((ld * p.oh + lh) * p.ow + lw) * 32 + 8 * cq) * 2);
    zpk[k] = (uint32_t)(lw | lh << 6 | ld << 9);
  }

  for (int i = slot;; i += per_xcd_blocks) {
    const int t = xcd * per + i;
    if (i >= per || t >= tiles) break;
    int r = t;
    const int tw = r % tiles_w; r /= tiles_w;
    const int th = r % tiles_h; r /= tiles_h;
    const int td = r % tiles_d;
    const int n = r / tiles_d;
    const int o0d = td * TD, o0h = th * TH, o0w = tw * TW;

    __syncthreads();  // every wave is done with the previous tile's LDS
    // ---- stage the input halo (DMA) and the dz tile ----------------------------
    {
      const int x0d = o0d - p.pd, x0h = o0h - p.ph, x0w = o0w - p.pw;  // halo origin (may be < 0)
      const uint32_t base = (uint32_t)(((n * p.d + x0d) * p.h + x0h) * p.w + x0w) * 32u;
      const bool xin = x0d >= 0 && x0d + HD <= p.d && x0h >= 0 && x0h + HH <= p.h && x0w >= 0 && x0w + HW <= p.w;
      if (xin) {
        // the whole halo is inside x: per-slot offsets as computed once, the
        // tile's base in the scalar offset
#pragma unroll
        for (int k = 0; k < NXC; ++k)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(xrsrc, (lds_void_t *)(xh + 64 * (wave + 4 * k)), 16, xrel[k],
                                                   (int)base, 0, 0);
      } else {
#pragma unroll
        for (int k = 0; k < NXC; ++k) {
          uint32_t pk = xpk[k];
          asm volatile("" : "+v"(pk));  // keep the decoded fields out of the tile loop's registers
          const int hw = pk & 63, hh = (pk >> 6) & 7, hd = pk >> 9;
          const bool ok = pk < (uint32_t)(HD << 9) && (unsigned)(x0w + hw) < (unsigned)p.w &&
                          (unsigned)(x0h + hh) < (unsigned)p.h && (unsigned)(x0d + hd) < (unsigned)p.d;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(xrsrc, (lds_void_t *)(xh + 64 * (wave + 4 * k)), 16,
                                                   ok ? xrel[k] + base : 0x80000000u, 0, 0, 0);
        }
      }
      if constexpr (!FUSED) {
        const uint32_t zbase = (uint32_t)(((n * p.od + o0d) * p.oh + o0h) * p.ow + o0w) * 64u;
#pragma unroll
        for (int k = 0; k < NZ; ++k) {
          uint32_t pk = zpk[k];
          asm volatile("" : "+v"(pk));
          const int lw = pk & 63, lh = (pk >> 6) & 7, ld = pk >> 9;
          const bool ok = o0w + lw < p.ow && o0h + lh < p.oh && o0d + ld < p.od;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(grsrc, (lds_void_t *)(dzt + 64 * (wave + 4 * k)), 16,
                                                   ok ? zrel[k] + zbase : 0x80000000u, 0, 0, 0);
        }
      }
    }
    float dbs[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) dbs[j] = 0.f;
    if constexpr (FUSED) {
      // unit k of this thread: voxel (ld, lh, lw) of the tile (packed in zpk),
      // channels 8 cq .. 8 cq + 7 with cq = tid & 3.  The tile origins are even
      // in every dimension, so voxel and pooled-voxel indices are a per-tile
      // base plus a per-unit offset; interior tiles skip the bounds tests.
      const int cq = tid & 3;
      const int vox0 = ((n * p.od + o0d) * p.oh + o0h) * p.ow + o0w;
      const int pool0 = ((n * p.pod + (o0d >> 1)) * p.poh + (o0h >> 1)) * p.pow_ + (o0w >> 1);
      // every voxel of the tile and its pooled voxel exist
      const bool interior = o0d + TD <= 2 * p.pod && o0h + TH <= 2 * p.poh && o0w + TW <= 2 * p.pow_;
      // dz = g / 8 * slope: the scale by 2^-3 is exact, so folding it into the
      // slope gives the same bits as scaling first
      const float s1 = 0.125f, sa = 0.125f * alpha;
      // 8 channels of one voxel: dz (bf16 pairs) and the running bias sums
      auto rebuild = [&](int pv, int vox) {
        Vec16<DT_BF16> gv;
        gv.u = *reinterpret_cast<const uint4 *>(g + (pv * 32 + 8 * cq));
        const uint32_t bits = mask[vox] >> (8 * cq);
        float d[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          // slope bits picked by the sign-extended mask bit (all ones or zero)
          const uint32_t m = (uint32_t)__builtin_amdgcn_sbfe((int)bits, j, 1);
          uint32_t sl;
          asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(sl) : "v"(m), "s"(__float_as_uint(s1)), "v"(__float_as_uint(sa)));
          d[j] = bf2f(gv.e[j]) * __uint_as_float(sl);
          dbs[j] += d[j];
        }
        return make_uint4(f2bf2(d[0], d[1]), f2bf2(d[2], d[3]), f2bf2(d[4], d[5]), f2bf2(d[6], d[7]));
      };
      if (interior) {
#pragma unroll
        for (int k = 0; k < NZ; ++k) {
          uint32_t pk = zpk[k];
          asm volatile("" : "+v"(pk));  // keep the decoded fields out of the tile loop's registers
          const int lw = pk & 63, lh = (pk >> 6) & 7, ld = pk >> 9;
          const int vox = vox0 + (int)__umul24(__umul24(ld, p.oh) + lh, p.ow) + lw;
          const int pv = pool0 + (int)__umul24(__umul24(ld >> 1, p.poh) + (lh >> 1), p.pow_) + (lw >> 1);
          const uint4 val = rebuild(pv, vox);
          if (dz_out) *reinterpret_cast<uint4 *>(dz_out + (vox * 32 + 8 * cq)) = val;
          dzt[tid + 256 * k] = val;  // the tile region is free: every read of it ended at the barrier above
        }
      } else {
#pragma unroll
        for (int k = 0; k < NZ; ++k) {
          uint32_t pk = zpk[k];
          asm volatile("" : "+v"(pk));
          const int lw = pk & 63, lh = (pk >> 6) & 7, ld = pk >> 9;
          const int od = o0d + ld, oh = o0h + lh, ow = o0w + lw;
          const bool in_dz = od < p.od && oh < p.oh && ow < p.ow;
          const bool in_p = (od >> 1) < p.pod && (oh >> 1) < p.poh && (ow >> 1) < p.pow_;
          const int vox = vox0 + (int)__umul24(__umul24(ld, p.oh) + lh, p.ow) + lw;
          const int pv = pool0 + (int)__umul24(__umul24(ld >> 1, p.poh) + (lh >> 1), p.pow_) + (lw >> 1);
          uint4 val = make_uint4(0, 0, 0, 0);
          if (in_dz) {
            if (in_p) val = rebuild(pv, vox);
            if (dz_out) *reinterpret_cast<uint4 *>(dz_out + (vox * 32 + 8 * cq)) = val;
          }
          dzt[tid + 256 * k] = val;
        }
      }
      float4 a = dbl[0], b = dbl[1];
      a.x += dbs[0]; a.y += dbs[1]; a.z += dbs[2]; a.w += dbs[3];
      b.x += dbs[4]; b.y += dbs[5]; b.z += dbs[6]; b.w += dbs[7];
      dbl[0] = a;
      dbl[1] = b;
    }
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this wave's DMA has landed
    __syncthreads();

    // ---- MFMA: taps kd = wave; reuse A (input row h') over kh ----------------
    if (wave < KE) {
#pragma unroll 1
      for (int ld = 0; ld < TD; ++ld) {
        bf16x8_t bfr[TH][2];
#pragma unroll
        for (int hh = 0; hh < TH; ++hh)
#pragma unroll
          for (int nf = 0; nf < 2; ++nf) {
            const int e0 = (((ld * TH + hh) * TW + 8 * q + trv) * 32) + 16 * nf + trc;
            bfr[hh][nf] = tr_frag(dz16, e0, e0 + 4 * 32);
          }
#pragma unroll
        for (int kw = 0; kw < KE; ++kw) {
          // input rows h' stream through a two-deep register pipeline: the next
          // row's transposing reads are in flight while this row's MFMAs issue
          auto arow = [&](int hi) {
            const int e0 = ((((ld + wave) * HH + hi) * HW + 8 * q + trv + kw) * 16) + trc;
            return tr_frag(xh16, e0, e0 + 4 * 16);
          };
          bf16x8_t a_cur = arow(0), a_nxt = a_cur;
#pragma unroll
          for (int hi = 0; hi < TH + KE - 1; ++hi) {
            if (hi + 1 < TH + KE - 1) a_nxt = arow(hi + 1);
#pragma unroll
            for (int kh = 0; kh < KE; ++kh) {
              const int hrow = hi - kh;
              if (hrow >= 0 && hrow < TH) {
                acc[kh][kw][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_cur, bfr[hrow][0], acc[kh][kw][0], 0, 0, 0);
                acc[kh][kw][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_cur, bfr[hrow][1], acc[kh][kw][1], 0, 0, 0);
              }
            }
            a_cur = a_nxt;
          }
        }
      }
    }
  }

  // ---- this workgroup's partials: D lane = co (16 nf + r16), rows 4q + j = ci ----
  if (wave < KE) {
    float *pw = part_w + (long long)blockIdx.x * (KE * KE * KE * 16 * 32);
#pragma unroll
    for (int kh = 0; kh < KE; ++kh)
#pragma unroll
      for (int kw = 0; kw < KE; ++kw) {
        const int tap = (wave * KE + kh) * KE + kw;
#pragma unroll
        for (int nf = 0; nf < 2; ++nf)
#pragma unroll
          for (int j = 0; j < 4; ++j) pw[(tap * 16 + 4 * q + j) * 32 + 16 * nf + r16] = acc[kh][kw][nf][j];
      }
  }
  if constexpr (FUSED) {
    // thread's channels: 8 * ((tid) & 3) .. +7 (staging unit e & 3 == tid & 3)
    // slot of thread u holds channels 8 (u & 3) .. +7: sum the 64 threads of each group in order
    __syncthreads();
    const float *red = reinterpret_cast<const float *>(smem + XH_PAD + DZ_VEC);
    if (tid < 32) {
      float s = 0.f;
      for (int k = 0; k < 64; ++k) s += red[(4 * k + (tid >> 3)) * 8 + (tid & 7)];
      part_b[(long long)blockIdx.x * 32 + tid] = s;
    }
  }
}

int wgrad_blocks(const C16Params &p) {
  const long long tiles = (long long)p.n * ((p.od + TD - 1) / TD) * ((p.oh + TH - 1) / TH) * ((p.ow + TW - 1) / TW);
  int blocks = (int)std::min<long long>(tiles, 2LL * kNumCUs);
  return std::max(8, (blocks + 7) / 8 * 8);
}

template <bool FUSED>
hipError_t launch_w(const C16Params &p, const void *x, const void *g, const uint32_t *mask, float alpha, float *pw,
                    float *pb, void *dz_out, int blocks, hipStream_t st) {
  hipLaunchKernelGGL((c16_wgrad_kernel<FUSED>), dim3(blocks), dim3(256), 0, st, (const uint16_t *)x,
                     (const uint16_t *)g, mask, alpha, pw, pb, (uint16_t *)dz_out, p);
  return hipGetLastError();
}

C16Params params_of(const ConvShape &s) {
  C16Params p{};
  p.n = s.n; p.d = s.d; p.h = s.h; p.w = s.w;
  p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.od = s.od; p.oh = s.oh; p.ow = s.ow;
  p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
  p.x_bytes = (int)((long long)s.n * s.d * s.h * s.w * 16 * 2);
  p.g_bytes = (int)((long long)s.n * s.od * s.oh * s.ow * 32 * 2);
  return p;
}

}  // namespace

// 32-bit byte offsets into x and dz
bool c16_wgrad_supported(const ConvShape &s) {
  return c16_fwd_supported(s) && s.kd == KE && (long long)s.n * s.od * s.oh * s.ow * 32 * 2 < (1LL << 31);
}

size_t c16_wgrad_workspace(const ConvShape &s) {
  const int blocks = wgrad_blocks(params_of(s));
  return (size_t)blocks * (KE * KE * KE * 16 * 32 + 32) * sizeof(float);
}

hipError_t launch_conv_bwd_weight_c16(const ConvShape &s, const void *x, const void *g, const uint32_t *mask,
                                      float alpha, float *dw, float *db, void *ws, bool fused, void *dz_out,
                                      hipStream_t st) {
  const C16Params p = params_of(s);
  const int blocks = wgrad_blocks(p);
  const int cols = KE * KE * KE * 16 * 32;
  float *pw = (float *)ws;
  float *pb = pw + (size_t)blocks * cols;
  hipError_t e = fused ? launch_w<true>(p, x, g, mask, alpha, pw, pb, dz_out, blocks, st)
                       : launch_w<false>(p, x, g, mask, alpha, pw, pb, nullptr, blocks, st);
  if (e != hipSuccess) return e;
  e = launch_sum_rows(pw, dw, blocks, cols, st);
  if (e != hipSuccess || !fused) return e;
  return launch_sum_rows(pb, db, blocks, 32, st);
}

}  // namespace cf
