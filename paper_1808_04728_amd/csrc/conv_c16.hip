// conv_c16.hip -- 16 -> 32 channel stride-1 3D convolution forward (gfx950, bf16).
//
// The second CosmoFlow layer (4^3 taps, 16 -> 32 channels) carries most of
// the network's convolution FLOPs.  Its forward pass is the direct
// convolution of Section III-C (Algorithm 1: every output voxel is an inner
// product over taps and input channels), mapped onto
// v_mfma_f32_32x32x16_bf16:
//   A (32 x 16)  = 32 consecutive output voxels along w, one tap, 16 input
//                  channels -- exactly one voxel row of the input halo;
//   B (16 x 32)  = the tap's 16 x 32 weight slice;
//   D (32 x 32)  = those 32 voxels x all 32 output channels.
// A persistent workgroup (4 waves, one per SIMD) packs the whole weight
// tensor into LDS once, then loops over 8x4x32-voxel output tiles: it stages
// the zero-padded input halo of the tile in LDS and each wave computes a
// 2x4x32 brick (eight 32x32 accumulators).  One A fragment (input row h',
// shift kw) serves every output row h = h' - kh of the brick, so each LDS
// read feeds up to k MFMAs.
//
// LDS layouts keep every fragment read a contiguous 512-byte run per half
// wave: halo [d][h][ci/8][w][8 ci], weights [tap][ci/8][co][8 ci].
//
// Epilogues: store z; or bias + leaky ReLU + slope mask (+ 2^3 pool).  The
// 32x32 accumulator layout (lane = output channel, registers = voxels along
// w in runs of four) puts a whole 2x2x2 pooling window of one channel in one
// lane, so the pool is register arithmetic.
//
// Tiles are handed out XCD-major: workgroup b runs on XCD b % 8, and the
// eight XCDs own contiguous tile ranges, so halos shared by neighbouring tiles
// meet in the same L2.

#include "cf_common.h"
#include "cf_kernels.h"

namespace cf {
namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int TD = 8, TH = 4, TW = 32;  // output tile (voxels)
constexpr int NWAVE = 8;                // wave (dp, hp) owns the 2 x 2 x 32 brick d = 2dp.., h = 2hp..
constexpr int BH = 2;                   // brick rows per wave

template <int KE>
struct C16 {
  static constexpr int HD = TD + KE - 1, HH = TH + KE - 1, HW = TW + KE - 1;
  static constexpr int HALO_VEC = HD * HH * 2 * HW;           // 16-byte vectors (8 channels)
  static constexpr int HALO_PAD = (HALO_VEC + 63) / 64 * 64;  // whole 64-slot DMA chunks
  static constexpr int TAPS = KE * KE * KE;
  static constexpr int W_VEC = TAPS * 2 * 32;                 // [tap][ci/8][co] x 8 ci
  // per wave: the slope-ballot stage (16 x 8 bytes) and 64 junk slots (+ 15 x 8 of offsets)
  static constexpr int MSTAGE_WAVE = 128 + 4 * 64 + 8 * 16;
  static constexpr int LDS_BYTES = (HALO_PAD + W_VEC) * 16 + 8 * MSTAGE_WAVE;
};

// AMAX: alpha <= 1, where lrelu(u) = max(u, alpha u); else min(u, alpha u).
// Either form equals u > 0 ? u : alpha u bit for bit, and needs no lane mask.
template <int KE, int EPI, bool AMAX>
__global__ __launch_bounds__(512, 1) void conv_c16_fwd_kernel(const uint16_t *__restrict__ x,
                                                              const uint16_t *__restrict__ w,
                                                              const float *__restrict__ bias, float alpha,
                                                              uint16_t *__restrict__ out,
                                                              uint32_t *__restrict__ mask, C16Params p) {
  using G = C16<KE>;
  __shared__ __attribute__((aligned(16))) uint4 smem[(G::LDS_BYTES + 15) / 16];
  uint4 *halo = smem;                 // [HD][HH][2][HW] (+ padding to whole DMA chunks)
  uint4 *wp = smem + G::HALO_PAD;     // [TAPS][2][32]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, half = lane >> 5;

  // ---- pack W[tap][ci][co] into [tap][ci/8][co][8 ci] once ---------------
  // item = (tap, ci, 8-channel group of co): one 16-byte load, eight 2-byte LDS stores
  {
    constexpr int ITEMS = G::TAPS * 16 * 4;
    constexpr int PER = (ITEMS + 64 * NWAVE - 1) / (64 * NWAVE);
    uint4 wv[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = tid + 64 * NWAVE * k;
      wv[k] = e < ITEMS ? *reinterpret_cast<const uint4 *>(w + (long long)e * 8) : make_uint4(0, 0, 0, 0);
    }
    uint16_t *wp16 = reinterpret_cast<uint16_t *>(wp);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = tid + 64 * NWAVE * k;
      if (e >= ITEMS) continue;
      const int cg = e & 3, ci = (e >> 2) & 15, tap = e >> 6;
      Vec16<DT_BF16> v;
      v.u = wv[k];
#pragma unroll
      for (int j = 0; j < 8; ++j) wp16[(((tap * 2 + (ci >> 3)) * 32) + 8 * cg + j) * 8 + (ci & 7)] = v.e[j];
    }
  }

  const int tiles_w = (p.ow + TW - 1) / TW, tiles_h = (p.oh + TH - 1) / TH, tiles_d = (p.od + TD - 1) / TD;
  const int tiles = p.n * tiles_d * tiles_h * tiles_w;
  // XCD-major tile order: XCD x owns tiles [x*per, (x+1)*per)
  const int nblk = gridDim.x;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, per_xcd_blocks = (nblk + 7) >> 3;
  const int per = (tiles + 7) >> 3;
  float bz = 0.f;
  if constexpr (EPI != 0) bz = bias[col];

  // Halo staging by buffer -> LDS DMA (buffer_load_dwordx4 ... lds): wave w
  // fills 64-slot chunks w, w + 8, ... of the halo, lane l slot 64 c + l.  A
  // padding voxel gets a byte offset past the input buffer, which the range
  // check turns into zeros.  The next tile's DMA is issued once every wave has
  // finished reading the halo and completes during the epilogue -- no
  // registers hold it.
  const __amdgpu_buffer_rsrc_t xrsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)x, (short)0, p.x_bytes, 0x00020000);
  constexpr int NCHUNK = G::HALO_PAD / 64;
  auto issue_halo = [&](int t) {
    int r = t;
    const int tw = r % tiles_w; r /= tiles_w;
    const int th = r % tiles_h; r /= tiles_h;
    const int td = r % tiles_d;
    const int n = r / tiles_d;
    const int od0 = td * TD, oh0 = th * TH, ow0 = tw * TW;
    for (int c = wave; c < NCHUNK; c += NWAVE) {
      const int s = 64 * c + lane;
      const int hw = s % G::HW;
      const int t1 = s / G::HW;
      const int hf = t1 & 1, t2 = t1 >> 1;
      const int hh = t2 % G::HH, hd = t2 / G::HH;
      const int id = od0 - p.pd + hd, ih = oh0 - p.ph + hh, iw = ow0 - p.pw + hw;
      uint32_t off = 0x80000000u;
      if (s < G::HALO_VEC && (unsigned)id < (unsigned)p.d && (unsigned)ih < (unsigned)p.h && (unsigned)iw < (unsigned)p.w)
        off = (uint32_t)((((n * p.d + id) * p.h + ih) * p.w + iw) * 32 + 16 * hf);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xrsrc, (__attribute__((address_space(3))) void *)(halo + 64 * c), 16,
                                               off, 0, 0, 0);
    }
  };
  auto tile_of = [&](int i) { return xcd * per + i; };
  if (slot < per && tile_of(slot) < tiles) issue_halo(tile_of(slot));

  for (int i = slot;; i += per_xcd_blocks) {
    const int t = tile_of(i);
    if (i >= per || t >= tiles) break;
    int r = t;
    const int tw = r % tiles_w; r /= tiles_w;
    const int th = r % tiles_h; r /= tiles_h;
    const int td = r % tiles_d;
    const int n = r / tiles_d;
    const int od0 = td * TD, oh0 = th * TH, ow0 = tw * TW;

    // this wave's halo DMA has landed; after the barrier every wave's has (and
    // the packed weights are visible)
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
    __syncthreads();

    // ---- 2 x 2 x 32 brick of this wave ------------------------------------
    const int dp2 = wave >> 1, hp2 = wave & 1;  // brick planes 2 dp2 + dd, rows 2 hp2 + hh
    f32x16_t acc[2][BH];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < BH; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[a][b][j] = bz;  // the bias enters as the accumulators' start

    // (kd, kw) steps, software-pipelined: the fragment reads of step s + 1 go
    // into the other register set before the MFMAs of step s are issued
    bf16x8_t bfr[2][KE];
    bf16x8_t afr[2][2][BH + KE - 1];
    auto load_step = [&](int st, bf16x8_t(&b)[KE], bf16x8_t(&a)[2][BH + KE - 1]) {
      const int kd = st / KE, kw = st % KE;
#pragma unroll
      for (int kh = 0; kh < KE; ++kh)
        b[kh] = __builtin_bit_cast(bf16x8_t, wp[(((kd * KE + kh) * KE + kw) * 2 + half) * 32 + col]);
#pragma unroll
      for (int dd = 0; dd < 2; ++dd)
#pragma unroll
        for (int hi = 0; hi < BH + KE - 1; ++hi)
          a[dd][hi] = __builtin_bit_cast(
              bf16x8_t, halo[(((2 * dp2 + dd + kd) * G::HH + 2 * hp2 + hi) * 2 + half) * G::HW + kw + col]);
    };
    auto mfma_step = [&](const bf16x8_t(&b)[KE], const bf16x8_t(&a)[2][BH + KE - 1]) {
#pragma unroll
      for (int dd = 0; dd < 2; ++dd)
#pragma unroll
        for (int hi = 0; hi < BH + KE - 1; ++hi)
#pragma unroll
          for (int kh = 0; kh < KE; ++kh) {
            const int hrow = hi - kh;
            if (hrow >= 0 && hrow < BH)
              acc[dd][hrow] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[dd][hi], b[kh], acc[dd][hrow], 0, 0, 0);
          }
    };
    constexpr int NSTEP = KE * KE;
    load_step(0, bfr[0], afr[0]);
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) {
      if (st + 1 < NSTEP) load_step(st + 1, bfr[(st + 1) & 1], afr[(st + 1) & 1]);
      mfma_step(bfr[st & 1], afr[st & 1]);
    }

    // every wave is done with the halo: the next tile's DMA overlaps the epilogue
    __syncthreads();
    {
      const int inext = i + per_xcd_blocks;
      if (inext < per && tile_of(inext) < tiles) issue_halo(tile_of(inext));
    }

    // ---- epilogue ----------------------------------------------------------
    // acc[dd][h][j]: channel col, voxel w = ow0 + 8*(j/4) + 4*half + (j%4)
    const int vd0 = od0 + 2 * dp2, vh0 = oh0 + 2 * hp2;
    if constexpr (EPI == 0) {
#pragma unroll
      for (int dd = 0; dd < 2; ++dd)
#pragma unroll
        for (int hh = 0; hh < BH; ++hh) {
          const int vd = vd0 + dd, vh = vh0 + hh;
          if (vd >= p.od || vh >= p.oh) continue;
          const long long rowv = (((long long)n * p.od + vd) * p.oh + vh) * p.ow;
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int vw = ow0 + 8 * (j >> 2) + 4 * half + (j & 3);
            if (vw < p.ow) out[(rowv + vw) * 32 + col] = f2bf(acc[dd][hh][j]);
          }
        }
    } else {
      // u = acc (started at b); the slope mask word of a voxel (32 channel
      // bits) is half of a wave ballot of one accumulator register.  Every lane
      // stores ballot >> (32 * half) to LDS without a branch (a branch would
      // have to keep the compare alive across it): lanes 0 and 32 into the
      // wave's stage (dword 2 j + half), every other lane into a private junk
      // slot.  After the 16 registers of an output row, 32 lanes write the
      // row's 128 mask bytes at once.  The leaky ReLU is a multiply and a
      // max (or min): a select on the compare would keep one lane mask per
      // register alive until the pooling below.
      unsigned char *mst = reinterpret_cast<unsigned char *>(wp + G::W_VEC) + wave * G::MSTAGE_WAVE;
      const int mslot = (lane & 31) == 0 ? 4 * half : 128 + 4 * lane;
#pragma unroll
      for (int dd = 0; dd < 2; ++dd)
#pragma unroll
        for (int hh = 0; hh < BH; ++hh) {
          const int vd = vd0 + dd, vh = vh0 + hh;
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const float u = acc[dd][hh][j];
            const unsigned long long bal = __ballot(u > 0.f);
            *reinterpret_cast<uint32_t *>(mst + mslot + 8 * j) = (uint32_t)(bal >> (32 * half));
            // one max (min) instruction: fmaxf would first canonicalize u, which
            // is a finite sum of products here
            const float au = alpha * u;
            float y;
            if constexpr (AMAX)
              asm("v_max_f32 %0, %1, %2" : "=v"(y) : "v"(u), "v"(au));
            else
              asm("v_min_f32 %0, %1, %2" : "=v"(y) : "v"(u), "v"(au));
            acc[dd][hh][j] = y;
          }
          if (mask != nullptr) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            // row voxel v = lane: register j = 4 (v / 8) + v % 4 of half (v / 4) % 2
            const int v = lane;
            if (v < 32 && vd < p.od && vh < p.oh && ow0 + v < p.ow) {
              const uint32_t word =
                  *reinterpret_cast<const uint32_t *>(mst + 4 * (2 * (4 * (v >> 3) + (v & 3)) + ((v >> 2) & 1)));
              mask[(((long long)n * p.od + vd) * p.oh + vh) * p.ow + ow0 + v] = word;
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
          }
        }
      if constexpr (EPI == 1) {  // y, no pool
#pragma unroll
        for (int dd = 0; dd < 2; ++dd)
#pragma unroll
          for (int hh = 0; hh < BH; ++hh) {
            const int vd = vd0 + dd, vh = vh0 + hh;
            if (vd >= p.od || vh >= p.oh) continue;
            const long long rowv = (((long long)n * p.od + vd) * p.oh + vh) * p.ow;
#pragma unroll
            for (int j = 0; j < 16; ++j) {
              const int vw = ow0 + 8 * (j >> 2) + 4 * half + (j & 3);
              if (vw < p.ow) out[(rowv + vw) * 32 + col] = f2bf(acc[dd][hh][j]);
            }
          }
      } else {  // 2^3 average pool: window = (dd 0..1) x (h pair) x (w pair), all in this lane
        const int pd_ = vd0 >> 1;
#pragma unroll
        for (int hp = 0; hp < BH / 2; ++hp) {
          const int ph_ = (vh0 >> 1) + hp;
          if (pd_ >= p.pod || ph_ >= p.poh) continue;
          const long long prow = (((long long)n * p.pod + pd_) * p.poh + ph_) * p.pow_;
#pragma unroll
          for (int j = 0; j < 16; j += 2) {
            float s = 0.f;
#pragma unroll
            for (int dd = 0; dd < 2; ++dd)
#pragma unroll
              for (int hh = 0; hh < 2; ++hh) s += acc[dd][2 * hp + hh][j] + acc[dd][2 * hp + hh][j + 1];
            const int pw_ = (ow0 >> 1) + 4 * (j >> 2) + 2 * half + ((j & 3) >> 1);
            if (pw_ < p.pow_) out[(prow + pw_) * 32 + col] = f2bf(s * 0.125f);
          }
        }
      }
    }
  }
}

template <int KE, int EPI, bool AMAX>
hipError_t launch_t(const C16Params &p, const void *x, const void *w, const float *bias, float alpha, void *out,
                    uint32_t *mask, hipStream_t st) {
  using G = C16<KE>;
  const long long tiles = (long long)p.n * ((p.od + TD - 1) / TD) * ((p.oh + TH - 1) / TH) * ((p.ow + TW - 1) / TW);
  int blocks = (int)std::min<long long>(tiles, kNumCUs);
  blocks = std::max(8, (blocks + 7) / 8 * 8);
  hipLaunchKernelGGL((conv_c16_fwd_kernel<KE, EPI, AMAX>), dim3(blocks), dim3(64 * NWAVE), 0, st,
                     (const uint16_t *)x, (const uint16_t *)w, bias, alpha, (uint16_t *)out, mask, p);
  return hipGetLastError();
}

}  // namespace

bool c16_fwd_supported(const ConvShape &s) {
  return s.dtype == DT_BF16 && s.ci == 16 && s.co == 32 && s.sd == 1 && s.sh == 1 && s.sw == 1 &&
         s.kd == s.kh && s.kd == s.kw && s.kd >= 2 && s.kd <= 4 &&
         (long long)s.n * s.d * s.h * s.w * s.ci * 2 < (1LL << 31);  // 32-bit buffer offsets
}

hipError_t launch_conv_fwd_c16(const ConvShape &s, const void *x, const void *w, const float *bias, float alpha,
                               void *out, uint32_t *mask, int epi, hipStream_t st) {
  C16Params p{};
  p.n = s.n; p.d = s.d; p.h = s.h; p.w = s.w;
  p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.od = s.od; p.oh = s.oh; p.ow = s.ow;
  p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
  p.x_bytes = (int)((long long)s.n * s.d * s.h * s.w * s.ci * 2);
#define CF_C16_CASE(KEV)                                                                      \
  if (s.kd == KEV) {                                                                          \
    if (epi == 0) return launch_t<KEV, 0, true>(p, x, w, bias, alpha, out, mask, st);         \
    if (alpha <= 1.f)                                                                         \
      return epi == 1 ? launch_t<KEV, 1, true>(p, x, w, bias, alpha, out, mask, st)           \
                      : launch_t<KEV, 2, true>(p, x, w, bias, alpha, out, mask, st);          \
    return epi == 1 ? launch_t<KEV, 1, false>(p, x, w, bias, alpha, out, mask, st)            \
                    : launch_t<KEV, 2, false>(p, x, w, bias, alpha, out, mask, st);           \
  }
  CF_C16_CASE(2) CF_C16_CASE(3) CF_C16_CASE(4)
#undef CF_C16_CASE
  return hipErrorInvalidValue;
}

}  // namespace cf
