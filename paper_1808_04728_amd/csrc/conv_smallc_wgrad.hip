// conv_smallc_wgrad.hip -- fused backward-weights of the first layer (gfx950).
//
// Backward weights (Section III-C) of a few-input-channel layer that was run
// with the fused forward epilogue (bias + leaky ReLU + 2^3 pool + slope mask):
// the full-resolution gradient dz is never stored.  Each workgroup rebuilds
// it tile by tile in LDS from the pooled-output gradient dp and the mask,
//     dz[v,c] = dp[pool(v),c] / 8 * (mask(v,c) ? 1 : alpha)   (0 off the pool grid)
// and contracts it with the input halo on MFMA:
//     dW[(t,ci),co] = sum_v x~[v + t, ci] * dz[v, co]          (K = voxels)
// The bias gradient db[c] = sum_v dz[v,c] is accumulated in the same pass.
//
// MFMA operands need the voxel axis contiguous per lane, so the tile is
// stored transposed: dz as [co][voxel] (each thread builds an 8-voxel x
// 8-channel block in registers and writes eight 16-byte rows), and the input
// halo once per kw shift as [kw][ci][d][h][32 w] so that every tap's 8-voxel
// run is a 16-byte aligned LDS read.  Each workgroup folds several 4x8x32
// output tiles into its accumulators and writes one fp32 partial; a second
// kernel sums the partials in workgroup order (deterministic).

#include "cf_common.h"
#include "cf_kernels.h"

#include <type_traits>

namespace cf {
namespace {

constexpr int TD = 4, TH = 8, TW = 32;
constexpr int TVOX = TD * TH * TW;  // 1024 voxels, 32 w-rows of 32
constexpr int KMAXE = 3;  // kernel extent limit of the fused path (the first layer is 3^3)

template <int DT, int CIN, int NF>
struct WgLds {
  using T = typename Store<DT>::T;
  static constexpr int COUT = 16 * NF;
  static constexpr int XS = KMAXE * CIN * (TD + KMAXE - 1) * (TH + KMAXE - 1) * TW;  // shifted halo copies
  static constexpr int DZ = COUT * TVOX;
};

template <int DT, int CIN, int NF, int MF, int KE>
__global__ __launch_bounds__(256) void smallc_wgrad_fused_kernel(
    const typename Store<DT>::T *__restrict__ x, const typename Store<DT>::T *__restrict__ dp,
    const uint16_t *__restrict__ mask16, float alpha, float *__restrict__ part_w,
    float *__restrict__ part_b, SmallcParams p) {
  using T = typename Store<DT>::T;
  using L = WgLds<DT, CIN, NF>;
  constexpr int COUT = L::COUT;
  constexpr bool BF = DT == DT_BF16;
  // the cross-wave reduction buffer reuses the halo / dz space after the last tile
  constexpr int RED = 4 * MF * 16 * COUT > 2048 ? 4 * MF * 16 * COUT : 2048;
  constexpr int STAGE_BYTES = (L::XS + L::DZ) * (int)sizeof(T);
  constexpr int SMEM = STAGE_BYTES > RED * 4 ? STAGE_BYTES : RED * 4;
  __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];
  T *xs = reinterpret_cast<T *>(smem);
  T *dzs = xs + L::XS;
  float *red = reinterpret_cast<float *>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  // cubic kernel of extent KE: halo and tap indices divide by constants
  constexpr int HD = TD + KE - 1, HH = TH + KE - 1, HWD = TW + KE - 1;
  constexpr int M = KE * KE * KE * CIN;
  const int tiles_w = (p.ow + TW - 1) / TW, tiles_h = (p.oh + TH - 1) / TH, tiles_d = (p.od + TD - 1) / TD;
  const int tiles_per_n = tiles_w * tiles_h * tiles_d;
  const long long total_tiles = (long long)p.n * tiles_per_n;

  // per-lane A offsets (rows = (tap, ci), padded rows read row 0's data)
  int aoff[MF];
#pragma unroll
  for (int mf = 0; mf < MF; ++mf) {
    int row = mf * 16 + r;
    if (row >= M) row = 0;
    int tap = row / CIN, ci = row % CIN;
    int kd_ = tap / (KE * KE), kh_ = (tap / KE) % KE, kw_ = tap % KE;
    aoff[mf] = (((kw_ * CIN + ci) * HD + kd_) * HH + kh_) * TW;
  }

  f32x4_t acc[MF][NF];
#pragma unroll
  for (int i = 0; i < MF; ++i)
#pragma unroll
    for (int f = 0; f < NF; ++f) acc[i][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // bias-gradient partials of this thread's dz block: 8 channels
  float dbs[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) dbs[j] = 0.f;

  // dz staging item of this thread: 8 consecutive voxels of one w-row x 8 channels
  constexpr int CG = COUT / 8;
  static_assert(TVOX / 8 * CG >= 256 && (TVOX / 8 * CG) % 256 == 0, "dz items");
  constexpr int NITEM = TVOX / 8 * CG / 256;

  for (int it = 0; it < p.tiles_per_block; ++it) {
    const long long gt = (long long)blockIdx.x * p.tiles_per_block + it;
    if (gt >= total_tiles) break;
    int t = (int)(gt % tiles_per_n);
    const int n = (int)(gt / tiles_per_n);
    const int tw = t % tiles_w; t /= tiles_w;
    const int th = t % tiles_h;
    const int td = t / tiles_h;
    const int od0 = td * TD, oh0 = th * TH, ow0 = tw * TW;

    // ---- stage the input halo, once per kw shift --------------------------
    // (all of the tile's global loads -- halo here, dz sources below -- are issued
    // before the first LDS store, so their latencies overlap)
    constexpr int helems = HD * HH * HWD * CIN;
    constexpr int NL = (helems + 255) / 256;
    T xv[NL];
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int e = tid + 256 * k;
      const int ci = e % CIN;
      const int v = e / CIN;
      const int a = v / (HH * HWD), b = (v / HWD) % HH, c = v % HWD;
      const int id = od0 - p.pd + a, ih = oh0 - p.ph + b, iw = ow0 - p.pw + c;
      T val = from_f32<DT>(0.f);
      if (e < helems && (unsigned)id < (unsigned)p.d && (unsigned)ih < (unsigned)p.h && (unsigned)iw < (unsigned)p.w)
        val = x[((((long long)n * p.d + id) * p.h + ih) * p.w + iw) * CIN + ci];
      xv[k] = val;
    }
    // ---- rebuild dz = dp/8 * slope(mask) for the tile, transposed ----------
#pragma unroll
    for (int i = 0; i < NITEM; ++i) {
      const int item = tid + 256 * i;
      const int cg = item % CG;
      const int vb = item / CG;           // 8-voxel block: row = vb / 4, w8 = vb % 4
      const int row = vb >> 2, w8 = vb & 3;
      const int ld = row / TH, lh = row % TH;
      const int vd = od0 + ld, vh = oh0 + lh, vw0 = ow0 + 8 * w8;
      float dz[8][8];  // [voxel][channel]
#pragma unroll
      for (int a = 0; a < 8; ++a)
#pragma unroll
        for (int j = 0; j < 8; ++j) dz[a][j] = 0.f;
      const int pd_ = vd >> 1, ph_ = vh >> 1;
      if (vd < p.od && vh < p.oh && pd_ < p.pod && ph_ < p.poh) {
        const long long vrow = (((long long)n * p.od + vd) * p.oh + vh) * p.ow;
        const long long prow = (((long long)n * p.pod + pd_) * p.poh + ph_) * p.pow_;
#pragma unroll
        for (int pp = 0; pp < 4; ++pp) {  // 4 pooled voxels cover the 8 voxels
          const int pw_ = (vw0 >> 1) + pp;
          if (pw_ >= p.pow_) continue;
          float g[8];
          if constexpr (BF) {
            Vec16<DT_BF16> v;
            v.u = *reinterpret_cast<const uint4 *>(dp + (prow + pw_) * COUT + 8 * cg);
#pragma unroll
            for (int j = 0; j < 8; ++j) g[j] = bf2f(v.e[j]) * 0.125f;
          } else {
            const float4 *src = reinterpret_cast<const float4 *>(dp + (prow + pw_) * COUT + 8 * cg);
            float4 v0 = src[0], v1 = src[1];
            g[0] = v0.x * 0.125f; g[1] = v0.y * 0.125f; g[2] = v0.z * 0.125f; g[3] = v0.w * 0.125f;
            g[4] = v1.x * 0.125f; g[5] = v1.y * 0.125f; g[6] = v1.z * 0.125f; g[7] = v1.w * 0.125f;
          }
#pragma unroll
          for (int hlf = 0; hlf < 2; ++hlf) {
            const int a = 2 * pp + hlf;
            const int vw = vw0 + a;
            const uint32_t bits = (uint32_t)(mask16[(vrow + vw) * NF + (8 * cg) / 16] >> ((8 * cg) % 16));
#pragma unroll
            for (int j = 0; j < 8; ++j) dz[a][j] = g[j] * (((bits >> j) & 1u) ? 1.f : alpha);
          }
        }
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        Vec16<DT> o[BF ? 1 : 2];
#pragma unroll
        for (int a = 0; a < 8; ++a) {
          dbs[j] += dz[a][j];
          if constexpr (BF) o[0].e[a] = f2bf(dz[a][j]);
          else o[a / 4].e[a % 4] = dz[a][j];
        }
        T *dst = dzs + (8 * cg + j) * TVOX + row * TW + 8 * w8;
        if constexpr (BF) {
          *reinterpret_cast<uint4 *>(dst) = o[0].u;
        } else {
          reinterpret_cast<uint4 *>(dst)[0] = o[0].u;
          reinterpret_cast<uint4 *>(dst)[1] = o[1].u;
        }
      }
    }
    // the halo, once per kw shift (xs[s][ci][a][b][w] = halo(a, b, w + s, ci))
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int e = tid + 256 * k;
      if (e >= helems) continue;
      const int ci = e % CIN;
      const int v = e / CIN;
      const int a = v / (HH * HWD), b = (v / HWD) % HH, c = v % HWD;
#pragma unroll
      for (int s = 0; s < KE; ++s) {
        const int wl = c - s;
        if (wl >= 0 && wl < TW) xs[(((s * CIN + ci) * HD + a) * HH + b) * TW + wl] = xv[k];
      }
    }
    __syncthreads();

    // ---- MFMA: each wave takes 8 of the tile's 32 w-rows ------------------
    for (int row = wave; row < TD * TH; row += 4) {
      const int ld = row / TH, lh = row % TH;
      const int xrow = (ld * HH + lh) * TW;
      if constexpr (BF) {
        bf16x8_t b[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f)
          b[f] = *reinterpret_cast<const bf16x8_t *>(dzs + (16 * f + r) * TVOX + row * TW + 8 * q);
#pragma unroll
        for (int mf = 0; mf < MF; ++mf) {
          bf16x8_t a = *reinterpret_cast<const bf16x8_t *>(xs + aoff[mf] + xrow + 8 * q);
#pragma unroll
          for (int f = 0; f < NF; ++f)
            acc[mf][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[f], acc[mf][f], 0, 0, 0);
        }
      } else {
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          float b[NF];
#pragma unroll
          for (int f = 0; f < NF; ++f) b[f] = dzs[(16 * f + r) * TVOX + row * TW + 4 * ks + q];
#pragma unroll
          for (int mf = 0; mf < MF; ++mf) {
            float a = xs[aoff[mf] + xrow + 4 * ks + q];
#pragma unroll
            for (int f = 0; f < NF; ++f)
              acc[mf][f] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b[f], acc[mf][f], 0, 0, 0);
          }
        }
      }
    }
    __syncthreads();
  }

  // ---- combine the four waves and write this workgroup's partials ---------
  __syncthreads();
  // acc[mf][f][j] = dW[row = mf*16 + 4q + j][co = 16f + r]
#pragma unroll
  for (int mf = 0; mf < MF; ++mf)
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        red[((wave * MF + mf) * 16 + 4 * q + j) * COUT + 16 * f + r] = acc[mf][f][j];
  __syncthreads();
  const int wsz = MF * 16 * COUT;
  for (int i = tid; i < M * COUT; i += 256) {
    float s = red[i] + red[wsz + i] + red[2 * wsz + i] + red[3 * wsz + i];
    part_w[(long long)blockIdx.x * M * COUT + i] = s;
  }
  __syncthreads();
  // bias partials: thread item cg = tid % CG holds channels 8cg..8cg+7
  {
    const int cg = tid % CG;
    const int slot = tid / CG;  // 256 / CG slots
#pragma unroll
    for (int j = 0; j < 8; ++j) red[slot * COUT + 8 * cg + j] = dbs[j];
  }
  __syncthreads();
  if (tid < COUT) {
    float s = 0.f;
    for (int k = 0; k < 256 / CG; ++k) s += red[k * COUT + tid];
    part_b[(long long)blockIdx.x * COUT + tid] = s;
  }
}

// ---------------------------------------------------------------------------
// One input channel, bf16: dz built straight in MFMA-operand registers.
//
// With s = alpha + (1 - alpha) * mask the weight gradient splits into
//     dW = alpha/8 * sum_v x~[v+t] dp[pool(v)] + (1-alpha)/8 * sum_v x~[v+t] (dp[pool(v)] & mask(v))
// (dp/8 * s(v) = dz exactly), so neither term needs per-element arithmetic
// beyond a bit mask: the B operand of the first term is the pooled gradient
// with every value twice (one per voxel of the w-pair), that of the second the
// same with the masked-off halves cleared.  A transposing LDS read
// (ds_read_b64_tr_b16) hands every lane the four pooled values of its channel
// for its eight voxels; the lane's 16 mask bytes come straight from global
// memory.  An extra A row of ones makes the bias gradient db = sum_v dz a row
// of the same MFMA accumulators.  The input halo is staged once per kw shift
// (16-byte rows of 8 voxels, built from aligned 16-byte loads with byte
// alignment shifts), so every A fragment is one 16-byte LDS read.
// ---------------------------------------------------------------------------

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));  // a plain 16-byte vector

// Input halo of one tile for the single-channel kernels: item (row a, b;
// 16-byte output vector i) needs the vectors i .. i+2 of the aligned window
// [ow0 - 8, ow0 + 40) of its input row (zeros outside the input).
template <int KE>
__device__ __forceinline__ void l1_load_x(const uint16_t *__restrict__ x, const SmallcParams &p, int tid, int n,
                                          int od0, int oh0, int ow0, u32x4_t (&xv)[3]) {
  constexpr int HD = TD + KE - 1, HH = TH + KE - 1;
  const int xa = tid / (HH * 4), xb = (tid / 4) % HH, xi = tid & 3;
#pragma unroll
  for (int j = 0; j < 3; ++j) xv[j] = u32x4_t{0u, 0u, 0u, 0u};
  if (tid < HD * HH * 4) {
    const int id = od0 - p.pd + xa, ih = oh0 - p.ph + xb;
    if ((unsigned)id < (unsigned)p.d && (unsigned)ih < (unsigned)p.h) {
      // 24-bit products: n d h, n od oh and the element counts are below 2^24 / 2^31
      const int rowoff = (int)__umul24(__umul24(n * p.d + id, p.h) + ih, p.w);
#pragma unroll
      for (int j = 0; j < 3; ++j) {
        const int iw = ow0 - 8 + 8 * (xi + j);
        if (iw >= 0 && iw < p.w) xv[j] = *reinterpret_cast<const u32x4_t *>(x + rowoff + iw);
      }
    }
  }
}

// ... and its KE shifted copies in LDS: copy kw, element i of a row = window
// element 8 - PW + kw + i (16-byte rows of 8 voxels, XP slots per row).
template <int KE, int PW, int XP>
__device__ __forceinline__ void l1_store_x(uint4 *xs, int tid, const u32x4_t (&xv)[3]) {
  constexpr int HD = TD + KE - 1, HH = TH + KE - 1;
  const int xa = tid / (HH * 4), xb = (tid / 4) % HH, xi = tid & 3;
  if (tid < HD * HH * 4) {
    const uint32_t dw[12] = {xv[0][0], xv[0][1], xv[0][2], xv[0][3], xv[1][0], xv[1][1],
                             xv[1][2], xv[1][3], xv[2][0], xv[2][1], xv[2][2], xv[2][3]};
#pragma unroll
    for (int kw = 0; kw < KE; ++kw) {
      const int s0 = 8 - PW + kw;
      uint32_t o[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int L = (s0 >> 1) + k;
        o[k] = (s0 & 1) ? __builtin_amdgcn_alignbyte(dw[L + 1], dw[L], 2) : dw[L];
      }
      xs[((kw * HD + xa) * HH + xb) * XP + xi] = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
}

template <int KE, int PW>
__global__ __launch_bounds__(256) void l1_wgrad_kernel(const uint16_t *__restrict__ x,
                                                       const uint16_t *__restrict__ dp,
                                                       const uint16_t *__restrict__ mask16, float alpha,
                                                       float *__restrict__ part_w, float *__restrict__ part_b,
                                                       SmallcParams p) {
  constexpr int HD = TD + KE - 1, HH = TH + KE - 1;
  constexpr int M = KE * KE * KE;  // weight-gradient rows; row M carries the bias gradient
  constexpr int MF = 2;
  static_assert(M + 1 <= 16 * MF, "rows");
  constexpr int PLANE = HD * HH;                 // 64-byte rows per shifted copy
  constexpr int XROWS = (KE + 2) * PLANE;        // KE copies, a plane of ones, a plane of zeros
  constexpr int NXI = PLANE * 4;                 // staging items: (row, 16-byte output vector)
  static_assert(NXI <= 256, "one staging item per thread");
  constexpr int XP = 5;  // 16-byte slots per staged row: 4 used, 1 of padding against bank conflicts
  __shared__ __attribute__((aligned(16))) uint4 xs[XROWS * XP];
  __shared__ __attribute__((aligned(16))) uint4 dps[2 * 4 * 16 * 2];  // pooled [pd][ph][pw][16 ch]
  __shared__ __attribute__((aligned(16))) uint4 mks[TD * TH * 4];      // mask [w-row][8-voxel group]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, q = lane >> 4;
  const int tiles_w = (p.ow + TW - 1) / TW, tiles_h = (p.oh + TH - 1) / TH, tiles_d = (p.od + TD - 1) / TD;
  const int tiles_per_n = tiles_w * tiles_h * tiles_d;
  const int total_tiles = p.n * tiles_per_n;  // the launcher keeps every index below 2^24

  // the constant planes: ones (A row M) and zeros (A rows beyond M)
  for (int e = tid; e < 2 * PLANE * XP; e += 256)
    xs[KE * PLANE * XP + e] = e < PLANE * XP ? make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u)
                                             : make_uint4(0, 0, 0, 0);

  // per-lane A plane offsets (64-byte rows): tap (kd, kh, kw) -> copy kw, plane row (kd, kh)
  int arow[MF];
#pragma unroll
  for (int mf = 0; mf < MF; ++mf) {
    const int t = 16 * mf + r;
    if (t < M) {
      const int kd = t / (KE * KE), kh = (t / KE) % KE, kw = t % KE;
      arow[mf] = (kw * HD + kd) * HH + kh;
    } else {
      arow[mf] = (t == M ? KE : KE + 1) * PLANE;
    }
  }
  // per-lane part of the transposing dp read: pooled voxel 4q + r/4, channels 4 (r%4) ..
  const int dpoff = (4 * q + (r >> 2)) * 32 + 8 * (r & 3);

  f32x4_t acc_u[MF], acc_m[MF];
#pragma unroll
  for (int mf = 0; mf < MF; ++mf) acc_u[mf] = acc_m[mf] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Tile pipeline: the global loads of tile it+1 (into registers) are issued
  // right after tile it's data reached LDS, so their latency overlaps tile
  // it's MFMAs; LDS is single-buffered (written only between two barriers).
  u32x4_t xv[3], dv, mv;
  int cur_n = 0, cur_od0 = 0, cur_oh0 = 0, cur_ow0 = 0;
  auto tile_origin = [&](int it, int &n, int &od0, int &oh0, int &ow0) -> bool {
    const int gt = (int)blockIdx.x * p.tiles_per_block + it;
    if (it >= p.tiles_per_block || gt >= total_tiles) return false;
    int t = gt % tiles_per_n;
    n = gt / tiles_per_n;
    const int tw = t % tiles_w; t /= tiles_w;
    const int th = t % tiles_h;
    const int td = t / tiles_h;
    od0 = td * TD; oh0 = th * TH; ow0 = tw * TW;
    return true;
  };
  auto load_tile = [&](int n, int od0, int oh0, int ow0) {
    l1_load_x<KE>(x, p, tid, n, od0, oh0, ow0, xv);
    // pooled gradient: pooled voxel (pd0 + tid>>7, ph0 + (tid>>5)&3, pw0 + (tid>>1)&15), 8 channels
    dv = u32x4_t{0u, 0u, 0u, 0u};
    {
      const int pd_ = (od0 >> 1) + (tid >> 7), ph_ = (oh0 >> 1) + ((tid >> 5) & 3), pw_ = (ow0 >> 1) + ((tid >> 1) & 15);
      if (pd_ < p.pod && ph_ < p.poh && pw_ < p.pow_)
        dv = *reinterpret_cast<const u32x4_t *>(
            dp + ((int)__umul24(__umul24(n * p.pod + pd_, p.poh) + ph_, p.pow_) + pw_) * 16 + 8 * (tid & 1));
    }
    // slope mask: thread tid < 128 loads 8 voxels (16 bytes) of w-row tid / 4
    mv = u32x4_t{0u, 0u, 0u, 0u};
    if (tid < 128) {
      const int row = tid >> 2;
      const int vd = od0 + row / TH, vh = oh0 + row % TH, vw = ow0 + 8 * (tid & 3);
      if (vd < p.od && vh < p.oh && vw < p.ow) {
        const uint16_t *mrow = mask16 + (int)__umul24(__umul24(n * p.od + vd, p.oh) + vh, p.ow);
        if (vw + 8 <= p.ow) {
          mv = *reinterpret_cast<const u32x4_t *>(mrow + vw);
        } else {
          // ragged end of a row: the voxels past it pool into no pooled voxel
          // (their B values are zero), so their bits may be anything; read only
          // the row's own voxels (the last row ends at the end of the buffer)
          uint32_t h[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) h[u] = vw + u < p.ow ? mrow[vw + u] : 0u;
          mv = u32x4_t{h[0] | h[1] << 16, h[2] | h[3] << 16, h[4] | h[5] << 16, h[6] | h[7] << 16};
        }
      }
    }
  };

  bool have = tile_origin(0, cur_n, cur_od0, cur_oh0, cur_ow0);
  if (have) load_tile(cur_n, cur_od0, cur_oh0, cur_ow0);
  for (int it = 0; have; ++it) {
    // ---- LDS: shifted input copies, the pooled-gradient tile, the mask tile
    l1_store_x<KE, PW, XP>(xs, tid, xv);
    dps[tid] = make_uint4(dv[0], dv[1], dv[2], dv[3]);
    if (tid < 128) mks[tid] = make_uint4(mv[0], mv[1], mv[2], mv[3]);
    __syncthreads();
    int nn = 0, nd0 = 0, nh0 = 0, nw0 = 0;
    have = tile_origin(it + 1, nn, nd0, nh0, nw0);
    if (have) load_tile(nn, nd0, nh0, nw0);

    // ---- MFMA over this wave's eight w-rows of 32 voxels: the four w-rows
    // (2a + i, 2b + j) of pooled rows (a, b) = wave and wave + 4, so that the
    // pooled-gradient operand of a pooled row is formed once for its four rows
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      const int prow = wave + 4 * pp;  // pooled row (a, b) = (prow / 4, prow % 4)
      const unsigned char *dpb = reinterpret_cast<const unsigned char *>(dps) + prow * 512;
      const v4i16_t g = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(dpb + dpoff));
      const uint32_t p0 = (uint32_t)(uint16_t)g[0] | ((uint32_t)(uint16_t)g[1] << 16);
      const uint32_t p1 = (uint32_t)(uint16_t)g[2] | ((uint32_t)(uint16_t)g[3] << 16);
      uint32_t bu[4];
      bu[0] = __builtin_amdgcn_perm(p0, p0, 0x01000100u);
      bu[1] = __builtin_amdgcn_perm(p0, p0, 0x03020302u);
      bu[2] = __builtin_amdgcn_perm(p1, p1, 0x01000100u);
      bu[3] = __builtin_amdgcn_perm(p1, p1, 0x03020302u);
      const bf16x8_t Bu = __builtin_bit_cast(bf16x8_t, make_uint4(bu[0], bu[1], bu[2], bu[3]));
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int ld = 2 * (prow >> 2) + (k >> 1), lh = 2 * (prow & 3) + (k & 1);
        const int row = ld * TH + lh;
        uint32_t bm[4];
        const uint4 mq = mks[row * 4 + q];
        const uint32_t mk[4] = {mq.x, mq.y, mq.z, mq.w};
        // mask dword d holds channel bits of voxels 2d (bits 0..15) and 2d+1 (16..31):
        // move bit r and bit 16+r to the two sign positions, spread each over its half
        typedef short v2i16_t __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const v2i16_t sg = __builtin_bit_cast(v2i16_t, mk[d] << (15 - r)) >> (v2i16_t){15, 15};
          bm[d] = bu[d] & __builtin_bit_cast(uint32_t, sg);
        }
        const bf16x8_t Bm = __builtin_bit_cast(bf16x8_t, make_uint4(bm[0], bm[1], bm[2], bm[3]));
#pragma unroll
        for (int mf = 0; mf < MF; ++mf) {
          const bf16x8_t a = __builtin_bit_cast(bf16x8_t, xs[(arow[mf] + ld * HH + lh) * XP + q]);
          acc_u[mf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, Bu, acc_u[mf], 0, 0, 0);
          acc_m[mf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, Bm, acc_m[mf], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }

  // ---- combine the two terms and the four waves; write the partials ------
  float *red = reinterpret_cast<float *>(xs);  // [wave][32 rows][16 channels]
  const float cu = 0.125f * alpha, cm = 0.125f * (1.f - alpha);
#pragma unroll
  for (int mf = 0; mf < MF; ++mf)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      red[(wave * 32 + 16 * mf + 4 * q + j) * 16 + r] = cu * acc_u[mf][j] + cm * acc_m[mf][j];
  __syncthreads();
  for (int i = tid; i < (M + 1) * 16; i += 256) {
    const float v = red[i] + red[512 + i] + red[1024 + i] + red[1536 + i];
    if (i < M * 16) part_w[(long long)blockIdx.x * M * 16 + i] = v;
    else part_b[(long long)blockIdx.x * 16 + (i - M * 16)] = v;
  }
}

// ---------------------------------------------------------------------------
// The same single-channel bf16 layer without the fused epilogue (the plain
// backward-weights call): dz comes from HBM.  A tile's dz (32 w-rows x 32
// voxels x 16 channels, 32 KiB) is staged in LDS voxel-major, the 16
// channels of a voxel in 32 bytes, with 128 bytes of padding after every 8
// voxels.  Lane (r, q)'s B fragment of a w-row (channel r of voxels
// 8q .. 8q+7) is two transposing reads of four voxels each; with the padding
// the 128-byte windows of the four 16-lane groups alternate between the two
// halves of the 64 banks.  The A side (input halo, shifted copies) and the
// tile pipeline are those of the fused kernel above.
// ---------------------------------------------------------------------------
template <int KE, int PW>
__global__ __launch_bounds__(256) void l1_wgrad_dz_kernel(const uint16_t *__restrict__ x,
                                                          const uint16_t *__restrict__ dz,
                                                          float *__restrict__ part_w, SmallcParams p) {
  constexpr int HD = TD + KE - 1, HH = TH + KE - 1;
  constexpr int M = KE * KE * KE;
  constexpr int MF = 2;
  static_assert(M <= 16 * MF, "rows");
  constexpr int PLANE = HD * HH;
  constexpr int XROWS = (KE + 1) * PLANE;  // KE shifted copies, a plane of zeros (A rows >= M)
  static_assert(PLANE * 4 <= 256, "one staging item per thread");
  constexpr int XP = 5;
  constexpr int ROWB = 32 * 32 + 4 * 128;  // bytes of one staged w-row of dz
  constexpr int NDZ = TD * TH * 32 * 2 / 256;  // 16-byte dz vectors per thread and tile
  __shared__ __attribute__((aligned(16))) uint4 xs[XROWS * XP];
  __shared__ __attribute__((aligned(16))) unsigned char dzs[TD * TH * ROWB];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, q = lane >> 4;
  const int tiles_w = (p.ow + TW - 1) / TW, tiles_h = (p.oh + TH - 1) / TH, tiles_d = (p.od + TD - 1) / TD;
  const int tiles_per_n = tiles_w * tiles_h * tiles_d;
  const int total_tiles = p.n * tiles_per_n;  // the launcher keeps every index below 2^24

  for (int e = tid; e < PLANE * XP; e += 256) xs[KE * PLANE * XP + e] = make_uint4(0, 0, 0, 0);
  int arow[MF];
#pragma unroll
  for (int mf = 0; mf < MF; ++mf) {
    const int t = 16 * mf + r;
    if (t < M) {
      const int kd = t / (KE * KE), kh = (t / KE) % KE, kw = t % KE;
      arow[mf] = (kw * HD + kd) * HH + kh;
    } else {
      arow[mf] = KE * PLANE;
    }
  }
  // B reads: voxel 8q + r/4 (its pad is 128 q bytes), channels 4 (r%4) .. 4 (r%4) + 3
  const int boff = (8 * q + (r >> 2)) * 32 + 128 * q + 8 * (r & 3);
  // dz staging: vector j of this thread is w-row 4j + tid/64, voxel (tid%64)/2, channel half tid%2
  const int sw = (tid & 63) >> 1, sc = tid & 1;
  const int soff = sw * 32 + (sw >> 3) * 128 + 16 * sc;

  f32x4_t acc[MF];
#pragma unroll
  for (int mf = 0; mf < MF; ++mf) acc[mf] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  u32x4_t xv[3], dv[NDZ];
  auto tile_origin = [&](int it, int &n, int &od0, int &oh0, int &ow0) -> bool {
    const int gt = (int)blockIdx.x * p.tiles_per_block + it;
    if (it >= p.tiles_per_block || gt >= total_tiles) return false;
    int t = gt % tiles_per_n;
    n = gt / tiles_per_n;
    const int tw = t % tiles_w; t /= tiles_w;
    const int th = t % tiles_h;
    const int td = t / tiles_h;
    od0 = td * TD; oh0 = th * TH; ow0 = tw * TW;
    return true;
  };
  auto load_tile = [&](int n, int od0, int oh0, int ow0) {
    l1_load_x<KE>(x, p, tid, n, od0, oh0, ow0, xv);
    const int vw = ow0 + sw;
#pragma unroll
    for (int j = 0; j < NDZ; ++j) {
      const int row = 4 * j + (tid >> 6);
      const int vd = od0 + row / TH, vh = oh0 + row % TH;
      dv[j] = u32x4_t{0u, 0u, 0u, 0u};
      if (vd < p.od && vh < p.oh && vw < p.ow)
        dv[j] = *reinterpret_cast<const u32x4_t *>(
            dz + ((int)__umul24(__umul24(n * p.od + vd, p.oh) + vh, p.ow) + vw) * 16 + 8 * sc);
    }
  };

  int n0 = 0, d0 = 0, h0 = 0, w0 = 0;
  bool have = tile_origin(0, n0, d0, h0, w0);
  if (have) load_tile(n0, d0, h0, w0);
  for (int it = 0; have; ++it) {
    l1_store_x<KE, PW, XP>(xs, tid, xv);
#pragma unroll
    for (int j = 0; j < NDZ; ++j)
      *reinterpret_cast<uint4 *>(dzs + (4 * j + (tid >> 6)) * ROWB + soff) =
          make_uint4(dv[j][0], dv[j][1], dv[j][2], dv[j][3]);
    __syncthreads();
    int nn = 0, nd0 = 0, nh0 = 0, nw0 = 0;
    have = tile_origin(it + 1, nn, nd0, nh0, nw0);
    if (have) load_tile(nn, nd0, nh0, nw0);

#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int row = wave + 4 * k;
      const int ld = row / TH, lh = row % TH;
      const unsigned char *rb = dzs + row * ROWB + boff;
      const v4i16_t g0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)rb);
      const v4i16_t g1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(rb + 128));
      const bf16x8_t b = __builtin_bit_cast(
          bf16x8_t, make_uint4((uint32_t)(uint16_t)g0[0] | ((uint32_t)(uint16_t)g0[1] << 16),
                               (uint32_t)(uint16_t)g0[2] | ((uint32_t)(uint16_t)g0[3] << 16),
                               (uint32_t)(uint16_t)g1[0] | ((uint32_t)(uint16_t)g1[1] << 16),
                               (uint32_t)(uint16_t)g1[2] | ((uint32_t)(uint16_t)g1[3] << 16)));
#pragma unroll
      for (int mf = 0; mf < MF; ++mf) {
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, xs[(arow[mf] + ld * HH + lh) * XP + q]);
        acc[mf] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[mf], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // ---- combine the four waves; write the partials -------------------------
  float *red = reinterpret_cast<float *>(dzs);  // [wave][32 rows][16 channels]
#pragma unroll
  for (int mf = 0; mf < MF; ++mf)
#pragma unroll
    for (int j = 0; j < 4; ++j) red[(wave * 32 + 16 * mf + 4 * q + j) * 16 + r] = acc[mf][j];
  __syncthreads();
  for (int i = tid; i < M * 16; i += 256)
    part_w[(long long)blockIdx.x * M * 16 + i] = red[i] + red[512 + i] + red[1024 + i] + red[1536 + i];
}

struct WPlan {
  int tpb;
  int blocks;
};

WPlan plan(const ConvShape &s) {
  const long long tiles = (long long)s.n * ((s.od + TD - 1) / TD) * ((s.oh + TH - 1) / TH) * ((s.ow + TW - 1) / TW);
  WPlan w;
  w.tpb = (int)std::max<long long>(1, (tiles + 2047) / 2048);
  w.blocks = (int)((tiles + w.tpb - 1) / w.tpb);
  return w;
}

template <int DT, int CIN, int NF, int MF, int KE>
hipError_t launch_t(const ConvShape &s, const SmallcParams &p, const void *x, const void *dp,
                    const uint16_t *mask, float alpha, float *dw, float *db, void *ws, int blocks,
                    hipStream_t st) {
  using T = typename Store<DT>::T;
  const int M = s.kd * s.kh * s.kw * s.ci;
  float *pw = (float *)ws;
  float *pb = pw + (size_t)blocks * M * s.co;
  hipLaunchKernelGGL((smallc_wgrad_fused_kernel<DT, CIN, NF, MF, KE>), dim3(blocks), dim3(256), 0, st,
                     (const T *)x, (const T *)dp, mask, alpha, pw, pb, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_sum_rows(pw, dw, blocks, M * s.co, st);
  if (e != hipSuccess) return e;
  return launch_sum_rows(pb, db, blocks, s.co, st);
}

// the register-built-dz kernel: one input channel, 16 output channels, bf16,
// input rows of whole 16-byte vectors, an even output width (every output
// voxel of a row lies in a pooling window, or the row's last one does not),
// left padding of at most one voxel
// and index arithmetic in 24-bit products: n d h and n od oh below 2^24 (the
// 128^3 stack at batch 8 has 2^17), every element offset below 2^31
bool l1_supported(const ConvShape &s) {
  const long long ndh = (long long)s.n * s.d * s.h, nodoh = (long long)s.n * s.od * s.oh;
  const long long xel = ndh * s.w, mel = nodoh * s.ow * 16;
  return s.dtype == DT_BF16 && s.ci == 1 && s.co == 16 && s.sd == 1 && s.sh == 1 && s.sw == 1 && s.kd == s.kh &&
         s.kd == s.kw && (s.kd == 2 || s.kd == 3) && s.pw <= 1 && (s.kd == 3 || s.pw == 0) && s.w % 8 == 0 &&
         s.ow % 2 == 0 && ndh < (1LL << 24) && nodoh < (1LL << 24) && s.w < (1 << 24) && s.ow < (1 << 24) &&
         xel < (1LL << 31) && mel < (1LL << 31);
}

// the unfused kernel: as l1_supported, with any output width and the dz
// element count (16 per output voxel) below 2^31
bool l1_dz_supported(const ConvShape &s) {
  const long long ndh = (long long)s.n * s.d * s.h, nodoh = (long long)s.n * s.od * s.oh;
  const long long xel = ndh * s.w, zel = nodoh * s.ow * 16;
  return s.dtype == DT_BF16 && s.ci == 1 && s.co == 16 && s.sd == 1 && s.sh == 1 && s.sw == 1 && s.kd == s.kh &&
         s.kd == s.kw && (s.kd == 2 || s.kd == 3) && s.pw <= 1 && (s.kd == 3 || s.pw == 0) && s.w % 8 == 0 &&
         ndh < (1LL << 24) && nodoh < (1LL << 24) && s.w < (1 << 24) && s.ow < (1 << 24) && xel < (1LL << 31) &&
         zel < (1LL << 31);
}

SmallcParams params(const ConvShape &s, const WPlan &w) {
  SmallcParams p{};
  p.n = s.n; p.d = s.d; p.h = s.h; p.w = s.w; p.ci = s.ci; p.co = s.co;
  p.kd = s.kd; p.kh = s.kh; p.kw = s.kw; p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.od = s.od; p.oh = s.oh; p.ow = s.ow;
  p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
  p.tiles_per_block = w.tpb;
  return p;
}

}  // namespace

bool smallc_wgrad_dz_supported(const ConvShape &s) { return l1_dz_supported(s); }

size_t smallc_wgrad_dz_workspace(const ConvShape &s) {
  const WPlan w = plan(s);
  return (size_t)w.blocks * s.kd * s.kh * s.kw * s.co * sizeof(float);
}

hipError_t launch_smallc_wgrad_dz(const ConvShape &s, const void *x, const void *dz, float *dw, void *ws,
                                  hipStream_t st) {
  const WPlan w = plan(s);
  const SmallcParams p = params(s, w);
  float *pw = (float *)ws;
  if (s.kd == 2)
    hipLaunchKernelGGL((l1_wgrad_dz_kernel<2, 0>), dim3(w.blocks), dim3(256), 0, st, (const uint16_t *)x,
                       (const uint16_t *)dz, pw, p);
  else if (s.pw == 0)
    hipLaunchKernelGGL((l1_wgrad_dz_kernel<3, 0>), dim3(w.blocks), dim3(256), 0, st, (const uint16_t *)x,
                       (const uint16_t *)dz, pw, p);
  else
    hipLaunchKernelGGL((l1_wgrad_dz_kernel<3, 1>), dim3(w.blocks), dim3(256), 0, st, (const uint16_t *)x,
                       (const uint16_t *)dz, pw, p);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_sum_rows(pw, dw, w.blocks, s.kd * s.kh * s.kw * s.co, st);
}

bool smallc_wgrad_fused_supported(const ConvShape &s) {
  if (s.sd != 1 || s.sh != 1 || s.sw != 1) return false;
  if (s.kd != s.kh || s.kd != s.kw || s.kd < 2 || s.kd > KMAXE) return false;  // cubic 2^3 or 3^3
  if (s.co != 16) return false;
  if (s.dtype == DT_BF16) return s.ci == 1 || s.ci == 4;
  return s.ci == 1;
}

size_t smallc_wgrad_fused_workspace(const ConvShape &s) {
  if (l1f32_wgrad_supported(s)) return l1f32_wgrad_workspace(s);
  WPlan w = plan(s);
  const int M = s.kd * s.kh * s.kw * s.ci;
  return (size_t)w.blocks * (M + 1) * s.co * sizeof(float);
}

hipError_t launch_smallc_wgrad_fused(const ConvShape &s, const void *x, const void *dp, const uint16_t *mask,
                                     float alpha, float *dw, float *db, void *ws, hipStream_t st) {
  if (l1f32_wgrad_supported(s))
    return launch_l1_wgrad_f32(s, (const float *)x, (const float *)dp, mask, alpha, dw, db, ws, st);
  WPlan w = plan(s);
  const SmallcParams p = params(s, w);
  const int M = s.kd * s.kh * s.kw * s.ci;
  if (l1_supported(s)) {
    float *pw = (float *)ws;
    float *pb = pw + (size_t)w.blocks * M * s.co;
    if (s.kd == 2)
      hipLaunchKernelGGL((l1_wgrad_kernel<2, 0>), dim3(w.blocks), dim3(256), 0, st, (const uint16_t *)x,
                         (const uint16_t *)dp, mask, alpha, pw, pb, p);
    else if (s.pw == 0)
      hipLaunchKernelGGL((l1_wgrad_kernel<3, 0>), dim3(w.blocks), dim3(256), 0, st, (const uint16_t *)x,
                         (const uint16_t *)dp, mask, alpha, pw, pb, p);
    else
      hipLaunchKernelGGL((l1_wgrad_kernel<3, 1>), dim3(w.blocks), dim3(256), 0, st, (const uint16_t *)x,
                         (const uint16_t *)dp, mask, alpha, pw, pb, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_sum_rows(pw, dw, w.blocks, M * s.co, st);
    if (e != hipSuccess) return e;
    return launch_sum_rows(pb, db, w.blocks, s.co, st);
  }
  if (s.kd == 2) {
    if (s.dtype == DT_BF16) {
      if (s.ci == 1) return launch_t<DT_BF16, 1, 1, 1, 2>(s, p, x, dp, mask, alpha, dw, db, ws, w.blocks, st);
      return launch_t<DT_BF16, 4, 1, 2, 2>(s, p, x, dp, mask, alpha, dw, db, ws, w.blocks, st);
    }
    return launch_t<DT_F32, 1, 1, 1, 2>(s, p, x, dp, mask, alpha, dw, db, ws, w.blocks, st);
  }
  if (s.dtype == DT_BF16) {
    if (s.ci == 1) return launch_t<DT_BF16, 1, 1, 2, 3>(s, p, x, dp, mask, alpha, dw, db, ws, w.blocks, st);
    return launch_t<DT_BF16, 4, 1, 7, 3>(s, p, x, dp, mask, alpha, dw, db, ws, w.blocks, st);
  }
  return launch_t<DT_F32, 1, 1, 2, 3>(s, p, x, dp, mask, alpha, dw, db, ws, w.blocks, st);
}

}  // namespace cf
