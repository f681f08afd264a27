// conv_f32.hip -- fp32 implicit-GEMM 3D convolution, forward and
// backward-data, on v_mfma_f32_16x16x4_f32 (the paper's own precision:
// Section V-A and Table I time fp32 convolutions).
//
// Forward (Section III-C, Algorithm 1)
//   z[o, co] = sum_{t, ci} x~[o*s + t - p, ci] W[t, ci, co]
// and backward-data, its adjoint in x,
//   dx[i, ci] = sum_{(o, t): o*s + t - p = i} sum_co dz[o, co] W[t, ci, co],
// split into s^3 parity classes of i (only the taps t = (i + p) mod s + s*u
// reach class i, so every class is a dense stride-one contraction).
//
// Data movement (one design for every fp32 layer with 16k contracted
// channels: the 16 -> 32 layer and the deep layers):
//  * rows (output voxels) x columns (output channels) tiles; a workgroup's
//    WM x WK waves split the rows WM ways and the taps WK ways; the WK partial
//    tiles meet once, in LDS, at the end.  WK > 1 is what keeps the small
//    deep layers (512 rows at batch 1) spread over the machine;
//  * no operand is staged: every lane loads its MFMA fragments straight into
//    registers, PF k-steps ahead of the MFMAs, with 32-bit-offset buffer
//    loads whose range check returns zero for padding voxels;
//  * a k-step is one tap x 16 channels.  Lane l (row l%16, K group g = l/16)
//    loads the 16 bytes of channels 4g..4g+3 of its gathered voxel in one
//    load; register j of that load is the A operand of MFMA j (K slot g <->
//    channel 4g + j), so one load feeds four MFMAs;
//  * backward-data weights W[t][ci][co] are K-contiguous (co fastest): lane l
//    loads W[t][col][4g..4g+3], the matching B registers;
//  * forward weights have the output channel contiguous: lane l loads FN
//    consecutive output channels W[t][4g+j][FN*(l%16) ..] for j = 0..3, and
//    register jj of load j is the B operand of MFMA (j, jj), which
//    accumulates columns co = FN*n + jj: FN interleaved accumulators cover
//    16*FN channels with one FN-wide load per K group;
//  * epilogues: store; bias + leaky ReLU (+ 1-bit slope mask); or, for the
//    pooled layer, bias + leaky ReLU + slope mask + 2^3 average pool, with
//    the workgroup's rows laid out as 2 x 2 x TW bricks so that every pooling
//    window lies inside one tile.
//
// v_mfma_f32_16x16x4_f32 lane layout: A lane l holds row l%16, K l/16; B
// lane l holds column l%16, K l/16; D lane l holds column l%16, rows
// 4*(l/16)..+3 in its four registers.

#include "cf_common.h"
#include "cf_kernels.h"
#include "conv_f32_wgrad_kernel.h"
#include "fastdiv.h"

#include <algorithm>
#include <cstdlib>
#include <type_traits>

namespace cf {
namespace {

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

constexpr int F_MAX_CLS = 8;
constexpr int F_MAX_TAPS = 64;

struct FClass {
  int m;                 // row tiles' unit count: rows (linear layout) or bricks (pooled layout)
  int slot0, per;        // XCD-major grid: tiles split into 8 contiguous runs of `per`
  int ntap, tap0;        // taps tap0 .. tap0 + ntap - 1 of the tap table
  FastDiv fw, fh, fd;    // linear: row = ((n*Jd + jd)*Jh + jh)*Jw + jw; brick: same over brick indices
  int bq_d, bq_h, bq_w;  // source base coordinate = j * bstr + bq
  int or_d, or_h, or_w;  // destination coordinate = j * ostr + or
};

struct FTap {
  int a_off;             // element offset of the tap's source voxel from the row's base voxel
  int w_off;             // element offset of W[tap][0][0]
  int dd, dh, dw;        // source coordinate offsets (bounds check)
};

struct FParams {
  int sd_, sh_, sw_, sc;       // gathered tensor extent and channels
  int dd, dh, dw, dc;          // destination extent and channels (GEMM columns)
  int bstr_d, bstr_h, bstr_w;  // source base stride per row coordinate
  int ostr_d, ostr_h, ostr_w;  // destination stride per row coordinate
  int wco;                     // weight row pitch (output channels of the layer)
  uint32_t src_bytes, w_bytes; // extents of the range-checked buffers
  int ncls;
  float alpha;
  int pod, poh, pow_;          // pooled extents (pooled epilogue)
  int rowtile;                 // output shift: a tile is one destination w row (C.m counts rows of w)
  FClass cls[F_MAX_CLS];
  FTap tap[F_MAX_TAPS];
};

__device__ __forceinline__ u32x4_t ld128(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
__device__ __forceinline__ u32x2_t ld64(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
}
__device__ __forceinline__ float f_of(uint32_t u) { return __uint_as_float(u); }

__device__ __forceinline__ float lrelu(float u, float a) { return u > 0.f ? u : a * u; }

// Shift mode: the operand of lane m (m = lane % 16) for kernel column uw is
// that of voxel m + uw (forward) or m - uw (backward-data) of the same
// 16-voxel fragment, a DPP row shift of the uw = 0 operand a; the lanes the
// shift leaves without a source take the edge fragment e (the next 16 voxels
// forward, the previous 16 backward) rotated into place.
template <int UWI, bool FWD>
__device__ __forceinline__ uint32_t shift_lane(uint32_t a, uint32_t e) {
  if constexpr (UWI == 0) {
    return a;
  } else {
    // a row rotate writes every lane: no old value to keep
    const int ed = __builtin_amdgcn_mov_dpp((int)e, FWD ? 0x120 + 16 - UWI : 0x120 + UWI, 0xf, 0xf, false);
    return (uint32_t)__builtin_amdgcn_update_dpp(ed, (int)a, FWD ? 0x100 + UWI : 0x110 + UWI, 0xf, 0xf, false);
  }
}

// EPI: 0 store the contraction, 1 bias + leaky ReLU (+ slope mask if mask != 0),
// 2 bias + leaky ReLU + slope mask + 2^3 average pool (forward, brick rows).
// UW > 0 (shift mode, a stride-1 class whose UW taps along w are consecutive in
// the tap table, destination w extent a multiple of 16): a k-step is one kernel
// row (kd, kh) x 16 channels.  A fragment's 16 lanes are 16 consecutive voxels
// along w, so the operand of tap column uw is the uw = 0 operand moved uw lanes
// along the 16-lane row (DPP row shift), the lanes shifted in at the edge coming
// from a second fragment 16 voxels further along (row rotate): two loads per
// fragment and kernel row instead of UW.
//
// DYY (backward-data of an unpooled fused layer): the gathered operand is
// dz = dy * (y > 0 ? 1 : alpha), formed from dy (src) and the layer's saved
// activation y (ysrc, the same layout) after both loads arrive.
//
// TK (taps in K, a stride-1 class whose 4 taps along w are consecutive in the
// tap table): a k-step is one kernel row (kd, kh) x 8 channels.  K slot g of an
// MFMA is tap column g of the row and register j of a lane's 16-byte load is
// channel c0 + j: lane (m, g) loads channels c0 .. c0 + 3 of its own source
// voxel, the one tap column g reads (m + g forward, m - g backward-data, along
// w), with its own range check.  Four loads per fragment and kernel row (two per
// k-step) instead of shift mode's two plus 24 lane moves, and no alignment of
// the fragments along w.  The launches use it for the forward.
//
// OS (output shift; backward-data of a stride-1 layer with 4 taps along w,
// tiles of whole destination w rows): one accumulator set per tap column uw
// holds P_uw[p] = sum over kernel rows and channels of dz[p] W[uw] for the
// source voxels p of the tile's own rows, unshifted; the epilogue adds
// P_uw[w + pw - uw] into dx[w].  One load per fragment and k-step, no lane moves.
//
// The kernel body runs as the workgroup of grid position (bx, by): the
// launch's own grid, or a share of the combined backward launch below.
template <bool FWD, int FM, int FN, int WM, int WK, int PF, int EPI, int UW = 0, bool DYY = false, bool TK = false,
          bool OS = false>
__device__ __forceinline__ void conv_f32_body(const float *__restrict__ src, const float *__restrict__ ysrc,
                                              const float *__restrict__ wt, const float *__restrict__ bias,
                                              float *__restrict__ dst, uint8_t *__restrict__ mask, const FParams p,
                                              int bx, int by) {
  constexpr int BM = 16 * FM * WM;           // rows of a tile
  constexpr int BN = 16 * FN;                // columns of a tile
  constexpr int RED_LD = BN + 4;             // fp32 row pitch of the reduction tile
  constexpr int NT = 64 * WM * WK;           // threads
  constexpr bool BRICK = EPI == 2;
  constexpr int TWB = BM / 4;                // brick: w extent of a tile (2 x 2 x TWB voxels)
  static_assert(!BRICK || (BM % 64 == 0 && FWD), "pooled tiles hold whole 16-row w segments");
  static_assert(FN == 1 || FN == 2 || FN == 4, "column groups");
  __shared__ __attribute__((aligned(16))) float red[WK * BM * RED_LD];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave % WM, wk = wave / WM;
  const int g4 = lane >> 4, r16 = lane & 15;

  // ---- class and tile of this workgroup (uniform), XCD-major --------------
  const int xcd = bx & 7, slot = bx >> 3;
  int c = 0;
  while (c + 1 < p.ncls && slot >= p.cls[c + 1].slot0) ++c;
  const FClass &C = p.cls[c];
  const int tile = xcd * C.per + slot - C.slot0;
  const int n0 = by * BN;
  int tb_n = 0, tb_d = 0, tb_h = 0, tb_w = 0;  // brick: sample, d pair, h pair, w tile
  if constexpr (BRICK) {
    if (tile >= C.m) return;
    const int t1 = fdiv(tile, C.fw), t2 = fdiv(t1, C.fh);
    tb_n = fdiv(t2, C.fd);
    tb_w = tile - t1 * (int)C.fw.div;
    tb_h = t1 - t2 * (int)C.fh.div;
    tb_d = t2 - tb_n * (int)C.fd.div;
  } else {
    if (p.rowtile ? tile >= C.m : tile * BM >= C.m) return;
  }
  const int m0 = tile * BM;

  const __amdgpu_buffer_rsrc_t srsrc = __builtin_amdgcn_make_buffer_rsrc((void *)src, (short)0, p.src_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t yrsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)ysrc, (short)0, DYY ? p.src_bytes : 0u, 0x00020000);
  const __amdgpu_buffer_rsrc_t wrsrc = __builtin_amdgcn_make_buffer_rsrc((void *)wt, (short)0, p.w_bytes, 0x00020000);
  // dz from dy and y, four channels at a time (DYY)
  auto slope4 = [&](u32x4_t d, u32x4_t y) {
    u32x4_t r;
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = __float_as_uint(f_of(d[j]) * (f_of(y[j]) > 0.f ? 1.f : p.alpha));
    return r;
  };
  (void)yrsrc;
  (void)slope4;

  // ---- source base of this lane's row in each of its fragments -------------
  int rbd[FM], rbh[FM], rbw[FM], roff[FM];
  bool rok[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int lrow = wm * 16 * FM + 16 * i + r16;  // row within the tile
    int n, jd, jh, jw;
    if constexpr (BRICK) {
      const int fi = lrow >> 4, seg = fi % (TWB / 16), dh2 = fi / (TWB / 16);
      n = tb_n;
      jd = 2 * tb_d + (dh2 >> 1);
      jh = 2 * tb_h + (dh2 & 1);
      jw = tb_w * TWB + seg * 16 + (lrow & 15);
      rok[i] = jd < p.dd && jh < p.dh && jw < p.dw;
    } else if (p.rowtile) {
      const int t2 = fdiv(tile, C.fh);
      n = fdiv(t2, C.fd);
      jw = lrow;
      jh = tile - t2 * (int)C.fh.div;
      jd = t2 - n * (int)C.fd.div;
      rok[i] = jw < (int)C.fw.div;
    } else {
      const int row = m0 + lrow;
      rok[i] = row < C.m;
      const int rr = rok[i] ? row : 0;
      const int t1 = fdiv(rr, C.fw), t2 = fdiv(t1, C.fh);
      n = fdiv(t2, C.fd);
      jw = rr - t1 * (int)C.fw.div;
      jh = t1 - t2 * (int)C.fh.div;
      jd = t2 - n * (int)C.fd.div;
    }
    if (!rok[i]) n = jd = jh = jw = 0;
    rbw[i] = jw * p.bstr_w + C.bq_w;
    rbh[i] = jh * p.bstr_h + C.bq_h;
    rbd[i] = jd * p.bstr_d + C.bq_d;
    roff[i] = (((n * p.sd_ + rbd[i]) * p.sh_ + rbh[i]) * p.sw_ + rbw[i]) * p.sc + 4 * g4;
  }

  // accumulators: forward acc[i][jj] holds columns co = n0 + FN*n + jj;
  // backward-data acc[i][v] holds columns n0 + 16 v + n
  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  f32x4_t acco[OS ? 4 : 1][OS ? FM : 1][OS ? FN : 1];  // output shift: one set per tap column
  if constexpr (OS) {
    static_assert(!FWD && !DYY && UW == 0 && !TK && WM == 1 && WK == 1 && EPI == 0, "output shift: backward-data");
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int v = 0; v < FN; ++v) acco[u][i][v] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int nch = p.sc >> 4;
    const int nsteps = (C.ntap >> 2) * nch;  // kernel rows x 16-channel chunks
    int ri = 0, cc = 0, ldstep = 0;
    auto next = [&]() {  // branch-free: see the linear cursor below
      ++ldstep;
      const int c1 = cc + (ldstep < nsteps ? 1 : 0);
      const bool wrap = c1 == nch;
      cc = wrap ? 0 : c1;
      ri += wrap ? 1 : 0;
    };
    // a row's source voxel along w is its own w (the tile's rows are whole w rows)
    int soff[FM];
    bool swok[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      soff[i] = roff[i] - C.bq_w * p.sc;
      swok[i] = rok[i] & ((unsigned)(rbw[i] - C.bq_w) < (unsigned)p.sw_);
    }
    int wl[FN];
#pragma unroll
    for (int v = 0; v < FN; ++v) wl[v] = (n0 + 16 * v + r16) * p.wco + 4 * g4;  // W[t][n0 + 16 v + r][4g ..]
    constexpr int NS = PF + 1;
    u32x4_t a_r[NS][FM];
    uint32_t b_r[NS][4][FN][4];
    auto load = [&](u32x4_t(&a)[FM], uint32_t(&b)[4][FN][4]) {
      const FTap &T = p.tap[C.tap0 + ri * 4];
      const int cofs = cc * 16;
      const bool live = ldstep < nsteps;
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const bool ok = live & swok[i] & ((unsigned)(rbd[i] + T.dd) < (unsigned)p.sd_) &
                        ((unsigned)(rbh[i] + T.dh) < (unsigned)p.sh_);
        // a valid byte offset is below 2^31: bit 31 sends the load past the buffer (zeros)
        a[i] = ld128(srsrc, ((uint32_t)(soff[i] + T.a_off + cofs) * 4u) | ((uint32_t)!ok << 31));
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int wbase = p.tap[C.tap0 + ri * 4 + u].w_off + cofs;
#pragma unroll
        for (int v = 0; v < FN; ++v) {
          const u32x4_t q = ld128(wrsrc, (uint32_t)(wl[v] + wbase) * 4u);
          b[u][v][0] = q[0]; b[u][v][1] = q[1]; b[u][v][2] = q[2]; b[u][v][3] = q[3];
        }
      }
    };
    if (nsteps > 0) {
      const int niter = (nsteps + NS - 1) / NS * NS;
#pragma unroll
      for (int q = 0; q < PF; ++q) {
        load(a_r[q], b_r[q]);
        next();
      }
      for (int s0 = 0; s0 < niter; s0 += NS) {
#pragma unroll
        for (int q = 0; q < NS; ++q) {
          load(a_r[(q + PF) % NS], b_r[(q + PF) % NS]);
          next();
          __builtin_amdgcn_sched_barrier(0);  // prefetch loads stay ahead of the MFMAs
#pragma unroll
          for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
              for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < FN; ++v)
                  acco[u][i][v] = __builtin_amdgcn_mfma_f32_16x16x4f32(f_of(a_r[q][i][j]), f_of(b_r[q][u][v][j]),
                                                                       acco[u][i][v], 0, 0, 0);
        }
      }
    }
  } else if constexpr (TK) {
    // ---- taps in K: k-steps are kernel rows (4 taps) x 8 channels ------------
    static_assert(!DYY && UW == 0, "taps-in-K mode reads a plain source");
    constexpr int SG = FWD ? 1 : -1;            // source voxel of tap column g: m + SG g along w
    const int nch = p.sc >> 3;
    const int nrows = C.ntap >> 2;
    const int myrows = nrows > wk ? (nrows - wk + WK - 1) / WK : 0;
    const int nsteps = myrows * nch;
    int ri = wk, cc = 0, ldstep = 0;
    auto next = [&]() {  // branch-free: see the linear cursor below
      ++ldstep;
      const int c1 = cc + (ldstep < nsteps ? 1 : 0);
      const bool wrap = c1 == nch;
      cc = wrap ? 0 : c1;
      ri += wrap ? WK : 0;
    };
    // this lane's K slot is tap column g4: its source voxel and w range check
    // (tap column 0 of every row has dw = 0), and the weights of its tap
    int aoff[FM];
    bool wok[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      aoff[i] = roff[i] - 4 * g4 + SG * g4 * p.sc;
      wok[i] = rok[i] & ((unsigned)(rbw[i] + SG * g4) < (unsigned)p.sw_);
    }
    const int tstr = p.wco * (FWD ? p.sc : p.dc);  // elements from one tap's weights to the next
    constexpr int NB = FWD ? 4 : FN;              // weight loads per channel quad
    constexpr int BW = FWD ? FN : 4;              // floats per weight load
    int wl[NB];
#pragma unroll
    for (int v = 0; v < NB; ++v)
      wl[v] = g4 * tstr + (FWD ? v * p.wco + n0 + FN * r16      // W[t_g][c0 + v][n0 + FN r ..]
                               : (n0 + 16 * v + r16) * p.wco);  // W[t_g][n0 + 16 v + r][c0 ..]
    constexpr int NS = PF + 1;
    u32x4_t a_r[NS][2][FM];
    uint32_t b_r[NS][2][NB][BW];
    auto load = [&](u32x4_t(&a)[2][FM], uint32_t(&b)[2][NB][BW]) {
      const FTap &T = p.tap[C.tap0 + ri * 4];
      const int cofs = cc * 8;
      const bool live = ldstep < nsteps;
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const bool ok = live & wok[i] & ((unsigned)(rbd[i] + T.dd) < (unsigned)p.sd_) &
                        ((unsigned)(rbh[i] + T.dh) < (unsigned)p.sh_);
        // a masked lane reads from 2^31, past the buffer (zeros) for both loads: OR-ing
        // bit 31 into a negative offset could wrap back into range at + 16
        const uint32_t o = ok ? (uint32_t)(aoff[i] + T.a_off + cofs) * 4u : 0x80000000u;
        a[0][i] = ld128(srsrc, o);
        a[1][i] = ld128(srsrc, o + 16u);
      }
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int wbase = T.w_off + (cofs + 4 * c) * (FWD ? p.wco : 1);
#pragma unroll
        for (int v = 0; v < NB; ++v) {
          const uint32_t off = (uint32_t)(wl[v] + wbase) * 4u;
          if constexpr (BW == 4) {
            const u32x4_t q = ld128(wrsrc, off);
            b[c][v][0] = q[0]; b[c][v][1] = q[1]; b[c][v][2] = q[2]; b[c][v][3] = q[3];
          } else if constexpr (BW == 2) {
            const u32x2_t q = ld64(wrsrc, off);
            b[c][v][0] = q[0]; b[c][v][1] = q[1];
          } else {
            b[c][v][0] = __builtin_amdgcn_raw_buffer_load_b32(wrsrc, off, 0, 0);
          }
        }
      }
    };
    if (nsteps > 0) {
      const int niter = (nsteps + NS - 1) / NS * NS;
#pragma unroll
      for (int q = 0; q < PF; ++q) {
        load(a_r[q], b_r[q]);
        next();
      }
      for (int s0 = 0; s0 < niter; s0 += NS) {
#pragma unroll
        for (int q = 0; q < NS; ++q) {
          load(a_r[(q + PF) % NS], b_r[(q + PF) % NS]);
          next();
          __builtin_amdgcn_sched_barrier(0);  // prefetch loads stay ahead of the MFMAs
#pragma unroll
          for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
              for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < FN; ++v) {
                  const float bv = FWD ? f_of(b_r[q][c][j][v]) : f_of(b_r[q][c][v][j]);
                  acc[i][v] = __builtin_amdgcn_mfma_f32_16x16x4f32(f_of(a_r[q][c][i][j]), bv, acc[i][v], 0, 0, 0);
                }
        }
      }
    }
  } else if constexpr (UW > 0) {
    // ---- shift mode: k-steps are kernel rows (UW taps) x 16 channels ---------
    const int nch = p.sc >> 4;
    const int nrows = C.ntap / UW;
    const int myrows = nrows > wk ? (nrows - wk + WK - 1) / WK : 0;
    const int nsteps = myrows * nch;
    int ri = wk, cc = 0, ldstep = 0;
    auto next = [&]() {  // branch-free: see the linear cursor below
      ++ldstep;
      const int c1 = cc + (ldstep < nsteps ? 1 : 0);
      const bool wrap = c1 == nch;
      cc = wrap ? 0 : c1;
      ri += wrap ? WK : 0;
    };
    constexpr int NB = FWD ? 4 : FN;
    constexpr int BW = FWD ? FN : 4;
    int wl[NB];
#pragma unroll
    for (int v = 0; v < NB; ++v)
      wl[v] = FWD ? (4 * g4 + v) * p.wco + n0 + FN * r16 : (n0 + 16 * v + r16) * p.wco + 4 * g4;
    constexpr int EDGE = FWD ? 16 : -16;  // voxels from a fragment to its edge fragment
    constexpr int NS = PF + 1;
    u32x4_t a_r[NS][FM], e_r[NS][FM];
    u32x4_t ya_r[DYY ? NS : 1][FM], ye_r[DYY ? NS : 1][FM];
    uint32_t b_r[NS][UW][NB][BW];
    auto load = [&](u32x4_t(&a)[FM], u32x4_t(&e)[FM], u32x4_t(&ya)[FM], u32x4_t(&ye)[FM],
                    uint32_t(&b)[UW][NB][BW]) {
      const FTap &T = p.tap[C.tap0 + ri * UW];
      const int cofs = cc * 16;
      const bool live = ldstep < nsteps;
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const bool dh = live & rok[i] & ((unsigned)(rbd[i] + T.dd) < (unsigned)p.sd_) &
                        ((unsigned)(rbh[i] + T.dh) < (unsigned)p.sh_);
        const int w0 = rbw[i] + T.dw;
        const bool oka = dh & ((unsigned)w0 < (unsigned)p.sw_);
        const bool oke = dh & ((unsigned)(w0 + EDGE) < (unsigned)p.sw_);
        const int o = roff[i] + T.a_off + cofs;
        a[i] = ld128(srsrc, ((uint32_t)o * 4u) | ((uint32_t)!oka << 31));
        e[i] = ld128(srsrc, ((uint32_t)(o + EDGE * p.sc) * 4u) | ((uint32_t)!oke << 31));
        if constexpr (DYY) {
          ya[i] = ld128(yrsrc, ((uint32_t)o * 4u) | ((uint32_t)!oka << 31));
          ye[i] = ld128(yrsrc, ((uint32_t)(o + EDGE * p.sc) * 4u) | ((uint32_t)!oke << 31));
        }
      }
#pragma unroll
      for (int uw = 0; uw < UW; ++uw) {
        const int wbase = p.tap[C.tap0 + ri * UW + uw].w_off + cofs * (FWD ? p.wco : 1);
#pragma unroll
        for (int v = 0; v < NB; ++v) {
          const uint32_t off = (uint32_t)(wl[v] + wbase) * 4u;
          if constexpr (BW == 4) {
            const u32x4_t q = ld128(wrsrc, off);
            b[uw][v][0] = q[0]; b[uw][v][1] = q[1]; b[uw][v][2] = q[2]; b[uw][v][3] = q[3];
          } else if constexpr (BW == 2) {
            const u32x2_t q = ld64(wrsrc, off);
            b[uw][v][0] = q[0]; b[uw][v][1] = q[1];
          } else {
            b[uw][v][0] = __builtin_amdgcn_raw_buffer_load_b32(wrsrc, off, 0, 0);
          }
        }
      }
    };
    if (nsteps > 0) {
      const int niter = (nsteps + NS - 1) / NS * NS;
#pragma unroll
      for (int q = 0; q < PF; ++q) {
        load(a_r[q], e_r[q], ya_r[DYY ? q : 0], ye_r[DYY ? q : 0], b_r[q]);
        next();
      }
      for (int s0 = 0; s0 < niter; s0 += NS) {
#pragma unroll
        for (int q = 0; q < NS; ++q) {
          load(a_r[(q + PF) % NS], e_r[(q + PF) % NS], ya_r[DYY ? (q + PF) % NS : 0], ye_r[DYY ? (q + PF) % NS : 0],
               b_r[(q + PF) % NS]);
          if constexpr (DYY) {
#pragma unroll
            for (int i = 0; i < FM; ++i) {
              a_r[q][i] = slope4(a_r[q][i], ya_r[q][i]);
              e_r[q][i] = slope4(e_r[q][i], ye_r[q][i]);
            }
          }
          next();
          __builtin_amdgcn_sched_barrier(0);  // prefetch loads stay ahead of the MFMAs
          // a column's shifted operands of every fragment first, then its MFMAs:
          // interleaved one operand at a time, the moves and the MFMA reading
          // their result stall on each other
          auto column = [&](auto uwc) {
            constexpr int uw = decltype(uwc)::value;
            uint32_t av[FM][4];
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
              for (int j = 0; j < 4; ++j) av[i][j] = shift_lane<uw, FWD>(a_r[q][i][j], e_r[q][i][j]);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
              for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < FN; ++v) {
                  const float bv = FWD ? f_of(b_r[q][uw][j][v]) : f_of(b_r[q][uw][v][j]);
                  acc[i][v] = __builtin_amdgcn_mfma_f32_16x16x4f32(f_of(av[i][j]), bv, acc[i][v], 0, 0, 0);
                }
          };
          column(std::integral_constant<int, 0>{});
          if constexpr (UW > 1) column(std::integral_constant<int, 1>{});
          if constexpr (UW > 2) column(std::integral_constant<int, 2>{});
          if constexpr (UW > 3) column(std::integral_constant<int, 3>{});
        }
      }
    }
  } else {
  // ---- this wave's k-steps: taps wk, wk + WK, ... of the class, 16 channels each
    const int nch = p.sc >> 4;
    const int mytaps = C.ntap > wk ? (C.ntap - wk + WK - 1) / WK : 0;
    const int nsteps = mytaps * nch;
    // load cursor: tap, channel chunk, and the number of steps loaded so far; past
    // the last real step the cursor stays put (valid weight addresses) and the A
    // loads take the out-of-range offset, so padded steps multiply zeros
    int ti = wk, cc = 0, ldstep = 0;
    // branch-free (scalar selects): control flow between the ring's steps lets
    // the compiler sink the prefetch loads and wait for all of them at once
    auto next = [&]() {
      ++ldstep;
      const int c1 = cc + (ldstep < nsteps ? 1 : 0);
      const bool wrap = c1 == nch;
      cc = wrap ? 0 : c1;
      ti += wrap ? WK : 0;
    };
  
    // lane part of the weight element offsets
    constexpr int NB = FWD ? 4 : FN;  // weight loads per k-step
    int wl[NB];
  #pragma unroll
    for (int v = 0; v < NB; ++v)
      wl[v] = FWD ? (4 * g4 + v) * p.wco + n0 + FN * r16      // W[t][4g + v][n0 + FN r ..]
                  : (n0 + 16 * v + r16) * p.wco + 4 * g4;     // W[t][n0 + 16 v + r][4g ..]
  
    constexpr int NS = PF + 1;
    constexpr int BW = FWD ? FN : 4;  // floats per weight load
    u32x4_t a_r[NS][FM];
    u32x4_t ya_r[DYY ? NS : 1][FM];
    uint32_t b_r[NS][NB][BW];
    auto load = [&](u32x4_t(&a)[FM], u32x4_t(&ya)[FM], uint32_t(&b)[NB][BW]) {
      const FTap &T = p.tap[C.tap0 + ti];
      const int cofs = cc * 16;
      const bool live = ldstep < nsteps;
  #pragma unroll
      for (int i = 0; i < FM; ++i) {
        // bitwise, not short-circuit: one select per load, no branch
        const bool ok = live & rok[i] & ((unsigned)(rbd[i] + T.dd) < (unsigned)p.sd_) &
                        ((unsigned)(rbh[i] + T.dh) < (unsigned)p.sh_) & ((unsigned)(rbw[i] + T.dw) < (unsigned)p.sw_);
        // a valid byte offset is below 2^31: setting bit 31 sends the load past the
        // buffer (it returns zeros) without a select the compiler could turn into a branch
        a[i] = ld128(srsrc, ((uint32_t)(roff[i] + T.a_off + cofs) * 4u) | ((uint32_t)!ok << 31));
        if constexpr (DYY) ya[i] = ld128(yrsrc, ((uint32_t)(roff[i] + T.a_off + cofs) * 4u) | ((uint32_t)!ok << 31));
      }
      const int wbase = T.w_off + cofs * (FWD ? p.wco : 1);
  #pragma unroll
      for (int v = 0; v < NB; ++v) {
        const uint32_t off = (uint32_t)(wl[v] + wbase) * 4u;
        if constexpr (BW == 4) {
          const u32x4_t q = ld128(wrsrc, off);
          b[v][0] = q[0]; b[v][1] = q[1]; b[v][2] = q[2]; b[v][3] = q[3];
        } else if constexpr (BW == 2) {
          const u32x2_t q = ld64(wrsrc, off);
          b[v][0] = q[0]; b[v][1] = q[1];
        } else {
          b[v][0] = __builtin_amdgcn_raw_buffer_load_b32(wrsrc, off, 0, 0);
        }
      }
    };
  
    // Branch-free steady state: the step count is padded to a multiple of the
    // ring size; padded steps load zero A fragments (see the cursor).
    if (nsteps > 0) {
      const int niter = (nsteps + NS - 1) / NS * NS;
  #pragma unroll
      for (int q = 0; q < PF; ++q) {
        load(a_r[q], ya_r[DYY ? q : 0], b_r[q]);
        next();
      }
      for (int s0 = 0; s0 < niter; s0 += NS) {
  #pragma unroll
        for (int q = 0; q < NS; ++q) {
          const int s = s0 + q;
          load(a_r[(q + PF) % NS], ya_r[DYY ? (q + PF) % NS : 0], b_r[(q + PF) % NS]);
          next();
          // keep the prefetch loads ahead of this step's MFMAs: sunk below them,
          // the wait before the next step would cover every load in flight
          __builtin_amdgcn_sched_barrier(0);
          (void)s;
  #pragma unroll
          for (int i = 0; i < FM; ++i) {
            u32x4_t av = a_r[q][i];
            if constexpr (DYY) av = slope4(av, ya_r[q][i]);
  #pragma unroll
            for (int j = 0; j < 4; ++j) {
  #pragma unroll
              for (int v = 0; v < FN; ++v) {
                const float bv = FWD ? f_of(b_r[q][j][v]) : f_of(b_r[q][v][j]);
                acc[i][v] = __builtin_amdgcn_mfma_f32_16x16x4f32(f_of(av[j]), bv, acc[i][v], 0, 0, 0);
              }
            }
          }
        }
      }
    }
  
  }

  if constexpr (OS) {
    // ---- output shift: dx[w] = sum over tap columns k of P_k[w + pw - k] (zero
    // past the ends of the w row), one tap column at a time through the LDS tile
    const int jwn = (int)C.fw.div;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int v = 0; v < FN; ++v)
#pragma unroll
          for (int e = 0; e < 4; ++e) red[(16 * i + 4 * g4 + e) * RED_LD + 16 * v + r16] = acco[k][i][v][e];
      __syncthreads();
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = 16 * i + 4 * g4 + e, jw = p.rowtile ? row : row % jwn;
          const int sw = jw + C.bq_w - k;
          if ((unsigned)sw < (unsigned)jwn) {
#pragma unroll
            for (int v = 0; v < FN; ++v) acc[i][v][e] += red[(row - jw + sw) * RED_LD + 16 * v + r16];
          }
        }
      __syncthreads();
    }
  }

  // ---- partial tiles meet in LDS -------------------------------------------
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int v = 0; v < FN; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = wm * 16 * FM + 16 * i + 4 * g4 + e;
        const int col = FWD ? FN * r16 + v : 16 * v + r16;
        red[(wk * BM + row) * RED_LD + col] = acc[i][v][e];
      }
  __syncthreads();

  constexpr int CV = BN / 8;  // 8-channel chunks per row
  for (int it = threadIdx.x; it < BM * CV; it += NT) {
    const int row = it / CV, c8 = it % CV;
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = 0.f;
#pragma unroll
    for (int k = 0; k < WK; ++k) {
      const float4 x0 = *reinterpret_cast<const float4 *>(&red[(k * BM + row) * RED_LD + 8 * c8]);
      const float4 x1 = *reinterpret_cast<const float4 *>(&red[(k * BM + row) * RED_LD + 8 * c8 + 4]);
      o[0] += x0.x; o[1] += x0.y; o[2] += x0.z; o[3] += x0.w;
      o[4] += x1.x; o[5] += x1.y; o[6] += x1.z; o[7] += x1.w;
    }
    // destination voxel of this row
    int n, od_, oh_, ow_;
    bool valid;
    if constexpr (BRICK) {
      const int fi = row >> 4, seg = fi % (TWB / 16), dh2 = fi / (TWB / 16);
      n = tb_n;
      od_ = 2 * tb_d + (dh2 >> 1);
      oh_ = 2 * tb_h + (dh2 & 1);
      ow_ = tb_w * TWB + seg * 16 + (row & 15);
      valid = od_ < p.dd && oh_ < p.dh && ow_ < p.dw;
    } else if (p.rowtile) {
      const int t2 = fdiv(tile, C.fh);
      n = fdiv(t2, C.fd);
      valid = row < (int)C.fw.div;
      ow_ = row * p.ostr_w + C.or_w;
      oh_ = (tile - t2 * (int)C.fh.div) * p.ostr_h + C.or_h;
      od_ = (t2 - n * (int)C.fd.div) * p.ostr_d + C.or_d;
    } else {
      const int grow = m0 + row;
      valid = grow < C.m;
      const int rr = valid ? grow : 0;
      const int t1 = fdiv(rr, C.fw), t2 = fdiv(t1, C.fh);
      n = fdiv(t2, C.fd);
      ow_ = (rr - t1 * (int)C.fw.div) * p.ostr_w + C.or_w;
      oh_ = (t1 - t2 * (int)C.fh.div) * p.ostr_h + C.or_h;
      od_ = (t2 - n * (int)C.fd.div) * p.ostr_d + C.or_d;
    }
    const long long e0 = ((((long long)n * p.dd + od_) * p.dh + oh_) * p.dw + ow_) * p.dc + n0 + 8 * c8;
    if constexpr (EPI >= 1) {
      uint32_t bits = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float u = o[e] + bias[n0 + 8 * c8 + e];
        bits |= (u > 0.f ? 1u : 0u) << e;
        o[e] = lrelu(u, p.alpha);
      }
      if (valid && mask) mask[e0 >> 3] = (uint8_t)bits;
    }
    if constexpr (BRICK) {
      // y stays in the tile for the pooling pass (each (row, chunk) has one owner)
      *reinterpret_cast<float4 *>(&red[row * RED_LD + 8 * c8]) = make_float4(o[0], o[1], o[2], o[3]);
      *reinterpret_cast<float4 *>(&red[row * RED_LD + 8 * c8 + 4]) = make_float4(o[4], o[5], o[6], o[7]);
    } else {
      if (valid) {
        *reinterpret_cast<float4 *>(dst + e0) = make_float4(o[0], o[1], o[2], o[3]);
        *reinterpret_cast<float4 *>(dst + e0 + 4) = make_float4(o[4], o[5], o[6], o[7]);
      }
    }
  }
  if constexpr (BRICK) {
    // ---- 2^3 average pool of the tile's y: TWB/2 pooled voxels x BN channels
    __syncthreads();
    constexpr int NSEG = TWB / 16;
    for (int it = threadIdx.x; it < (TWB / 2) * CV; it += NT) {
      const int pw = it / CV, c8 = it % CV;
      const int pwg = tb_w * (TWB / 2) + pw;
      if (tb_d >= p.pod || tb_h >= p.poh || pwg >= p.pow_) continue;
      float s[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] = 0.f;
#pragma unroll
      for (int dh2 = 0; dh2 < 4; ++dh2)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int wl_ = 2 * pw + t;
          const int row = (dh2 * NSEG + (wl_ >> 4)) * 16 + (wl_ & 15);
          const float4 x0 = *reinterpret_cast<const float4 *>(&red[row * RED_LD + 8 * c8]);
          const float4 x1 = *reinterpret_cast<const float4 *>(&red[row * RED_LD + 8 * c8 + 4]);
          s[0] += x0.x; s[1] += x0.y; s[2] += x0.z; s[3] += x0.w;
          s[4] += x1.x; s[5] += x1.y; s[6] += x1.z; s[7] += x1.w;
        }
      const long long q0 = ((((long long)tb_n * p.pod + tb_d) * p.poh + tb_h) * p.pow_ + pwg) * p.dc + n0 + 8 * c8;
      *reinterpret_cast<float4 *>(dst + q0) =
          make_float4(s[0] * 0.125f, s[1] * 0.125f, s[2] * 0.125f, s[3] * 0.125f);
      *reinterpret_cast<float4 *>(dst + q0 + 4) =
          make_float4(s[4] * 0.125f, s[5] * 0.125f, s[6] * 0.125f, s[7] * 0.125f);
    }
  }
}

template <bool FWD, int FM, int FN, int WM, int WK, int PF, int EPI, int UW = 0, bool DYY = false, bool TK = false,
          bool OS = false>
__global__ __launch_bounds__(64 * WM * WK) void conv_f32_kernel(const float *__restrict__ src,
                                                                const float *__restrict__ ysrc,
                                                                const float *__restrict__ wt,
                                                                const float *__restrict__ bias,
                                                                float *__restrict__ dst, uint8_t *__restrict__ mask,
                                                                const FParams p) {
  conv_f32_body<FWD, FM, FN, WM, WK, PF, EPI, UW, DYY, TK, OS>(src, ysrc, wt, bias, dst, mask, p, blockIdx.x,
                                                               blockIdx.y);
}

// Class and tap tables (forward: one class; backward-data: s^3 parity classes).
void f_tables(const ConvShape &s, bool fwd, FParams &p) {
  const int S[3] = {s.sd, s.sh, s.sw}, P[3] = {s.pd, s.ph, s.pw}, K[3] = {s.kd, s.kh, s.kw};
  const int IN[3] = {s.d, s.h, s.w}, OUT[3] = {s.od, s.oh, s.ow};
  const int *SRC = fwd ? IN : OUT;
  const int *DST = fwd ? OUT : IN;
  p.sd_ = SRC[0]; p.sh_ = SRC[1]; p.sw_ = SRC[2];
  p.dd = DST[0]; p.dh = DST[1]; p.dw = DST[2];
  p.sc = fwd ? s.ci : s.co;
  p.dc = fwd ? s.co : s.ci;
  p.bstr_d = fwd ? s.sd : 1; p.bstr_h = fwd ? s.sh : 1; p.bstr_w = fwd ? s.sw : 1;
  p.ostr_d = fwd ? 1 : s.sd; p.ostr_h = fwd ? 1 : s.sh; p.ostr_w = fwd ? 1 : s.sw;
  p.wco = s.co;
  p.ncls = fwd ? 1 : s.sd * s.sh * s.sw;
  int ntaps = 0;
  for (int c = 0; c < p.ncls; ++c) {
    const int r[3] = {fwd ? 0 : c / (s.sh * s.sw), fwd ? 0 : (c / s.sw) % s.sh, fwd ? 0 : c % s.sw};
    int J[3], U[3], T0[3], Q[3];
    for (int a = 0; a < 3; ++a) {
      if (fwd) {
        J[a] = OUT[a]; U[a] = K[a]; T0[a] = 0; Q[a] = -P[a];
      } else {
        J[a] = IN[a] > r[a] ? (IN[a] - r[a] + S[a] - 1) / S[a] : 0;
        T0[a] = (r[a] + P[a]) % S[a];
        U[a] = T0[a] < K[a] ? (K[a] - T0[a] + S[a] - 1) / S[a] : 0;
        Q[a] = (r[a] + P[a] - T0[a]) / S[a];
      }
    }
    FClass &C = p.cls[c];
    C.m = s.n * J[0] * J[1] * J[2];
    C.fw = make_fastdiv(std::max(J[2], 1));
    C.fh = make_fastdiv(std::max(J[1], 1));
    C.fd = make_fastdiv(std::max(J[0], 1));
    C.bq_d = Q[0]; C.bq_h = Q[1]; C.bq_w = Q[2];
    C.or_d = r[0]; C.or_h = r[1]; C.or_w = r[2];
    C.tap0 = ntaps;
    C.ntap = U[0] * U[1] * U[2];
    const int sg = fwd ? 1 : -1;
    const int st_d = fwd ? 1 : S[0], st_h = fwd ? 1 : S[1], st_w = fwd ? 1 : S[2];
    for (int ud = 0; ud < U[0]; ++ud)
      for (int uh = 0; uh < U[1]; ++uh)
        for (int uw = 0; uw < U[2]; ++uw) {
          FTap &T = p.tap[ntaps++];
          T.dd = sg * ud; T.dh = sg * uh; T.dw = sg * uw;
          T.a_off = ((T.dd * p.sh_ + T.dh) * p.sw_ + T.dw) * p.sc;
          const int tap = ((T0[0] + st_d * ud) * s.kh + (T0[1] + st_h * uh)) * s.kw + (T0[2] + st_w * uw);
          T.w_off = tap * s.ci * s.co;
        }
  }
  p.src_bytes = (uint32_t)((long long)s.n * p.sd_ * p.sh_ * p.sw_ * p.sc * 4);
  p.w_bytes = (uint32_t)((long long)s.kd * s.kh * s.kw * s.ci * s.co * 4);
}

// XCD-major grid over tiles of `unit` rows (bricks: units are bricks, unit = 1);
// returns its size (a multiple of 8)
int f_assign(FParams &p, int unit) {
  int slots = 0;
  for (int c = 0; c < p.ncls; ++c) {
    const int tiles = (p.cls[c].m + unit - 1) / unit;
    p.cls[c].slot0 = slots;
    p.cls[c].per = (tiles + 7) / 8;
    slots += p.cls[c].per;
  }
  return 8 * slots;
}

struct FCfg {
  int fm, wm, wk;
};

// the tile shapes instantiated for the linear layout (fm, wm, wk)
constexpr FCfg kCand[] = {{4, 1, 1}, {4, 2, 1}, {2, 2, 1}, {4, 1, 4}, {2, 1, 4}, {1, 1, 4}, {1, 1, 8}, {2, 1, 8}};
constexpr int kNCand = sizeof(kCand) / sizeof(kCand[0]);

template <bool FWD, int FN, int EPI, int FM, int WM, int WK, int UW = 0, bool DYY = false, bool TK = false,
          bool OS = false>
hipError_t launch_f(const FParams &p, int tiles, const float *src, const float *w, const float *bias, float *dst,
                    uint8_t *mask, hipStream_t st, const float *ysrc = nullptr) {
  dim3 grid((unsigned)tiles, p.dc / (16 * FN), 1);
  if (grid.x == 0 || grid.y == 0) return hipSuccess;
  // shift-mode and taps-in-K k-steps hold four taps: one step of prefetch covers
  // the latency
  constexpr int PF = UW > 0 || TK || OS ? 1 : 2;
  hipLaunchKernelGGL((conv_f32_kernel<FWD, FM, FN, WM, WK, PF, EPI, UW, DYY, TK, OS>), grid, dim3(64 * WM * WK), 0, st,
                     src, ysrc, w, bias, dst, mask, p);
  return hipGetLastError();
}

// shift mode applies to one stride-1 class (forward, or backward-data of a
// stride-1 layer) with 4 taps along w, a destination w extent that is a
// multiple of 16 (every fragment is 16 consecutive voxels of one row) and
// source w stride 1.  CF_F32_SHIFT=0 turns it off, =1 uses it wherever it
// applies, whatever the size (the tests cover both on small shapes).
int f_shift_env() {
  const char *e = getenv("CF_F32_SHIFT");
  return e ? (e[0] == '0' ? 0 : 1) : -1;
}
// Taps in K replaces shift mode in the forward (the 16 -> 32 layer's pooled
// forward at 128^3: 169 -> 155 us) and, needing no 16-voxel alignment, the
// linear tiles of 4-wide forwards whose w extent is not a multiple of 16 (the
// paper's 63^3 -> 60^3 layer at batch 1: 160 -> 146 us).  Backward-data keeps shift mode: its source
// holds 32 channels, 128 bytes per voxel, so each 16-byte lane load touches its
// own cache line, and taps in K issues twice the loads (measured 195 -> 281 us).
// CF_F32_TK=0 keeps shift mode everywhere.
bool f_tk() {
  const char *e = getenv("CF_F32_TK");
  return !(e && e[0] == '0');
}
// Output shift replaces shift mode in backward-data (16 destination channels)
// where the destination w rows tile the 64-row tiles exactly (w extent 16, 32
// or 64), or fill one tile each (other w extents from 33 to 63: a tile per w
// row, the rows past the extent idle; the paper's 60^3 -> 63^3 backward-data),
// the source no wider along w.  CF_F32_OS=0 keeps shift mode.
bool f_os_ok(const ConvShape &s, const FParams &p) {
  const char *e = getenv("CF_F32_OS");
  if (e && e[0] == '0') return false;
  const int jw = (int)p.cls[0].fw.div;
  return f_shift_env() != 0 && p.ncls == 1 && s.kw == 4 && (jw == 16 || (jw >= 32 && jw <= 64)) && p.sw_ <= jw;
}
// taps in K needs 4 taps along w in one class (any stride, any w extent), and
// is used on 16-channel sources: with 32 channels, 128 bytes per voxel, every
// lane's 16-byte load touches its own cache line (the paper's 30^3 -> 27^3
// layer inside its step: 83 -> 139 us)
bool f_tk_ok(const ConvShape &s, const FParams &p) {
  return f_shift_env() != 0 && p.ncls == 1 && s.kw == 4 && p.sc == 16;
}
bool f_shift_ok(const ConvShape &s, const FParams &p) {
  if (f_shift_env() == 0) return false;
  return p.ncls == 1 && s.sw == 1 && s.kw == 4 && p.dw % 16 == 0 && p.bstr_w == 1 && p.ostr_w == 1;
}

// Relative cost of a tile shape: a wave's MFMAs (k-steps x 4 x FM x FN) plus a
// fixed per-wave overhead (prologue, reduction, epilogue; about 200 MFMAs,
// fitted to the stack's layers), times the rounds of 2048 waves (two per SIMD)
// the launch needs.  Ranks the shapes as measured on the 16 -> 32 layer and
// the deep layers at batch 1.
double f_cost(FParams &p, const FCfg &c, int fn) {
  const long long ny = p.dc / (16 * fn);
  const long long waves = (long long)f_assign(p, 16 * c.fm * c.wm) * ny * c.wm * c.wk;
  int maxtap = 0;
  for (int k = 0; k < p.ncls; ++k) maxtap = std::max(maxtap, p.cls[k].ntap);
  const double steps = (double)((maxtap + c.wk - 1) / c.wk) * (p.sc / 16);
  const double rounds = std::max(1.0, (double)waves / (8.0 * kNumCUs));
  return rounds * (steps * 4.0 * c.fm * fn + 200.0);
}

// The tile of a linear-layout launch: shift mode (pick -1) for the large
// stride-1 4-wide layers, else the candidate of least cost.
template <int FN>
int f_pick(const ConvShape &s, FParams &p, double *cost, bool fwd) {
  const bool four = fwd && f_tk() ? f_tk_ok(s, p) : (!fwd && FN == 1 && f_os_ok(s, p)) || f_shift_ok(s, p);
  if (four && !getenv("CF_F32_TILE") &&
      (f_shift_env() == 1 || f_assign(p, 64) * (p.dc / (16 * FN)) >= 4 * kNumCUs)) {
    *cost = 0.0;
    return -1;
  }
  int pick = 0;
  double best = 0.0;
  for (int i = 0; i < kNCand; ++i) {
    const double c = f_cost(p, kCand[i], FN);
    if (i == 0 || c < best) {
      best = c;
      pick = i;
    }
  }
  // CF_F32_TILE=i forces candidate i (the tests cover every one this way)
  if (const char *forced = getenv("CF_F32_TILE")) pick = std::min(kNCand - 1, std::max(0, atoi(forced)));
  *cost = best;
  return pick;
}

template <bool FWD, int FN, int EPI, bool DYY = false>
hipError_t launch_lin(const ConvShape &s, FParams &p, const float *src, const float *w, const float *bias, float *dst,
                      uint8_t *mask, hipStream_t st, const float *ysrc = nullptr) {
  double cost;
  const int pick = f_pick<FN>(s, p, &cost, FWD);
  if (pick < 0) {
    if constexpr (FWD && !DYY) {
      if (f_tk()) return launch_f<FWD, FN, EPI, 4, 1, 1, 0, false, true>(p, f_assign(p, 64), src, w, bias, dst, mask, st);
    }
    if constexpr (!FWD && !DYY && FN == 1 && EPI == 0) {
      if (f_os_ok(s, p)) {
        const int jw = (int)p.cls[0].fw.div;
        if (64 % jw != 0) {  // a tile per destination w row
          p.rowtile = 1;
          p.cls[0].m /= (int)p.cls[0].fw.div;
          return launch_f<FWD, FN, EPI, 4, 1, 1, 0, false, false, true>(p, f_assign(p, 1), src, w, bias, dst, mask, st);
        }
        return launch_f<FWD, FN, EPI, 4, 1, 1, 0, false, false, true>(p, f_assign(p, 64), src, w, bias, dst, mask, st);
      }
    }
    return launch_f<FWD, FN, EPI, 4, 1, 1, 4, DYY>(p, f_assign(p, 64), src, w, bias, dst, mask, st, ysrc);
  }
  const FCfg c = kCand[pick];
  const int tiles = f_assign(p, 16 * c.fm * c.wm);
#define CF_F32_CASE(I, FM_, WM_, WK_) \
  case I: return launch_f<FWD, FN, EPI, FM_, WM_, WK_, 0, DYY>(p, tiles, src, w, bias, dst, mask, st, ysrc);
  switch (pick) {
    CF_F32_CASE(0, 4, 1, 1)
    CF_F32_CASE(1, 4, 2, 1)
    CF_F32_CASE(2, 2, 2, 1)
    CF_F32_CASE(3, 4, 1, 4)
    CF_F32_CASE(4, 2, 1, 4)
    CF_F32_CASE(5, 1, 1, 4)
    CF_F32_CASE(6, 1, 1, 8)
    default: return launch_f<FWD, FN, EPI, 2, 1, 8, 0, DYY>(p, tiles, src, w, bias, dst, mask, st, ysrc);
  }
#undef CF_F32_CASE
}

// Column groups per workgroup (FN x 16 output columns): the widest that
// divides the columns unless a narrower one costs less -- narrow groups give
// the small deep layers (a few hundred rows at batch 1) several times more
// workgroups, each with a share of the columns, instead of a few dozen that
// leave most compute units idle.  CF_F32_FN=1|2|4 forces a width.
int f_pick_fn(const ConvShape &s, FParams &p, int fnmax, bool fwd) {
  if (const char *e = getenv("CF_F32_FN")) {
    const int f = atoi(e);
    if ((f == 1 || f == 2 || f == 4) && f <= fnmax && p.dc % (16 * f) == 0) return f;
  }
  int best_fn = fnmax;
  double best = 0.0;
  for (int f = fnmax; f >= 1; f >>= 1) {
    if (p.dc % (16 * f) != 0) continue;
    double c;
    const int pick = f == 4 ? f_pick<4>(s, p, &c, fwd) : f == 2 ? f_pick<2>(s, p, &c, fwd) : f_pick<1>(s, p, &c, fwd);
    if (pick < 0) return fnmax;  // shift mode: the large layers keep the widest groups
    if (f == fnmax || c < best) {
      best = c;
      best_fn = f;
    }
  }
  return best_fn;
}

}  // namespace

bool f32conv_supported(const ConvShape &s, bool fwd) {
  if (s.dtype != DT_F32) return false;
  const int gc = fwd ? s.ci : s.co;  // contracted channels (16 per k-step)
  const int nc = fwd ? s.co : s.ci;  // GEMM columns
  if (gc % 16 != 0) return false;
  if (fwd ? nc % 32 != 0 : nc % 16 != 0) return false;
  if (s.sd * s.sh * s.sw > F_MAX_CLS) return false;
  if (s.kd * s.kh * s.kw > F_MAX_TAPS) return false;
  const long long xin = (long long)s.n * s.d * s.h * s.w * s.ci, zout = (long long)s.n * s.od * s.oh * s.ow * s.co;
  const long long wn = (long long)s.kd * s.kh * s.kw * s.ci * s.co;
  // 32-bit byte offsets (the range check's out-of-range offset lies above them)
  if (xin * 4 >= (1LL << 31) || zout * 4 >= (1LL << 31) || wn * 4 >= (1LL << 31)) return false;
  return true;
}

bool f32conv_pool_supported(const ConvShape &s) {
  // any stride: the bricks are laid over output voxels; 32 output channels per workgroup
  return f32conv_supported(s, true) && s.co % 32 == 0 && s.od >= 2 && s.oh >= 2 && s.ow >= 2;
}

hipError_t launch_conv_fwd_f32(const ConvShape &s, const float *x, const float *w, const float *bias, float alpha,
                               float *out, uint8_t *mask, int epi, hipStream_t st) {
  FParams p{};
  f_tables(s, true, p);
  p.alpha = alpha;
  if (epi == 2) {
    // pooled: bricks of 2 x 2 x 16 voxels; each of the four waves holds all
    // four 16-voxel w segments of the brick and a quarter of the taps
    FClass &C = p.cls[0];
    const int bd = (s.od + 1) / 2, bh = (s.oh + 1) / 2, bw = (s.ow + 15) / 16;
    C.m = s.n * bd * bh * bw;
    C.fw = make_fastdiv(bw);
    C.fh = make_fastdiv(bh);
    C.fd = make_fastdiv(bd);
    p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
    const int tiles = f_assign(p, 1);
    // taps (kernel rows in taps-in-K mode) split eight ways and 16-channel column
    // groups when the bricks alone leave compute units idle (the stride-2 layer
    // at batch 1)
    if ((long long)tiles * (s.co / 32) < 2LL * kNumCUs && f_shift_env() != 1) {
      if (f_tk() && f_tk_ok(s, p)) return launch_f<true, 1, 2, 4, 1, 8, 0, false, true>(p, tiles, x, w, bias, out, mask, st);
      return launch_f<true, 1, 2, 4, 1, 8>(p, tiles, x, w, bias, out, mask, st);
    }
    // taps in K (or shift mode): one wave per brick with every tap (measured on the
    // 16 -> 32 layer at 128^3, shift mode: 177 -> 168 us against four waves with a
    // quarter of the taps each)
    if (f_tk() && f_tk_ok(s, p)) return launch_f<true, 2, 2, 4, 1, 1, 0, false, true>(p, tiles, x, w, bias, out, mask, st);
    if (f_shift_ok(s, p)) return launch_f<true, 2, 2, 4, 1, 1, 4>(p, tiles, x, w, bias, out, mask, st);
    return launch_f<true, 2, 2, 4, 1, 4>(p, tiles, x, w, bias, out, mask, st);
  }
  const int fn = f_pick_fn(s, p, s.co % 64 == 0 ? 4 : 2, true);
  if (epi == 1) {
    if (fn == 4) return launch_lin<true, 4, 1>(s, p, x, w, bias, out, mask, st);
    if (fn == 2) return launch_lin<true, 2, 1>(s, p, x, w, bias, out, mask, st);
    return launch_lin<true, 1, 1>(s, p, x, w, bias, out, mask, st);
  }
  if (fn == 4) return launch_lin<true, 4, 0>(s, p, x, w, nullptr, out, nullptr, st);
  if (fn == 2) return launch_lin<true, 2, 0>(s, p, x, w, nullptr, out, nullptr, st);
  return launch_lin<true, 1, 0>(s, p, x, w, nullptr, out, nullptr, st);
}

namespace {

// ---------------------------------------------------------------------------
// Backward of an unpooled fused layer in one launch, dz = dy * slope(y) formed
// inside both products: the weight-gradient workgroups (its grid gx x gy x
// nsplit, flattened, first) and the backward-data workgroups (tiles x column
// groups, from an offset rounded up to a multiple of 8 so that their XCD-major
// tile order keeps its XCDs) share one grid.  The stack's deep layers run
// both kernels with a few hundred latency-bound workgroups each; side by side
// they share the machine that either leaves mostly idle, with no second queue
// to synchronise.  One tile shape per side is instantiated: the one the
// launch planners pick for the deep layers (backward-data 16-row tiles, one
// 16-column group, K split over 8 waves; weight gradient one 64-channel row
// unit per wave), the weight gradient with two column groups.
// ---------------------------------------------------------------------------
// The tile shapes instantiated: the deep layers' (dy, y) form (backward-data
// kCand[6] = 16-row tiles, one 16-column group, K split over 8 waves; weight
// gradient one 64-channel row unit per wave, two column groups instead of the
// planned four, so that the kernel stays within 128 registers and two
// 8-wave workgroups fit per compute unit) and the stride-2 layer's plain form
// on a stored dz (backward-data kCand[3] = 64-row tiles, two column groups, K
// over 4 waves, 142 registers alone; weight gradient 16-channel row units on
// 4 waves, four column groups: three 4-wave workgroups per compute unit).
// A launch keeps the weight gradient's planned slices, so every partial is
// the one its plain launch writes, bit for bit.
static_assert(kCand[6].fm == 1 && kCand[6].wm == 1 && kCand[6].wk == 8, "deep-layer pair tile");
static_assert(kCand[3].fm == 4 && kCand[3].wm == 1 && kCand[3].wk == 4, "stride-2 pair tile");

template <int GM, bool WKW4, int WV, int WFN, int DFN, int DFM, int DWM, int DWK, bool DYY, int MINW>
__global__ __launch_bounds__(64 * WV, MINW) void bwd_pair_f32_kernel(
    const float *__restrict__ x, const float *__restrict__ dy, const float *__restrict__ y,
    const float *__restrict__ w, float *__restrict__ dx, float *__restrict__ part_w, float *__restrict__ part_b,
    const FParams fp, const WF32Params wp, int wgx, int wgy, int nw, int dbase, int dtiles) {
  static_assert(WV == DWM * DWK, "one block size for both products");
  const int b = blockIdx.x;
  if (b < nw) {
    const int t = b / wgx;
    wgrad_f32_body<GM, WKW4, 1, WFN, WV, 2>(x, dy, y, part_w, part_b, nullptr, wp, b - t * wgx, t % wgy, t / wgy);
  } else if (b >= dbase) {
    const int j = b - dbase;
    conv_f32_body<false, DFM, DFN, DWM, DWK, 2, 0, 0, DYY>(dy, y, w, nullptr, dx, nullptr, fp, j % dtiles,
                                                            j / dtiles);
  }
}

// CF_F32_PAIR=0 runs the two products as separate launches
bool pair_env() {
  const char *e = getenv("CF_F32_PAIR");
  return !(e && e[0] == '0');
}

}  // namespace

namespace {
// one grid for both products: the weight-gradient workgroups of plan wpl (with
// WV waves and two column groups), then, from an offset rounded up to a multiple
// of 8, the backward-data tiles of plan fp
template <int GM, bool WKW4, int WV, int WFN, int DFN, int DFM, int DWM, int DWK, bool DYY, int MINW>
hipError_t launch_pair(const ConvShape &s, const WPlan &wpl, FParams &fp, const float *x, const float *g,
                       const float *y, const float *w, float alpha, float *dw, float *db, float *dx, void *ws,
                       hipStream_t st) {
  const int dtiles = f_assign(fp, 16 * DFM * DWM);
  const int dcols = fp.dc / (16 * DFN);
  WF32Params wp = f32w_params(s, wpl, alpha);
  wp.g_bytes = (uint32_t)((long long)wp.vox * s.co * 4);
  if (GM == GM_DY_Y) wp.m_bytes = wp.g_bytes;
  const int wgx = (wpl.units + WV - 1) / WV;  // one row unit per wave
  const int wgy = s.co / (16 * WFN);
  const int nw = wgx * wgy * wpl.nsplit;
  const int dbase = (nw + 7) / 8 * 8;
  const long long blocks = (long long)dbase + (long long)dtiles * dcols;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  float *pw = (float *)ws;
  float *pb = GM == GM_DZ ? nullptr : pw + (size_t)wpl.nsplit * wp.m * s.co;
  hipLaunchKernelGGL((bwd_pair_f32_kernel<GM, WKW4, WV, WFN, DFN, DFM, DWM, DWK, DYY, MINW>), dim3((unsigned)blocks),
                     dim3(64 * WV), 0, st, x, g, y, w, dx, pw, pb, fp, wp, wgx, wgy, nw, dbase, dtiles);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_sum_rows(pw, dw, wpl.nsplit, wp.m * s.co, st);
  if (e != hipSuccess || GM == GM_DZ) return e;
  return launch_sum_rows(pb, db, wpl.nsplit, s.co, st);
}

// the backward-data plan, as launch_conv_bwd_data_f32 makes it: column groups
// and the kCand tile (-1 for the shift / output-shift modes)
int dgrad_plan(const ConvShape &s, FParams &fp, float alpha, int *fn) {
  f_tables(s, false, fp);
  fp.alpha = alpha;
  *fn = f_pick_fn(s, fp, s.ci % 64 == 0 ? 4 : (s.ci % 32 == 0 ? 2 : 1), false);
  double cost = 0.0;
  return *fn == 1 ? f_pick<1>(s, fp, &cost, false) : *fn == 2 ? f_pick<2>(s, fp, &cost, false)
                                                              : f_pick<4>(s, fp, &cost, false);
}
}  // namespace

hipError_t launch_conv_bwd_fused_f32(const ConvShape &s, const float *x, const float *dy, const float *y,
                                     const float *w, float alpha, float *dw, float *db, float *dx, void *ws,
                                     hipStream_t st) {
  FParams fp{};
  int fn = 0;
  const int pick = dgrad_plan(s, fp, alpha, &fn);
  const WPlan wpl = f32w_plan(s, GM_DY_Y);
  if (fn == 1 && pick == 6 && !wpl.kw4 && wpl.ru == 1 && wpl.fn >= 2 && s.co % 32 == 0 && pair_env())
    return launch_pair<GM_DY_Y, false, 8, 2, 1, 1, 1, 8, true, 4>(s, wpl, fp, x, dy, y, w, alpha, dw, db, dx, ws, st);
  hipError_t e = launch_conv_bwd_weight_f32(s, x, dy, y, alpha, dw, db, ws, GM_DY_Y, nullptr, st);
  if (e != hipSuccess) return e;
  return launch_conv_bwd_data_f32(s, dy, w, dx, st, y, alpha);
}

hipError_t launch_conv_bwd_f32(const ConvShape &s, const float *x, const float *dz, const float *w, float *dw,
                               float *dx, void *ws, hipStream_t st) {
  FParams fp{};
  int fn = 0;
  const int pick = dgrad_plan(s, fp, 0.f, &fn);
  const WPlan wpl = f32w_plan(s, GM_DZ);
  if (fn == 2 && pick == 3 && wpl.kw4 && wpl.ru == 1 && wpl.fn == 4 && pair_env())
    return launch_pair<GM_DZ, true, 4, 4, 2, 4, 1, 4, false, 3>(s, wpl, fp, x, dz, nullptr, w, 0.f, dw, nullptr, dx, ws,
                                                                st);
  hipError_t e = launch_conv_bwd_weight_f32(s, x, dz, nullptr, 0.f, dw, nullptr, ws, GM_DZ, nullptr, st);
  if (e != hipSuccess) return e;
  return launch_conv_bwd_data_f32(s, dz, w, dx, st, nullptr, 0.f);
}

hipError_t launch_conv_bwd_data_f32(const ConvShape &s, const float *dz, const float *w, float *dx, hipStream_t st,
                                    const float *y, float alpha) {
  FParams p{};
  f_tables(s, false, p);
  p.alpha = alpha;
  const int fn = f_pick_fn(s, p, s.ci % 64 == 0 ? 4 : (s.ci % 32 == 0 ? 2 : 1), false);
  if (y) {
    if (fn == 4) return launch_lin<false, 4, 0, true>(s, p, dz, w, nullptr, dx, nullptr, st, y);
    if (fn == 2) return launch_lin<false, 2, 0, true>(s, p, dz, w, nullptr, dx, nullptr, st, y);
    return launch_lin<false, 1, 0, true>(s, p, dz, w, nullptr, dx, nullptr, st, y);
  }
  if (fn == 4) return launch_lin<false, 4, 0>(s, p, dz, w, nullptr, dx, nullptr, st);
  if (fn == 2) return launch_lin<false, 2, 0>(s, p, dz, w, nullptr, dx, nullptr, st);
  return launch_lin<false, 1, 0>(s, p, dz, w, nullptr, dx, nullptr, st);
}

}  // namespace cf
