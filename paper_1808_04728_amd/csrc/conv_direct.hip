// conv_direct.hip -- implicit-GEMM 3D convolution (forward and backward-data)
// for the deep layers of the stack: 32 or more channels on the contracted
// side, few output voxels (a few thousand GEMM rows at batch 8), bf16.
//
// Forward (Section III-C, Algorithm 1) is the contraction
//   z[o, co] = sum_{t, ci} x~[o*s + t - p, ci] W[t, ci, co]
// and backward-data the adjoint
//   dx[i, ci] = sum_{(o, t): o*s + t - p = i} sum_co dz[o, co] W[t, ci, co],
// split into s^3 parity classes of i (only taps t = (i + p) mod s + s*u reach
// class i; every class is a dense stride-one contraction over ceil(k/s)^3
// taps, no multiply-by-zero work).
//
// Why a second implicit-GEMM kernel: at a few thousand rows, a 128-row
// output tile per workgroup leaves most of the 256 compute units idle and
// every workgroup serialises dozens of load -> LDS -> MFMA stages.  Here:
//  * a workgroup's four waves split the reduction over taps (a wave owns
//    taps w, w+4, ... or w, w+2, ...) and, optionally, the rows, so a 16- to
//    128-row tile still gives every wave its own stream of loads; partial
//    sums meet once, in LDS, at the end;
//  * the im2col operand is never staged: every lane loads its MFMA fragment
//    (8 consecutive channels of one gathered voxel, 16 bytes of NDHWC)
//    straight into registers, PF k-steps ahead of the MFMAs;
//  * forward weights W[t][ci][co] have the output channel contiguous, but the
//    MFMA B operand wants 8 consecutive input channels per lane: each wave
//    copies its 32 x 64 weight slice into a private LDS buffer (swizzled
//    against bank conflicts) and reads it back with the gfx950 transposing
//    read ds_read_b64_tr_b16; backward-data weights are already K-contiguous
//    (co fastest) and are loaded straight into registers;
//  * index arithmetic is kept off the critical path: the host tabulates every
//    class (row counts, launch-time divisors for the row decode, coordinate
//    bases) and every tap (source and weight offsets) in the kernel
//    arguments; loads are 32-bit-offset buffer loads whose hardware range
//    check returns zero for an offset beyond the buffer, which is how padding
//    voxels read as zero without a branch or a select;
//  * the epilogue sums the waves' partial tiles in LDS and writes whole
//    16-byte vectors of the destination (optionally bias + leaky ReLU and
//    the slope mask, the fused forward of an unpooled layer).
//
// v_mfma_f32_16x16x32_bf16 lane layout: A lane l holds row l%16 and K
// 8*(l/16)..+7; B lane l holds column l%16, same K; D lane l holds column
// l%16 and rows 4*(l/16)..+3.

#include "cf_common.h"
#include "cf_kernels.h"
#include "fastdiv.h"

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>

namespace cf {
namespace {

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;
// plain 16-byte vector (a HIP uint4 is a struct, and its copies between
// address spaces stay memcpys through private memory)
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

constexpr int DIR_MAX_CLS = 8;
constexpr int DIR_MAX_TAPS = 64;
constexpr uint32_t DIR_OOB = 0x80000000u;  // a byte offset past every buffer: the load returns zeros

struct DirClass {
  int m;                // GEMM rows (destination voxels) of the class
  int slot0, per;       // XCD-major grid: the class's row tiles are split into 8 contiguous
                        // runs of `per`, one per XCD, at per-XCD slots slot0 .. slot0 + per - 1
  int ntap, tap0;       // the class's taps: entries tap0 .. tap0 + ntap - 1 of the tap table
  FastDiv fw, fh, fd;   // row = ((n * Jd + jd) * Jh + jh) * Jw + jw: divisors Jw, Jh, Jd
  int bq_d, bq_h, bq_w; // source base coordinate = j * bstr + bq
  int or_d, or_h, or_w; // destination coordinate = j * ostr + or
};

struct DirTap {
  int a_off;            // element offset of the tap's source voxel from the row's base voxel
  int w_off;            // element offset of W[tap][0][0]
  int dd, dh, dw;       // source coordinate offsets (bounds check)
};

struct DirParams {
  int sd_, sh_, sw_, sc;        // gathered tensor extent and channels (x forward, dz backward)
  int dd, dh, dw, dc;           // destination extent and channels (z forward, dx backward; GEMM N)
  int bstr_d, bstr_h, bstr_w;   // source base stride per row coordinate
  int ostr_d, ostr_h, ostr_w;   // destination stride per row coordinate
  int wco;                      // weight row pitch (output channels)
  int src_bytes, w_bytes;       // extents of the range-checked buffers
  int ncls;
  float alpha;
  int aux_bytes;                // fused backward-data: extent of the slope mask or of y
  int pod, poh, pow_;           // fused backward-data from a pooled gradient: pooled extents
  DirClass cls[DIR_MAX_CLS];
  DirTap tap[DIR_MAX_TAPS];
};

// swizzled byte offset of (row, 32-byte chunk) in a wave's 32 x 64 bf16 weight
// slice: rows are 128 B, the chunk index is XORed with bits 1 and 3 of the row
// so that the eight rows a transposing read touches per half-wave land in
// distinct banks
__device__ __forceinline__ int wslice_off(int row, int chunk) {
  const int h = ((row >> 1) & 1) | (((row >> 3) & 1) << 1);
  return row * 128 + ((chunk ^ h) << 5);
}

__device__ __forceinline__ u32x4_t buf_load(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0);
}

// GM (backward-data only): the gathered operand is dz itself (GRAD_DZ), or dz
// made of the pooled-output gradient (src) and the slope mask (aux), GRAD_POOL,
// or of dy (src) and the activation y (aux), GRAD_DYY -- the backward-data of a
// fused layer, dz never stored.  The fused forms run the split form of dz: the
// loaded gradient and its masked copy feed two accumulator sets, scaled and
// added once in the epilogue (a mask AND per element instead of a multiply and
// a rounding).
template <bool FWD, int FM, int FN, int WM, int WK, int PF, bool ACT, int GM = GRAD_DZ>
__global__ __launch_bounds__(256) void conv_direct_kernel(const uint16_t *__restrict__ src,
                                                          const uint16_t *__restrict__ wt,
                                                          const float *__restrict__ bias,
                                                          uint16_t *__restrict__ dst, uint8_t *__restrict__ mask,
                                                          const void *__restrict__ aux, const DirParams p) {
  constexpr int BM = 16 * FM * WM, BN = 16 * FN;
  static_assert(WM * WK == 4, "four waves");
  static_assert(!FWD || FN == 4, "forward weight slices are 64 output channels wide");
  static_assert(!FWD || GM == GRAD_DZ, "the fused gathers are backward-data forms");
  constexpr int WSLICE = 32 * 64 * 2;                     // bytes of one staged weight slice
  constexpr int STAGE_BYTES = FWD ? 4 * 2 * WSLICE : 0;   // per wave, double buffered
  constexpr int RED_LD = BN + 4;                          // fp32 row pitch of the reduction tile
  constexpr int RED_BYTES = WK * BM * RED_LD * 4;
  constexpr int SMEM = STAGE_BYTES > RED_BYTES ? STAGE_BYTES : RED_BYTES;
  constexpr int NW = FWD ? 4 : FN;                        // 16-byte weight loads per lane per k-step
  __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave % WM, wk = wave / WM;
  const int g4 = lane >> 4, r16 = lane & 15;

  // ---- class and row tile of this workgroup (uniform) -----------------------
  // workgroup b runs on XCD b % 8; XCD x takes run x of every class, so its
  // tiles cover one contiguous range of voxels (a share of the batch) and
  // their overlapping source reads meet in that XCD's L2
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  int c = 0;
  while (c + 1 < p.ncls && slot >= p.cls[c + 1].slot0) ++c;
  const DirClass &C = p.cls[c];
  const int m0 = (xcd * C.per + slot - C.slot0) * BM;
  if (m0 >= C.m) return;  // uniform: the whole workgroup leaves
  const int n0 = blockIdx.y * BN;

  const __amdgpu_buffer_rsrc_t srsrc = __builtin_amdgcn_make_buffer_rsrc((void *)src, (short)0, p.src_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wrsrc = __builtin_amdgcn_make_buffer_rsrc((void *)wt, (short)0, p.w_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t arsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)aux, (short)0, GM != GRAD_DZ ? p.aux_bytes : 0, 0x00020000);
  (void)arsrc;

  // ---- rows of this lane's A fragments ---------------------------------------
  int rbd[FM], rbh[FM], rbw[FM], roff[FM], rpn[FM];
  bool rok[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int row = m0 + wm * 16 * FM + 16 * i + r16;
    rok[i] = row < C.m;
    const int rr = rok[i] ? row : 0;
    const int t1 = fdiv(rr, C.fw), t2 = fdiv(t1, C.fh), n = fdiv(t2, C.fd);
    rbw[i] = (rr - t1 * (int)C.fw.div) * p.bstr_w + C.bq_w;
    rbh[i] = (t1 - t2 * (int)C.fh.div) * p.bstr_h + C.bq_h;
    rbd[i] = (t2 - n * (int)C.fd.div) * p.bstr_d + C.bq_d;
    roff[i] = (((n * p.sd_ + rbd[i]) * p.sh_ + rbh[i]) * p.sw_ + rbw[i]) * p.sc + 8 * g4;
    rpn[i] = n * p.pod;
  }
  (void)rpn;

  // ---- this wave's k-steps: taps wk, wk + WK, ... of the class; 32 channels each
  const int nch = p.sc >> 5;
  const int mytaps = C.ntap > wk ? (C.ntap - wk + WK - 1) / WK : 0;
  const int nsteps = mytaps * nch;
  int ti = wk, cc = 0, ldstep = 0;  // load cursor: tap, channel chunk, step
  auto next = [&]() {
    if (ldstep + 1 < nsteps) {
      ++ldstep;
      if (++cc == nch) {
        cc = 0;
        ti += WK;
      }
    }
  };

  // lane parts of the weight byte offsets
  int wl[NW];
#pragma unroll
  for (int v = 0; v < NW; ++v) {
    if constexpr (FWD) {
      const int q = lane + 64 * v;  // 16-byte vector q of the 32 x 64 slice: row q/8, columns 8 (q%8) ..
      wl[v] = ((q >> 3) * p.wco + n0 + 8 * (q & 7)) * 2;
    } else {
      wl[v] = ((n0 + 16 * v + r16) * p.wco + 8 * g4) * 2;  // column ci, K = 8 output channels
    }
  }

  // Register ring of NS = PF + 1 slots: the loads of step s + PF are issued
  // (into the slot step s - 1 used) before the MFMAs of step s.
  constexpr int NS = PF + 1;
  u32x4_t a_r[NS][FM], w_r[NS][NW], x_r[NS][FM];
  auto load = [&](u32x4_t(&a)[FM], u32x4_t(&wv)[NW], u32x4_t(&xa)[FM]) {
    const DirTap &T = p.tap[C.tap0 + ti];
    const int cofs = cc * 32;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int vd = rbd[i] + T.dd, vh = rbh[i] + T.dh, vw = rbw[i] + T.dw;
      const bool ok = rok[i] && (unsigned)vd < (unsigned)p.sd_ && (unsigned)vh < (unsigned)p.sh_ &&
                      (unsigned)vw < (unsigned)p.sw_;
      const uint32_t eoff = (uint32_t)(roff[i] + T.a_off + cofs);  // element offset in dz
      if constexpr (GM == GRAD_POOL) {
        // dz voxels outside complete pooling windows have a zero gradient
        const bool inp = ok && vd < 2 * p.pod && vh < 2 * p.poh && vw < 2 * p.pow_;
        const int pv = ((rpn[i] + (vd >> 1)) * p.poh + (vh >> 1)) * p.pow_ + (vw >> 1);
        a[i] = buf_load(srsrc, inp ? (uint32_t)(pv * p.sc + 8 * g4 + cofs) * 2u : DIR_OOB);
        xa[i][0] = __builtin_amdgcn_raw_buffer_load_b8(arsrc, ok ? eoff >> 3 : DIR_OOB, 0, 0);
      } else {
        a[i] = buf_load(srsrc, ok ? eoff * 2u : DIR_OOB);
        if constexpr (GM == GRAD_DYY) xa[i] = buf_load(arsrc, ok ? eoff * 2u : DIR_OOB);
      }
    }
    const int wbase = (T.w_off + cofs * (FWD ? p.wco : 1)) * 2;
#pragma unroll
    for (int v = 0; v < NW; ++v) wv[v] = buf_load(wrsrc, (uint32_t)(wl[v] + wbase));
  };

  unsigned char *wbuf = smem + wave * 2 * WSLICE;
  // LDS byte offsets of this lane's four 16-byte weight vectors in a slice
  int wst[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int q = lane + 64 * v;
    wst[v] = wslice_off(q >> 3, (q & 7) >> 1) + (q & 1) * 16;
  }
  auto stage_w = [&](const u32x4_t(&wv)[NW], int buf) {
#pragma unroll
    for (int v = 0; v < 4; ++v) *reinterpret_cast<u32x4_t *>(wbuf + buf * WSLICE + wst[v]) = wv[v];
  };

  constexpr bool SPLIT = GM != GRAD_DZ;
  f32x4_t acc[FM][FN], acc2[SPLIT ? FM : 1][FN];  // acc2: the masked copy (split form)
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < (SPLIT ? FM : 1); ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc2[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Branch-free steady state (a conditional load would make the compiler wait
  // for every load in flight at the merge): the step count is padded to a
  // multiple of the ring size, the load cursor stops at the last real step
  // (re-loading valid addresses), and padded steps multiply a zero A fragment.
  if (nsteps > 0) {
    const int niter = (nsteps + NS - 1) / NS * NS;
#pragma unroll
    for (int q = 0; q < PF; ++q) {
      load(a_r[q], w_r[q], x_r[q]);
      next();
    }
    if constexpr (FWD) stage_w(w_r[0], 0);
    for (int s0 = 0; s0 < niter; s0 += NS) {
#pragma unroll
      for (int q = 0; q < NS; ++q) {
        const int s = s0 + q;
        load(a_r[(q + PF) % NS], w_r[(q + PF) % NS], x_r[(q + PF) % NS]);
        next();
        bf16x8_t bf[FN];
        if constexpr (FWD) {
          const unsigned char *rb = wbuf + (s & 1) * WSLICE;
#pragma unroll
          for (int j = 0; j < FN; ++j) {
            const int row = 8 * g4 + (r16 >> 2);
            const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_v4i16_t *)(rb + wslice_off(row, j) + (r16 & 3) * 8));
            const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_v4i16_t *)(rb + wslice_off(row + 4, j) + (r16 & 3) * 8));
            typedef short v8i16_t __attribute__((ext_vector_type(8)));
            const v8i16_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            bf[j] = __builtin_bit_cast(bf16x8_t, v);
          }
        } else {
#pragma unroll
          for (int j = 0; j < FN; ++j) bf[j] = __builtin_bit_cast(bf16x8_t, w_r[q][j]);
        }
        const bool real = s < nsteps;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          const u32x4_t av = real ? a_r[q][i] : u32x4_t{0u, 0u, 0u, 0u};
          const bf16x8_t af = __builtin_bit_cast(bf16x8_t, av);
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bf[j], acc[i][j], 0, 0, 0);
          if constexpr (SPLIT) {
            const u32x4_t sel = GM == GRAD_POOL ? sel_of_bits8(x_r[q][i][0]) : sel_of_pos8(x_r[q][i]);
            const bf16x8_t am = __builtin_bit_cast(bf16x8_t, av & sel);
#pragma unroll
            for (int j = 0; j < FN; ++j)
              acc2[i % (SPLIT ? FM : 1)][j] =
                  __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, bf[j], acc2[i % (SPLIT ? FM : 1)][j], 0, 0, 0);
          }
        }
        if constexpr (FWD) stage_w(w_r[(q + 1) % NS], (s + 1) & 1);
      }
    }
  }

  if constexpr (SPLIT) {  // dz x W = s1 (src x W) + s2 ((src & sel) x W)
    const float s1 = GM == GRAD_POOL ? 0.125f * p.alpha : p.alpha;
    const float s2 = GM == GRAD_POOL ? 0.125f * (1.f - p.alpha) : 1.f - p.alpha;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[i][j][e] = s1 * acc[i][j][e] + s2 * acc2[i % (SPLIT ? FM : 1)][j][e];
  }

  // ---- partial tiles meet in LDS ---------------------------------------------
  __syncthreads();  // every wave is done with its weight slices
  float *red = reinterpret_cast<float *>(smem);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        red[(wk * BM + wm * 16 * FM + 16 * i + 4 * g4 + e) * RED_LD + 16 * j + r16] = acc[i][j][e];
  __syncthreads();

  constexpr int CV = BN / 8;  // 16-byte output vectors per row
  for (int v = threadIdx.x; v < BM * CV; v += 256) {
    const int row = v / CV, c8 = v % CV;
    const int grow = m0 + row;
    if (grow >= C.m) continue;
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
    const int t1 = fdiv(grow, C.fw), t2 = fdiv(t1, C.fh), n = fdiv(t2, C.fd);
    const int ow_ = (grow - t1 * (int)C.fw.div) * p.ostr_w + C.or_w;
    const int oh_ = (t1 - t2 * (int)C.fh.div) * p.ostr_h + C.or_h;
    const int od_ = (t2 - n * (int)C.fd.div) * p.ostr_d + C.or_d;
    const int e0 = (((n * p.dd + od_) * p.dh + oh_) * p.dw + ow_) * p.dc + n0 + 8 * c8;
    uint32_t bits = 0;
    if constexpr (ACT) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float u = o[e] + bias[n0 + 8 * c8 + e];
        bits |= (u > 0.f ? 1u : 0u) << e;
        o[e] = u > 0.f ? u : p.alpha * u;
      }
    }
    Vec16<DT_BF16> pk;
#pragma unroll
    for (int e = 0; e < 8; ++e) pk.e[e] = f2bf(o[e]);
    *reinterpret_cast<uint4 *>(dst + e0) = pk.u;
    if (ACT && mask) mask[e0 >> 3] = (uint8_t)bits;
  }
}

// ---------------------------------------------------------------------------
// LDS-staged variant for launches with many row tiles (the stride-2 layer and
// its backward-data classes at batch 8).  Same contraction, class and tap
// tables as above, different data movement:
//  * a workgroup's four waves split the rows (BM = 64 FM rows, 16 FM per
//    wave) and share every k-step's operands, which arrive by buffer -> LDS
//    DMA: the A tile (BM gathered voxels x 32 channels, padding voxels read as
//    zero through the range check) and the B tile (32 x BN weights);
//  * NS stages (4 or 8) of KS k-steps each (KS = 2: half the barriers and
//    per-step overhead per MFMA), each stage its own LDS array, visited in an
//    unrolled ring: the loads of stages s + 1 .. s + NS - 1 are in flight
//    while stage s runs, one barrier per stage; the fragments of stage s + 1
//    are read while the MFMAs of stage s run.  Distinct arrays and a compile-time stage per unrolled step let
//    the compiler see that a stage's reads do not alias the other stages'
//    DMA, so the only wait is the explicit one on this step's loads; the
//    barrier is a bare s_barrier because a release fence would wait for all
//    of them;
//  * the DMA writes each lane's 16 bytes at a fixed LDS slot, so the bank
//    swizzles are applied on the global side: lane slot (row, chunk) fetches
//    logical channel chunk chunk ^ ((row >> 2) & 3) (A, and backward-data's
//    [ci][co] B tile), which makes the fragment reads (16 consecutive rows,
//    one chunk) conflict-free; forward B tiles use the weight-slice swizzle
//    and transposing reads of the kernel above;
//  * the class's tap fields sit one tap per lane (at most 64 taps) and reach
//    the scalar unit by readlane: no memory access or division per k-step;
//  * no split over taps, so the epilogue needs no cross-wave sum: each wave
//    passes its own fp32 rows through its own stage array to leave as whole
//    16-byte vectors.
template <int N>
struct StageIx {
  static constexpr int v = N;
};

// f(StageIx<I>), ..., f(StageIx<N - 1>) in order, as straight-line code
template <int I, int N, class F>
__device__ __forceinline__ void for_stages(F &&f) {
  if constexpr (I < N) {
    f(StageIx<I>{});
    for_stages<I + 1, N>(f);
  }
}

// POOL (forward with ACT): the bias + leaky ReLU + slope mask epilogue is
// followed by the 2^3 average pool; a tile's rows are then a brick of
// 2 (d) x 2 (h) x 16 FM (w) output voxels (wave w holds the w line of (d, h)
// pair w), so every pooling window lies inside one tile, and the tile writes
// only the pooled output and the mask.
//
// GM = GRAD_POOL (backward-data of a pooled fused layer): the A tile is the
// pooled-output gradient, each slot's 16 bytes DMA'd from the pooled voxel of
// its gathered dz voxel, and every row's 32 mask bits of the k-step arrive by
// a 4-byte DMA into a mask area of the stage; the fragments run the split form
// of dz (the gradient and its masked copy into two accumulator sets).
template <bool FWD, int FM, int FN, bool ACT, int NS, int KS, bool POOL = false, int GM = GRAD_DZ>
__global__ __launch_bounds__(256) void conv_lds_kernel(const uint16_t *__restrict__ src,
                                                       const uint16_t *__restrict__ wt,
                                                       const float *__restrict__ bias,
                                                       uint16_t *__restrict__ dst, uint8_t *__restrict__ mask,
                                                       const void *__restrict__ aux, const DirParams p) {
  constexpr int BM = 64 * FM, BN = 16 * FN;
  constexpr int A_SLOTS = BM * 4;                     // 16-byte slots of the A tile
  constexpr int B_SLOTS = 32 * BN / 8;                // 16-byte slots of the B tile
  constexpr int A_BYTES = A_SLOTS * 16, B_BYTES = B_SLOTS * 16;
  constexpr bool MSK = GM == GRAD_POOL;                // mask words staged with the A tile
  constexpr int M_BYTES = MSK ? 1024 : 0;             // one 4-byte slot per thread
  constexpr int STAGE = A_BYTES + B_BYTES + M_BYTES;  // one k-step's tiles; KS of them per stage
  constexpr int NA = A_SLOTS / 256;                   // A DMA instructions per wave and step
  constexpr int NB = (B_SLOTS + 255) / 256;           // B DMA instructions per wave and step
  constexpr int NMK = MSK ? 1 : 0;                    // mask DMA instructions per wave and step
  constexpr int RED_LD = BN + 4;
  static_assert(A_SLOTS % 256 == 0, "whole DMA instructions");
  static_assert(!FWD || FN == 4, "forward weight tiles are 64 output channels wide");
  static_assert(16 * FM * RED_LD * 4 <= STAGE, "a wave's fp32 rows fit its stage array");
  static_assert(NS == 4 || NS == 8, "four or eight stages");
  static_assert(KS == 1 || KS == 2, "one or two k-steps per stage");
  static_assert(NS * KS <= 8, "at most eight k-step arrays");
  static_assert(!POOL || (FWD && ACT), "the pooled epilogue follows the forward activation");
  static_assert(GM == GRAD_DZ || GM == GRAD_POOL, "dz or the pooled gradient and mask");
  static_assert(!MSK || !FWD, "the pooled-gradient gather is a backward-data form");
  constexpr int TWB = 16 * FM;  // brick: w extent of a tile
  // k-step u of stage S lives in array S + NS u: every array is written by
  // one DMA pattern, so the compiler matches each fragment read to its DMA
  __shared__ __attribute__((aligned(16))) unsigned char stg0[STAGE], stg1[STAGE], stg2[STAGE], stg3[STAGE];
  __shared__ __attribute__((aligned(16))) unsigned char stg4[NS * KS > 4 ? STAGE : 16], stg5[NS * KS > 4 ? STAGE : 16];
  __shared__ __attribute__((aligned(16))) unsigned char stg6[NS * KS > 4 ? STAGE : 16], stg7[NS * KS > 4 ? STAGE : 16];
  typedef __attribute__((address_space(3))) void lds_void_t;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g4 = lane >> 4, r16 = lane & 15;

  // workgroup b runs on XCD b % 8; XCD x takes run x of every class, so its
  // tiles cover one contiguous range of voxels (a share of the batch) and
  // their overlapping source reads meet in that XCD's L2
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  int c = 0;
  while (c + 1 < p.ncls && slot >= p.cls[c + 1].slot0) ++c;
  const DirClass &C = p.cls[c];
  const int tile = xcd * C.per + slot - C.slot0;
  int tb_n = 0, tb_d = 0, tb_h = 0, tb_w = 0;  // brick: sample, d pair, h pair, w segment
  if constexpr (POOL) {
    if (tile >= C.m) return;  // C.m counts bricks
    const int t1 = fdiv(tile, C.fw), t2 = fdiv(t1, C.fh);
    tb_n = fdiv(t2, C.fd);
    tb_w = tile - t1 * (int)C.fw.div;
    tb_h = t1 - t2 * (int)C.fh.div;
    tb_d = t2 - tb_n * (int)C.fd.div;
  } else {
    if (tile * BM >= C.m) return;
  }
  const int m0 = tile * BM;
  const int n0 = blockIdx.y * BN;

  const __amdgpu_buffer_rsrc_t srsrc = __builtin_amdgcn_make_buffer_rsrc((void *)src, (short)0, p.src_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wrsrc = __builtin_amdgcn_make_buffer_rsrc((void *)wt, (short)0, p.w_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t mrsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)aux, (short)0, MSK ? p.aux_bytes : 0, 0x00020000);
  (void)mrsrc;

  // output voxel of tile row lrow (false: past the extents or the class)
  auto row_voxel = [&](int lrow, int &n, int &jd, int &jh, int &jw) -> bool {
    if constexpr (POOL) {
      const int dh2 = lrow / TWB;
      n = tb_n;
      jd = 2 * tb_d + (dh2 >> 1);
      jh = 2 * tb_h + (dh2 & 1);
      jw = tb_w * TWB + lrow % TWB;
      return jd < p.dd && jh < p.dh && jw < p.dw;
    } else {
      const int grow = m0 + lrow;
      const int rr = grow < C.m ? grow : 0;
      const int t1 = fdiv(rr, C.fw), t2 = fdiv(t1, C.fh);
      n = fdiv(t2, C.fd);
      jw = rr - t1 * (int)C.fw.div;
      jh = t1 - t2 * (int)C.fh.div;
      jd = t2 - n * (int)C.fd.div;
      return grow < C.m;
    }
  };

  // ---- the class's taps, one per lane -----------------------------------------
  const int ntap = C.ntap;
  int v_aoff = 0, v_woff = 0, v_dd = 0, v_dh = 0, v_dw = 0;
  if (lane < ntap) {
    const DirTap &T = p.tap[C.tap0 + lane];
    v_aoff = T.a_off; v_woff = T.w_off; v_dd = T.dd; v_dh = T.dh; v_dw = T.dw;
  }
  const int v_voff = (v_dd * p.sh_ + v_dh) * p.sw_ + v_dw;  // the tap's voxel offset
  (void)v_voff;

  // ---- this lane's A slots: row, swizzled channel chunk, source base --------
  int rbd[NA], rbh[NA], rbw[NA], roff[NA], rpn[NA], rch[NA];
#pragma unroll
  for (int k = 0; k < NA; ++k) {
    const int sl = 256 * k + tid, row = sl >> 2, lch = (sl & 3) ^ ((row >> 2) & 3);
    int n, jd, jh, jw;
    const bool valid = row_voxel(row, n, jd, jh, jw);
    if (!valid) n = jd = jh = jw = 0;
    rbw[k] = jw * p.bstr_w + C.bq_w;
    rbh[k] = jh * p.bstr_h + C.bq_h;
    rbd[k] = jd * p.bstr_d + C.bq_d;
    roff[k] = (((n * p.sd_ + rbd[k]) * p.sh_ + rbh[k]) * p.sw_ + rbw[k]) * p.sc + 8 * lch;
    rpn[k] = n * p.pod;  // pooled gather: the sample's first pooled plane, the slot's channels
    rch[k] = 8 * lch;
    if (!valid) rbd[k] = -(1 << 20);  // rows past the class fail every bounds check
  }
  (void)rpn;
  (void)rch;
  // mask rows: thread tid stages the mask word of tile row tid (threads past
  // the tile's rows load nothing: their row fails the bounds check)
  int mbd = -(1 << 20), mbh = 0, mbw = 0, mvox = 0;
  if (MSK && tid < BM) {
    int n, jd, jh, jw;
    if (row_voxel(tid, n, jd, jh, jw)) {
      mbw = jw * p.bstr_w + C.bq_w;
      mbh = jh * p.bstr_h + C.bq_h;
      mbd = jd * p.bstr_d + C.bq_d;
      mvox = ((n * p.sd_ + mbd) * p.sh_ + mbh) * p.sw_ + mbw;
    }
  }
  (void)mbd; (void)mbh; (void)mbw; (void)mvox;
  // this lane's B slot(s): element offset inside a step's weight tile
  int boff[NB];
#pragma unroll
  for (int k = 0; k < NB; ++k) {
    const int sl = (256 * k + tid) % B_SLOTS;  // narrow tiles: the spare waves repeat a slot
    if constexpr (FWD) {
      // [32 ci rows][64 co]: 16-byte slot j of row ci sits in 32-byte chunk j/2, which
      // holds logical chunk (j/2) ^ h(row) (the swizzle of wslice_off)
      const int row = sl >> 3, j = sl & 7;
      const int h = ((row >> 1) & 1) | (((row >> 3) & 1) << 1);
      const int lc = (j >> 1) ^ h;
      boff[k] = row * p.wco + n0 + 16 * lc + 8 * (j & 1);
    } else {
      // [BN ci rows][32 co], chunk swizzle as the A tile
      const int row = sl >> 2, lch = (sl & 3) ^ ((row >> 2) & 3);
      boff[k] = (n0 + row) * p.wco + 8 * lch;
    }
  }

  auto arr = [&](auto ix) -> unsigned char * {
    constexpr int S = decltype(ix)::v;
    if constexpr (S == 0) return stg0;
    else if constexpr (S == 1) return stg1;
    else if constexpr (S == 2) return stg2;
    else if constexpr (S == 3) return stg3;
    else if constexpr (S == 4) return stg4;
    else if constexpr (S == 5) return stg5;
    else if constexpr (S == 6) return stg6;
    else return stg7;
  };

  const int nch = p.sc >> 5;
  const int nsteps = ntap * nch;
  // issue state: tap and channel chunk of the next step to load, and the steps
  // left.  The k-loop runs whole rounds of NS steps (straight-line code, in
  // which the compiler keeps track of which stage each DMA fills); the steps
  // past the end stay on the last tap with every A slot out of range, so they
  // load zeros and add nothing.
  int iti = 0, icc = 0, ileft = 0;
  auto issue_one = [&](unsigned char *stg) {
    const int dd = __builtin_amdgcn_readlane(v_dd, iti), dh = __builtin_amdgcn_readlane(v_dh, iti);
    const int dw = __builtin_amdgcn_readlane(v_dw, iti);
    const int aoff = __builtin_amdgcn_readlane(v_aoff, iti) + 32 * icc;
    const int wbase = __builtin_amdgcn_readlane(v_woff, iti) + 32 * icc * (FWD ? p.wco : 1);
#pragma unroll
    for (int k = 0; k < NA; ++k) {
      const int vd = rbd[k] + dd, vh = rbh[k] + dh, vw = rbw[k] + dw;
      const bool ok = ((unsigned)vd < (unsigned)p.sd_) & ((unsigned)vh < (unsigned)p.sh_) &
                      ((unsigned)vw < (unsigned)p.sw_) & (ileft > 0);
      uint32_t off;
      if constexpr (MSK) {
        // the slot's 8 channels of the pooled gradient at the dz voxel's pooling
        // window (zero outside complete windows)
        const bool inp = ok & (vd < 2 * p.pod) & (vh < 2 * p.poh) & (vw < 2 * p.pow_);
        const int pv = ((rpn[k] + (vd >> 1)) * p.poh + (vh >> 1)) * p.pow_ + (vw >> 1);
        off = inp ? (uint32_t)(pv * p.sc + rch[k] + 32 * icc) * 2u : DIR_OOB;
      } else {
        off = ok ? (uint32_t)(roff[k] + aoff) * 2u : DIR_OOB;
      }
      __builtin_amdgcn_raw_ptr_buffer_load_lds(srsrc, (lds_void_t *)(stg + (256 * k + 64 * wave) * 16), 16, off, 0, 0, 0);
    }
    if constexpr (MSK) {
      const int vd = mbd + dd, vh = mbh + dh, vw = mbw + dw;
      const bool ok = ((unsigned)vd < (unsigned)p.sd_) & ((unsigned)vh < (unsigned)p.sh_) &
                      ((unsigned)vw < (unsigned)p.sw_) & (ileft > 0);
      const int voff = __builtin_amdgcn_readlane(v_voff, iti);
      // bits of (voxel, channels 32 icc .. + 31): one aligned word
      const uint32_t off = ok ? (uint32_t)((mvox + voff) * (p.sc >> 3) + 4 * icc) : DIR_OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(mrsrc, (lds_void_t *)(stg + A_BYTES + B_BYTES + 256 * wave), 4, off,
                                               0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      const int sl0 = (256 * k + 64 * wave) % B_SLOTS;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wrsrc, (lds_void_t *)(stg + A_BYTES + sl0 * 16), 16,
                                               (uint32_t)(wbase + boff[k]) * 2u, 0, 0, 0);
    }
    --ileft;
    if (icc + 1 < nch) {
      ++icc;
    } else if (iti + 1 < ntap) {
      icc = 0;
      ++iti;
    }
  };
  auto issue = [&](auto ix) {
    constexpr int S = decltype(ix)::v;
    for_stages<0, KS>([&](auto u) { issue_one(arr(StageIx<S + NS * decltype(u)::v>{})); });
  };

  f32x4_t acc[FM][FN], acc2[MSK ? FM : 1][FN];  // acc2: the masked copy (split form)
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < (MSK ? FM : 1); ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc2[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // MFMA fragments of k-step u of stage ix (and, pooled gather, the mask words of their rows)
  auto read_frags = [&](auto ix, auto u, bf16x8_t (&af)[FM], bf16x8_t (&bf)[FN], uint32_t (&mw)[FM]) {
    const unsigned char *stg = arr(StageIx<decltype(ix)::v + NS * decltype(u)::v>{});
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wave * 16 * FM + 16 * i + r16;
      af[i] = *reinterpret_cast<const bf16x8_t *>(stg + (row * 4 + (g4 ^ ((row >> 2) & 3))) * 16);
      if constexpr (MSK) mw[i] = *reinterpret_cast<const uint32_t *>(stg + A_BYTES + B_BYTES + row * 4);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      if constexpr (FWD) {
        const unsigned char *rb = stg + A_BYTES;
        const int row = 8 * g4 + (r16 >> 2);
        const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(rb + wslice_off(row, j) + (r16 & 3) * 8));
        const v4i16_t hi =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(rb + wslice_off(row + 4, j) + (r16 & 3) * 8));
        typedef short v8i16_t __attribute__((ext_vector_type(8)));
        const v8i16_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        bf[j] = __builtin_bit_cast(bf16x8_t, v);
      } else {
        const int row = 16 * j + r16;
        bf[j] = *reinterpret_cast<const bf16x8_t *>(stg + A_BYTES + (row * 4 + (g4 ^ ((row >> 2) & 3))) * 16);
      }
    }
  };

  // fragments of the stage about to run (read one stage ahead)
  bf16x8_t af[KS][FM], bf[KS][FN];
  uint32_t mf[KS][FM];

  // stage s (KS k-steps) on array ix, its fragments already in af / bf: wait
  // for this wave's loads of stage s + 1 (those of the next NS - 3 stages may
  // stay in flight) and for its fragment reads of stage s, barrier
  // (everyone's loads of stage s + 1 landed; nobody reads the array of stage
  // s - 1 any more), refill that array with stage s + NS - 1, read the
  // fragments of stage s + 1 while the MFMAs of stage s run
  auto kstep = [&](auto ix) {
    constexpr int S = decltype(ix)::v;
    constexpr int VMC = (NS - 3) * (NA + NB + NMK) * KS;
    __builtin_amdgcn_s_waitcnt(0x0070 | (VMC & 15) | ((VMC >> 4) << 14));  // vmcnt(VMC) lgkmcnt(0)
    asm volatile("s_barrier" ::: "memory");
    issue(StageIx<(S + NS - 1) % NS>{});
    bf16x8_t an[KS][FM], bn[KS][FN];
    uint32_t mn[KS][FM];
    for_stages<0, KS>([&](auto u) {
      read_frags(StageIx<(S + 1) % NS>{}, u, an[decltype(u)::v], bn[decltype(u)::v], mn[decltype(u)::v]);
    });
#pragma unroll
    for (int u = 0; u < KS; ++u)
#pragma unroll
      for (int i = 0; i < FM; ++i) {
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[u][i], bf[u][j], acc[i][j], 0, 0, 0);
        if constexpr (MSK) {
          const u32x4_t sel = sel_of_bits8(mf[u][i] >> (8 * g4));
          const bf16x8_t am = __builtin_bit_cast(bf16x8_t, __builtin_bit_cast(u32x4_t, af[u][i]) & sel);
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc2[i % (MSK ? FM : 1)][j] =
                __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, bf[u][j], acc2[i % (MSK ? FM : 1)][j], 0, 0, 0);
        }
      }
#pragma unroll
    for (int u = 0; u < KS; ++u) {
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        af[u][i] = an[u][i];
        mf[u][i] = mn[u][i];
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) bf[u][j] = bn[u][j];
    }
  };

  if (nsteps > 0) {  // a class without taps leaves zeros
    ileft = nsteps;
    for_stages<0, NS - 1>([&](auto ix) { issue(ix); });
    // stage 0 landed everywhere, its fragments in registers
    constexpr int VMC0 = (NS - 2) * (NA + NB + NMK) * KS;
    __builtin_amdgcn_s_waitcnt(0x0f70 | (VMC0 & 15) | ((VMC0 >> 4) << 14));  // vmcnt(VMC0)
    asm volatile("s_barrier" ::: "memory");
    for_stages<0, KS>([&](auto u) {
      read_frags(StageIx<0>{}, u, af[decltype(u)::v], bf[decltype(u)::v], mf[decltype(u)::v]);
    });
    for (int s = 0; s < nsteps; s += NS * KS) for_stages<0, NS>([&](auto ix) { kstep(ix); });
  }

  if constexpr (MSK) {  // dz x W = alpha/8 (g x W) + (1 - alpha)/8 ((g & sel) x W)
    const float s1 = 0.125f * p.alpha, s2 = 0.125f * (1.f - p.alpha);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[i][j][e] = s1 * acc[i][j][e] + s2 * acc2[i % (MSK ? FM : 1)][j][e];
  }

  // ---- each wave's fp32 rows leave through its stage array as 16-byte vectors
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): the trailing loads have landed
  __syncthreads();                      // and every wave is done with every stage
  float *red = reinterpret_cast<float *>(wave == 0 ? stg0 : wave == 1 ? stg1 : wave == 2 ? stg2 : stg3);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) red[(16 * i + 4 * g4 + e) * RED_LD + 16 * j + r16] = acc[i][j][e];
  constexpr int CV = BN / 8;
#pragma unroll
  for (int v = lane; v < 16 * FM * CV; v += 64) {
    const int row = v / CV, c8 = v % CV;
    int n, od_, oh_, ow_;
    const bool valid = row_voxel(wave * 16 * FM + row, n, od_, oh_, ow_);
    if (!POOL && !valid) continue;
    float o[8];
    const float4 x0 = *reinterpret_cast<const float4 *>(&red[row * RED_LD + 8 * c8]);
    const float4 x1 = *reinterpret_cast<const float4 *>(&red[row * RED_LD + 8 * c8 + 4]);
    o[0] = x0.x; o[1] = x0.y; o[2] = x0.z; o[3] = x0.w;
    o[4] = x1.x; o[5] = x1.y; o[6] = x1.z; o[7] = x1.w;
    od_ = od_ * p.ostr_d + C.or_d;
    oh_ = oh_ * p.ostr_h + C.or_h;
    ow_ = ow_ * p.ostr_w + C.or_w;
    const int e0 = (((n * p.dd + od_) * p.dh + oh_) * p.dw + ow_) * p.dc + n0 + 8 * c8;
    uint32_t bits = 0;
    if constexpr (ACT) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float u = o[e] + bias[n0 + 8 * c8 + e];
        bits |= (u > 0.f ? 1u : 0u) << e;
        o[e] = u > 0.f ? u : p.alpha * u;
      }
    }
    if constexpr (POOL) {
      // y stays in the wave's array for the pooling pass (each (row, chunk) has one owner)
      *reinterpret_cast<float4 *>(&red[row * RED_LD + 8 * c8]) = make_float4(o[0], o[1], o[2], o[3]);
      *reinterpret_cast<float4 *>(&red[row * RED_LD + 8 * c8 + 4]) = make_float4(o[4], o[5], o[6], o[7]);
      if (valid) mask[e0 >> 3] = (uint8_t)bits;
    } else {
      Vec16<DT_BF16> pk;
#pragma unroll
      for (int e = 0; e < 8; ++e) pk.e[e] = f2bf(o[e]);
      *reinterpret_cast<uint4 *>(dst + e0) = pk.u;
      if (ACT && mask) mask[e0 >> 3] = (uint8_t)bits;
    }
  }
  if constexpr (POOL) {
    // ---- 2^3 average pool of the brick: TWB/2 pooled voxels x BN channels;
    // the window's four (d, h) lines are the four waves' arrays
    __syncthreads();
    const float *lines[4] = {reinterpret_cast<const float *>(stg0), reinterpret_cast<const float *>(stg1),
                             reinterpret_cast<const float *>(stg2), reinterpret_cast<const float *>(stg3)};
    for (int it = tid; it < (TWB / 2) * CV; it += 256) {
      const int pw = it / CV, c8 = it % CV;
      const int pwg = tb_w * (TWB / 2) + pw;
      if (tb_d >= p.pod || tb_h >= p.poh || pwg >= p.pow_) continue;
      float sm[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) sm[e] = 0.f;
#pragma unroll
      for (int dh2 = 0; dh2 < 4; ++dh2)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const float *r = lines[dh2] + (2 * pw + t) * RED_LD + 8 * c8;
          const float4 x0 = *reinterpret_cast<const float4 *>(r);
          const float4 x1 = *reinterpret_cast<const float4 *>(r + 4);
          sm[0] += x0.x; sm[1] += x0.y; sm[2] += x0.z; sm[3] += x0.w;
          sm[4] += x1.x; sm[5] += x1.y; sm[6] += x1.z; sm[7] += x1.w;
        }
      const int q0 = (((tb_n * p.pod + tb_d) * p.poh + tb_h) * p.pow_ + pwg) * p.dc + n0 + 8 * c8;
      Vec16<DT_BF16> pk;
#pragma unroll
      for (int e = 0; e < 8; ++e) pk.e[e] = f2bf(sm[e] * 0.125f);
      *reinterpret_cast<uint4 *>(dst + q0) = pk.u;
    }
  }
}

struct DirCfg {
  int fm, wm, wk, pf;
};

template <bool FWD, int FN, int PF, bool ACT, int GM>
hipError_t launch_dir_t(const DirCfg &c, const DirParams &p, int tiles, const void *src, const void *w,
                        const float *bias, void *dst, void *mask, const void *aux, hipStream_t st) {
  dim3 grid((unsigned)tiles, p.dc / (16 * FN), 1);
  if (grid.x == 0 || grid.y == 0) return hipSuccess;  // no destination rows
  const uint16_t *s16 = (const uint16_t *)src, *w16 = (const uint16_t *)w;
  uint16_t *d16 = (uint16_t *)dst;
  uint8_t *m8 = (uint8_t *)mask;
#define CF_DIR_LAUNCH(FM_, WM_, WK_)                                                                               \
  hipLaunchKernelGGL((conv_direct_kernel<FWD, FM_, FN, WM_, WK_, PF, ACT, GM>), grid, dim3(256), 0, st, s16, w16, \
                     bias, d16, m8, aux, p)
  if (c.fm == 4 && c.wm == 2) CF_DIR_LAUNCH(4, 2, 2);
  else if (c.fm == 4 && c.wm == 1) CF_DIR_LAUNCH(4, 1, 4);
  else if (c.fm == 2 && c.wm == 2) CF_DIR_LAUNCH(2, 2, 2);
  else if (c.fm == 2 && c.wm == 1) CF_DIR_LAUNCH(2, 1, 4);
  else CF_DIR_LAUNCH(1, 1, 4);
#undef CF_DIR_LAUNCH
  return hipGetLastError();
}

template <bool FWD, int FN, bool ACT, int GM = GRAD_DZ>
hipError_t launch_dir_pf(const DirCfg &c, const DirParams &p, int tiles, const void *src, const void *w,
                         const float *bias, void *dst, void *mask, hipStream_t st, const void *aux = nullptr) {
  switch (c.pf) {
    case 1: return launch_dir_t<FWD, FN, 1, ACT, GM>(c, p, tiles, src, w, bias, dst, mask, aux, st);
    case 2: return launch_dir_t<FWD, FN, 2, ACT, GM>(c, p, tiles, src, w, bias, dst, mask, aux, st);
    default: return launch_dir_t<FWD, FN, 3, ACT, GM>(c, p, tiles, src, w, bias, dst, mask, aux, st);
  }
}

// Class and tap tables.  Forward: one class, rows = output voxels, source
// base = j*s - p, taps u with source offset +u and weight tap u.  Backward-
// data: class r in [0, s)^3 per dimension: rows j with input coordinate
// j*s + r, first reaching tap t0 = (r + p) mod s, taps t0 + s*u with source
// offset -u from base j + (r + p - t0)/s.
void build_tables(const ConvShape &s, bool fwd, DirParams &p) {
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
    DirClass &C = p.cls[c];
    C.m = s.n * J[0] * J[1] * J[2];
    C.fw = make_fastdiv(std::max(J[2], 1));
    C.fh = make_fastdiv(std::max(J[1], 1));
    C.fd = make_fastdiv(std::max(J[0], 1));
    C.bq_d = Q[0]; C.bq_h = Q[1]; C.bq_w = Q[2];
    C.or_d = r[0]; C.or_h = r[1]; C.or_w = r[2];
    C.tap0 = ntaps;
    C.ntap = U[0] * U[1] * U[2];
    const int sg = fwd ? 1 : -1;
    for (int ud = 0; ud < U[0]; ++ud)
      for (int uh = 0; uh < U[1]; ++uh)
        for (int uw = 0; uw < U[2]; ++uw) {
          DirTap &T = p.tap[ntaps++];
          T.dd = sg * ud; T.dh = sg * uh; T.dw = sg * uw;
          T.a_off = ((T.dd * p.sh_ + T.dh) * p.sw_ + T.dw) * p.sc;
          // weight tap step: 1 forward, the stride between the taps of a class backward
          const int st_d = fwd ? 1 : S[0], st_h = fwd ? 1 : S[1], st_w = fwd ? 1 : S[2];
          const int tap = ((T0[0] + st_d * ud) * s.kh + (T0[1] + st_h * uh)) * s.kw + (T0[2] + st_w * uw);
          T.w_off = tap * s.ci * s.co;
        }
  }
  p.src_bytes = (int)((long long)s.n * p.sd_ * p.sh_ * p.sw_ * p.sc * 2);
  p.w_bytes = s.kd * s.kh * s.kw * s.ci * s.co * 2;
}

// Lays out the XCD-major grid for row tiles of bm rows; returns its size (a
// multiple of 8; workgroups past a class's last tile leave at once).
int assign_tiles(DirParams &p, int bm) {
  int slots = 0;
  for (int c = 0; c < p.ncls; ++c) {
    const int tiles = (p.cls[c].m + bm - 1) / bm;
    p.cls[c].slot0 = slots;
    p.cls[c].per = (tiles + 7) / 8;
    slots += p.cls[c].per;
  }
  return 8 * slots;
}

// Tile choice (measured on the deep layers of the stack): the largest row
// tile that still yields 256 workgroups (one per compute unit); more rows per
// wave amortise the weight stream, waves along K keep every wave busy when
// rows are few.  The 128-row tile pays off only for backward-data, whose
// weights come straight from global memory.  Prefetch: three k-steps for the
// forward kernels (their per-step weight staging leaves load latency exposed
// at these row counts), one for backward-data (bound by L2 -> L1 traffic,
// where a deeper ring only adds registers) -- measured on the stack's layers.
// CF_DIRECT_TILE="fm,wm,wk" and CF_DIRECT_PF force a variant (tests cover
// every one this way).
DirCfg choose_cfg(DirParams &p, int fn, bool fwd) {
  static const DirCfg cand[] = {{4, 2, 2, 1}, {2, 2, 2, 1}, {4, 1, 4, 1}, {2, 1, 4, 1}, {1, 1, 4, 1}};
  int pf = 0;
  if (const char *e = getenv("CF_DIRECT_PF")) pf = atoi(e);
  DirCfg pick = cand[4];
  bool forced = false;
  if (const char *e = getenv("CF_DIRECT_TILE")) {
    int fm = 0, wm = 0, wk = 0;
    if (sscanf(e, "%d,%d,%d", &fm, &wm, &wk) == 3)
      for (const DirCfg &c : cand)
        if (c.fm == fm && c.wm == wm && c.wk == wk) {
          pick = c;
          forced = true;
        }
  }
  if (!forced) {
    const int ny = p.dc / (16 * fn);
    for (int i = fwd ? 1 : 0; i < 5; ++i)
      if ((long long)assign_tiles(p, 16 * cand[i].fm * cand[i].wm) * ny >= 256) {
        pick = cand[i];
        break;
      }
  }
  if (fwd) pick.pf = 3;
  if (pf >= 1 && pf <= 3) pick.pf = pf;
  return pick;
}

}  // namespace

bool direct_supported(const ConvShape &s, bool fwd) {
  if (s.dtype != DT_BF16) return false;
  const int gc = fwd ? s.ci : s.co;  // contracted channels (32 per k-step)
  const int nc = fwd ? s.co : s.ci;  // GEMM columns
  if (gc % 32 != 0 || nc % 32 != 0) return false;
  if (fwd && nc % 64 != 0) return false;
  if (s.sd * s.sh * s.sw > DIR_MAX_CLS) return false;
  // every class's taps fit the table (k <= 4 per dimension gives at most 64)
  if (s.kd * s.kh * s.kw > DIR_MAX_TAPS) return false;
  // 32-bit element offsets and buffer extents
  const long long xin = (long long)s.n * s.d * s.h * s.w * s.ci, zout = (long long)s.n * s.od * s.oh * s.ow * s.co;
  const long long wn = (long long)s.kd * s.kh * s.kw * s.ci * s.co;
  if (xin * 2 >= (1LL << 31) || zout * 2 >= (1LL << 31) || wn * 2 >= (1LL << 31)) return false;
  return true;
}

// LDS-staged kernel when its row tiles alone fill the machine (>= 256
// workgroups), with 128-row tiles if they do, else 64-row tiles; 0 = the
// register-streaming kernel.  CF_DIRECT_KERNEL=reg / lds128 / lds64 forces a
// choice (tests cover every kernel on small shapes this way).
int choose_lds(DirParams &p, int ny) {
  if (const char *e = getenv("CF_DIRECT_KERNEL")) {
    if (!strcmp(e, "reg")) return 0;
    if (!strcmp(e, "lds128")) return 2;
    if (!strcmp(e, "lds64")) return 1;
  }
  if ((long long)assign_tiles(p, 128) * ny >= 256) return 2;
  if ((long long)assign_tiles(p, 64) * ny >= 256) return 1;
  return 0;
}

template <bool FWD, int FN, bool ACT, bool POOL = false, int GM = GRAD_DZ>
hipError_t launch_lds(int fm, DirParams &p, const void *src, const void *w, const float *bias, void *dst,
                      void *mask, hipStream_t st, const void *aux = nullptr) {
  const int tiles = assign_tiles(p, POOL ? 1 : 64 * fm);  // pooled: the class counts bricks
  dim3 grid((unsigned)tiles, p.dc / (16 * FN), 1);
  if (grid.x == 0 || grid.y == 0) return hipSuccess;
  const uint16_t *s16 = (const uint16_t *)src, *w16 = (const uint16_t *)w;
  // four stages (measured on the stack's stride-2 layer: an eight-stage ring
  // gains nothing there, where the waves are issue-bound, and halves the
  // backward-data workgroups per compute unit); CF_DIRECT_STAGES=8 selects
  // the deeper ring (tests cover both)
  const char *e = getenv("CF_DIRECT_STAGES");
  const bool ns4 = !(e && atoi(e) == 8);
  // k-steps per stage (four-stage ring): two forward (measured on the
  // stride-2 layer: 30 -> 26 us), one for backward-data (its classes have few
  // k-steps, and the larger stage halves the workgroups per compute unit);
  // CF_DIRECT_KSUB=1|2 forces either; the eight-stage ring takes one
  int ks = FWD ? 2 : 1;
  if (const char *k = getenv("CF_DIRECT_KSUB")) ks = atoi(k) == 1 ? 1 : 2;
#define CF_LDS_LAUNCH(FM_, NS_, KS_)                                                                             \
  hipLaunchKernelGGL((conv_lds_kernel<FWD, FM_, FN, ACT, NS_, KS_, POOL, GM>), grid, dim3(256), 0, st, s16, w16, \
                     bias, (uint16_t *)dst, (uint8_t *)mask, aux, p)
  if (fm == 2) {
    if (!ns4) CF_LDS_LAUNCH(2, 8, 1);
    else if (ks == 2) CF_LDS_LAUNCH(2, 4, 2);
    else CF_LDS_LAUNCH(2, 4, 1);
  } else {
    if (!ns4) CF_LDS_LAUNCH(1, 8, 1);
    else if (ks == 2) CF_LDS_LAUNCH(1, 4, 2);
    else CF_LDS_LAUNCH(1, 4, 1);
  }
#undef CF_LDS_LAUNCH
  return hipGetLastError();
}

hipError_t launch_conv_fwd_direct(const ConvShape &s, const void *x, const void *w, const float *bias, float alpha,
                                  void *out, void *mask, bool act, hipStream_t st) {
  DirParams p{};
  build_tables(s, true, p);
  p.alpha = alpha;
  if (const int fm = choose_lds(p, p.dc / 64))
    return act ? launch_lds<true, 4, true>(fm, p, x, w, bias, out, mask, st)
               : launch_lds<true, 4, false>(fm, p, x, w, nullptr, out, nullptr, st);
  const DirCfg c = choose_cfg(p, 4, true);
  const int tiles = assign_tiles(p, 16 * c.fm * c.wm);
  return act ? launch_dir_pf<true, 4, true>(c, p, tiles, x, w, bias, out, mask, st)
             : launch_dir_pf<true, 4, false>(c, p, tiles, x, w, nullptr, out, nullptr, st);
}

bool direct_pool_supported(const ConvShape &s) {
  return direct_supported(s, true) && s.od >= 2 && s.oh >= 2 && s.ow >= 2;
}

// Pooled forward: the LDS-staged kernel over bricks of 2 x 2 x 16 FM output
// voxels (32-wide bricks when the rows are wider than 16, else 16-wide).
hipError_t launch_conv_fwd_direct_pool(const ConvShape &s, const void *x, const void *w, const float *bias,
                                       float alpha, void *out, void *mask, hipStream_t st) {
  DirParams p{};
  build_tables(s, true, p);
  p.alpha = alpha;
  p.pod = s.od / 2;
  p.poh = s.oh / 2;
  p.pow_ = s.ow / 2;
  const int fm = s.ow > 16 ? 2 : 1;
  const int jw = (s.ow + 16 * fm - 1) / (16 * fm), jh = (s.oh + 1) / 2, jd = (s.od + 1) / 2;
  DirClass &C = p.cls[0];
  C.m = s.n * jd * jh * jw;
  C.fw = make_fastdiv(jw);
  C.fh = make_fastdiv(jh);
  C.fd = make_fastdiv(jd);
  return launch_lds<true, 4, true, true>(fm, p, x, w, bias, out, mask, st);
}

hipError_t launch_conv_bwd_data_direct(const ConvShape &s, const void *dz, const void *w, void *dx,
                                       hipStream_t st) {
  DirParams p{};
  build_tables(s, false, p);
  const int fn = p.dc % 64 == 0 ? 4 : 2;
  if (const int fm = choose_lds(p, p.dc / (16 * fn)))
    return fn == 4 ? launch_lds<false, 4, false>(fm, p, dz, w, nullptr, dx, nullptr, st)
                   : launch_lds<false, 2, false>(fm, p, dz, w, nullptr, dx, nullptr, st);
  const DirCfg c = choose_cfg(p, fn, false);
  const int tiles = assign_tiles(p, 16 * c.fm * c.wm);
  return fn == 4 ? launch_dir_pf<false, 4, false>(c, p, tiles, dz, w, nullptr, dx, nullptr, st)
                 : launch_dir_pf<false, 2, false>(c, p, tiles, dz, w, nullptr, dx, nullptr, st);
}

template <int GM>
static hipError_t bwd_data_fused_t(const DirCfg &c, const DirParams &p, int tiles, int fn, const void *g,
                                   const void *aux, const void *w, void *dx, hipStream_t st) {
  return fn == 4 ? launch_dir_pf<false, 4, false, GM>(c, p, tiles, g, w, nullptr, dx, nullptr, st, aux)
                 : launch_dir_pf<false, 2, false, GM>(c, p, tiles, g, w, nullptr, dx, nullptr, st, aux);
}

hipError_t launch_conv_bwd_data_direct_fused(const ConvShape &s, const void *g, const void *aux, int gm, float alpha,
                                             const void *w, void *dx, hipStream_t st) {
  DirParams p{};
  build_tables(s, false, p);
  p.alpha = alpha;
  p.pod = s.od / 2;
  p.poh = s.oh / 2;
  p.pow_ = s.ow / 2;
  const long long zel = (long long)s.n * s.od * s.oh * s.ow * s.co;
  if (gm == GRAD_POOL) {
    // the gathered buffer is the pooled gradient; the mask has a bit per dz element
    p.src_bytes = (int)((long long)s.n * p.pod * p.poh * p.pow_ * s.co * 2);
    p.aux_bytes = (int)((zel + 31) / 32 * 4);
  } else {
    p.aux_bytes = (int)(zel * 2);
  }
  const int fn = p.dc % 64 == 0 ? 4 : 2;
  // pooled gradient: the LDS-staged kernel when its row tiles fill the machine
  // (as the plain backward-data); the register kernel otherwise and for (dy, y)
  if (gm == GRAD_POOL)
    if (const int fm = choose_lds(p, p.dc / (16 * fn)))
      return fn == 4 ? launch_lds<false, 4, false, false, GRAD_POOL>(fm, p, g, w, nullptr, dx, nullptr, st, aux)
                     : launch_lds<false, 2, false, false, GRAD_POOL>(fm, p, g, w, nullptr, dx, nullptr, st, aux);
  const DirCfg c = choose_cfg(p, fn, false);
  const int tiles = assign_tiles(p, 16 * c.fm * c.wm);
  return gm == GRAD_POOL ? bwd_data_fused_t<GRAD_POOL>(c, p, tiles, fn, g, aux, w, dx, st)
                         : bwd_data_fused_t<GRAD_DYY>(c, p, tiles, fn, g, aux, w, dx, st);
}

}  // namespace cf
