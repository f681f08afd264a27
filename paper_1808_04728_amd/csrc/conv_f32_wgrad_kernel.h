// conv_f32_wgrad_kernel.h -- the fp32 backward-weights kernel body (gfx950),
// shared by its own launches (conv_f32_wgrad.hip) and by the combined backward
// launch of an unpooled layer (conv_f32.hip), which runs it beside the
// backward-data kernel in one grid.  The operator and the operand layout are
// described at the top of conv_f32_wgrad.hip.

#pragma once

#include "cf_common.h"
#include "cf_kernels.h"
#include "fastdiv.h"

namespace cf {

struct WF32Params {
  int n, d, h, w, ci;          // input
  int od, oh, ow, co;          // conv output
  int sd, sh, sw, pd, ph, pw;  // stride, padding before
  int kh, kw;                  // kernel extents (tap decode)
  int m;                       // kd*kh*kw*ci (GEMM rows)
  int units;                   // row units of 64 rows
  int cunits;                  // channel chunks per unit position (ci/16 or ci/64)
  int vox;                     // n*od*oh*ow (reduction length)
  int rows_per;                // output rows (n, od, oh) per slice
  int nws;                     // steps of four voxels per output row
  FastDiv fh, fd;              // row decode divisors oh, od
  uint32_t x_bytes, g_bytes, m_bytes;
  float alpha;
  int pod, poh, pow_;          // fused: pooled extents
};

// gradient operand of the weight-gradient kernel
enum : int { GM_DZ = 0, GM_POOL_MASK = 1, GM_DY_Y = 3 };

// launch shape of one backward-weights call: row units per wave, column
// groups, grid (gx, gy, nsplit) and the slice length in output rows
struct WPlan {
  bool kw4;
  int ru, fn, wv;
  int units, cunits;
  int gx, gy, nsplit, rows_per;
};
WPlan f32w_plan(const ConvShape &s, int gm);
WF32Params f32w_params(const ConvShape &s, const WPlan &pl, float alpha);

namespace {

__device__ __forceinline__ uint32_t wg_ld32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4_t wg_ld128(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// KW4: units are (kd, kh, 16 channels) of a kernel 4 wide; else (tap, 64 channels).
// GM_DZ: g is dz; GM_POOL_MASK: g is the pooled gradient, aux the slope mask;
// GM_DY_Y: g is dy, aux the activation y.
// The kernel body, run by the workgroup of grid position (bx, by, bz): the
// weight-gradient launch's own grid, or a share of a combined backward launch.
template <int GM, bool KW4, int RU, int FN, int WV, int PF>
__device__ __forceinline__ void wgrad_f32_body(const float *__restrict__ x, const float *__restrict__ g,
                                               const void *__restrict__ aux, float *__restrict__ part_w,
                                               float *__restrict__ part_b, float *__restrict__ dz_out,
                                               const WF32Params p, int bx, int by, int bz) {
  // no contraction of the products into sums: dz and db round the same way in
  // every launch that runs this body
#pragma clang fp contract(off)
  __shared__ float dbs[4][16 * FN];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g4 = lane >> 4, r16 = lane & 15;
  const int co0 = by * 16 * FN;
  const int slice = bz;
  // the bias gradient and the stored dz come from one wave of the slice
  constexpr bool FUSED = GM != GM_DZ;
  const bool lead = FUSED && bx == 0 && wave == 0;

  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc((void *)x, (short)0, p.x_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t gr = __builtin_amdgcn_make_buffer_rsrc((void *)g, (short)0, p.g_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t mr =
      __builtin_amdgcn_make_buffer_rsrc((void *)aux, (short)0, FUSED ? p.m_bytes : 0u, 0x00020000);

  // ---- this wave's row units: the lane's tap and channel, and its dW rows ---
  const int u0 = (bx * WV + wave) * RU;
  int tkd[RU], tkh[RU], tkw[RU], toff[RU], rbase[RU];
  bool uok[RU];
#pragma unroll
  for (int i = 0; i < RU; ++i) {
    const int u = u0 + i;
    uok[i] = u < p.units;
    const int uu = uok[i] ? u : 0;
    const int pos = uu / p.cunits, cc = uu - pos * p.cunits;
    int c0, tap;
    if constexpr (KW4) {
      // pos = kd * kh_extent + kh; this lane's column kw = r16 / 4, channels c0 + 4 (r16 % 4) ..
      tkd[i] = pos / p.kh;
      tkh[i] = pos - tkd[i] * p.kh;
      tkw[i] = r16 >> 2;
      c0 = 16 * cc;
      tap = (tkd[i] * p.kh + tkh[i]) * 4 + tkw[i];
      toff[i] = c0 + 4 * (r16 & 3);  // channel offset; the tap's voxel comes from the row base
      // D row 4 g + e of MFMA j: column kw = g, channel c0 + 4 e + j
      rbase[i] = ((tkd[i] * p.kh + tkh[i]) * 4 + g4) * p.ci + c0;
    } else {
      tap = pos;
      tkw[i] = tap % p.kw;
      tkh[i] = (tap / p.kw) % p.kh;
      tkd[i] = tap / (p.kw * p.kh);
      c0 = 64 * cc;
      toff[i] = c0 + 4 * r16;
      // D row 4 g + e of MFMA j: channel c0 + 16 g + 4 e + j
      rbase[i] = tap * p.ci + c0 + 16 * g4;
    }
    (void)tap;
  }

  // ---- the slice's output rows (n, od, oh), four voxels along w per step -----
  // The load cursor is kept per lane: the output w of the lane's K slot, per
  // unit the w and element offset of its x value, the gradient's offset (and,
  // pooled, its pooled w and the mask word).  It is set at the start of every
  // output row, under a uniform branch marked unlikely, and advanced by
  // additions between: computed per step, the offsets cost about 35 vector
  // instructions (four of them quarter-rate multiplies) per 16 MFMAs, and the
  // vector ALU does not run beside the MFMAs.  Steps past the slice (ring
  // padding) load zeros.
  const int nrow_all = p.n * p.od * p.oh;
  const int r0 = slice * p.rows_per, r1 = min(r0 + p.rows_per, nrow_all);
  const int nsteps = r1 > r0 ? (r1 - r0) * p.nws : 0;
  int crow = r0, cws = 0, ldstep = 0;  // load cursor (uniform)
  int cw = 0, cv = 0, cg = 0, cm = 0, cpw = 0;
  int cxw[RU], cxo[RU];
  bool dok[RU], winrow = false;
  (void)cm;
  (void)cpw;
  // always inlined: called at two sites, an outlined copy would keep the
  // captured per-lane arrays in scratch memory
  auto setrow = [&](int row) __attribute__((always_inline)) {
    const int t1 = fdiv(row, p.fh), nn = fdiv(t1, p.fd);
    const int oh_ = row - t1 * (int)p.fh.div, od_ = t1 - nn * (int)p.fd.div;
    const int bd = od_ * p.sd - p.pd, bh = oh_ * p.sh - p.ph;
    cw = g4;
    const int bw = g4 * p.sw - p.pw;
#pragma unroll
    for (int i = 0; i < RU; ++i) {
      dok[i] = uok[i] & ((unsigned)(bd + tkd[i]) < (unsigned)p.d) & ((unsigned)(bh + tkh[i]) < (unsigned)p.h);
      cxw[i] = bw + tkw[i];
      cxo[i] = (((nn * p.d + bd + tkd[i]) * p.h + bh + tkh[i]) * p.w + cxw[i]) * p.ci + toff[i];
    }
    cv = row * p.ow + g4;
    if constexpr (GM == GM_POOL_MASK) {
      const int pd_ = od_ >> 1, ph_ = oh_ >> 1;
      winrow = (pd_ < p.pod) & (ph_ < p.poh);
      cpw = g4 >> 1;
      cg = (((nn * p.pod + pd_) * p.poh + ph_) * p.pow_ + cpw) * p.co + co0 + r16;
      cm = cv * (p.co >> 5) + (co0 >> 5);
    } else {
      cg = cv * p.co + co0 + r16;
    }
  };
  if (nsteps > 0) setrow(r0);
  // per-step advances: 4 output voxels along w
  const int dxw = 4 * p.sw, dxo = 4 * p.sw * p.ci;
  const int dg = (GM == GM_POOL_MASK ? 2 : 4) * p.co, dm = 4 * (p.co >> 5);
  auto next = [&]() {
    ++ldstep;
    const bool adv = ldstep < nsteps;
    const int c1 = cws + (adv ? 1 : 0);
    const bool wrap = c1 == p.nws;
    cws = wrap ? 0 : c1;
    crow += wrap ? 1 : 0;
    cw += adv ? 4 : 0;
    cv += adv ? 4 : 0;
#pragma unroll
    for (int i = 0; i < RU; ++i) {
      cxw[i] += adv ? dxw : 0;
      cxo[i] += adv ? dxo : 0;
    }
    cg += adv ? dg : 0;
    if constexpr (GM == GM_POOL_MASK) {
      cpw += adv ? 2 : 0;
      cm += adv ? dm : 0;
    }
    if (__builtin_expect(wrap, 0)) setrow(min(crow, nrow_all - 1));
  };

  constexpr int NS = PF + 1;
  u32x4_t a_r[NS][RU];
  float b_r[NS][FN];
  uint32_t m_r[NS];
  float y_r[NS][FN];
  int v_r[NS];  // voxel of the lane's K slot (-1: none), for the stored dz
  (void)m_r;
  (void)y_r;
  (void)v_r;

  auto load = [&](u32x4_t(&a)[RU], float(&b)[FN], uint32_t &mw, float(&yv)[FN], int &vx) {
    const bool wok = (ldstep < nsteps) & (cw < p.ow);
#pragma unroll
    for (int i = 0; i < RU; ++i) {
      // bitwise, not short-circuit: one select per load, no branch
      const bool ok = dok[i] & wok & ((unsigned)cxw[i] < (unsigned)p.w);
      // a valid byte offset is below 2^31: bit 31 sends the load past the buffer (zeros)
      a[i] = wg_ld128(xr, ((uint32_t)cxo[i] * 4u) | ((uint32_t)!ok << 31));
    }
    vx = wok ? cv : -1;
    if constexpr (GM == GM_POOL_MASK) {
      const bool win = winrow & wok & (cpw < p.pow_);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = __uint_as_float(wg_ld32(gr, ((uint32_t)(cg + 16 * j) * 4u) | ((uint32_t)!win << 31)));
      // the workgroup's 32 channels of voxel v are one mask word
      mw = wg_ld32(mr, ((uint32_t)cm * 4u) | ((uint32_t)!wok << 31));
    } else {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const uint32_t off = ((uint32_t)(cg + 16 * j) * 4u) | ((uint32_t)!wok << 31);
        b[j] = __uint_as_float(wg_ld32(gr, off));
        if constexpr (GM == GM_DY_Y) yv[j] = __uint_as_float(wg_ld32(mr, off));  // y: the layout of dy
      }
    }
  };

  f32x4_t acc[RU][4][FN];
#pragma unroll
  for (int i = 0; i < RU; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int k = 0; k < FN; ++k) acc[i][j][k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float dsum[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j) dsum[j] = 0.f;
  const float s1 = 0.125f, sa = 0.125f * p.alpha;

  if (nsteps > 0) {
    const int niter = (nsteps + NS - 1) / NS * NS;
#pragma unroll
    for (int q = 0; q < PF; ++q) {
      load(a_r[q], b_r[q], m_r[q], y_r[q], v_r[q]);
      next();
    }
    for (int s0 = 0; s0 < niter; s0 += NS) {
#pragma unroll
      for (int q = 0; q < NS; ++q) {
        const int sl = (q + PF) % NS;
        load(a_r[sl], b_r[sl], m_r[sl], y_r[sl], v_r[sl]);
        next();
        // keep this step's prefetch loads ahead of its MFMAs: the scheduler would
        // otherwise sink them, and the wait before the next step's MFMAs would
        // then cover every load in flight
        __builtin_amdgcn_sched_barrier(0);
        // dz and its running sum each rounded once (see the pragma above)
        float bv[FN];
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          float b = b_r[q][j];
          if constexpr (GM == GM_POOL_MASK) {
            const bool on = (m_r[q] >> ((co0 + 16 * j + r16) & 31)) & 1u;
            b *= on ? s1 : sa;
          } else if constexpr (GM == GM_DY_Y) {
            b *= y_r[q][j] > 0.f ? 1.f : p.alpha;
          }
          bv[j] = b;
        }
        if (lead) {
#pragma unroll
          for (int j = 0; j < FN; ++j) {
            dsum[j] += bv[j];
            if (dz_out && v_r[q] >= 0) dz_out[(long long)v_r[q] * p.co + co0 + 16 * j + r16] = bv[j];
          }
        }
#pragma unroll
        for (int i = 0; i < RU; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int k = 0; k < FN; ++k)
              acc[i][j][k] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a_r[q][i][j]), bv[k],
                                                                  acc[i][j][k], 0, 0, 0);
      }
    }
  }

  // ---- partial dW of this slice ----------------------------------------------
  float *pw = part_w + (long long)slice * p.m * p.co;
#pragma unroll
  for (int i = 0; i < RU; ++i) {
    if (!uok[i]) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = rbase[i] + 4 * e + j;
#pragma unroll
        for (int k = 0; k < FN; ++k) pw[(long long)row * p.co + co0 + 16 * k + r16] = acc[i][j][k][e];
      }
  }
  if constexpr (FUSED) {
    // bias-gradient partial: the four voxel slots of each channel, in order
    if (lead)
#pragma unroll
      for (int j = 0; j < FN; ++j) dbs[g4][16 * j + r16] = dsum[j];
    __syncthreads();
    if (bx == 0 && threadIdx.x < 16 * FN) {
      const int c = threadIdx.x;
      part_b[(long long)slice * p.co + co0 + c] = ((dbs[0][c] + dbs[1][c]) + dbs[2][c]) + dbs[3][c];
    }
  }
}

}  // namespace
}  // namespace cf
