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
// every workgroup serialises dozens of load -> LDS -> MFMA stages, so the
// contraction runs at memory latency.  Here:
//  * a workgroup's four waves split the reduction over taps (a wave owns
//    taps u = w, w+4, ... or w, w+2, ...) and, optionally, the rows, so a
//    16- to 128-row tile still gives every wave its own independent stream
//    of loads; partial sums meet once, in LDS, at the end;
//  * the im2col operand is never staged: every lane loads its MFMA fragment
//    (8 consecutive channels of one gathered voxel, 16 bytes of NDHWC)
//    straight into registers, one k-step ahead of the MFMAs;
//  * forward weights W[t][ci][co] have the output channel contiguous, but the
//    MFMA B operand wants 8 consecutive input channels per lane: each wave
//    copies its 32 x 64 weight slice into a private LDS buffer (swizzled
//    against bank conflicts) and reads it back with the gfx950 transposing
//    read ds_read_b64_tr_b16; backward-data weights are already K-contiguous
//    (co fastest) and are loaded straight into registers;
//  * the epilogue sums the waves' partial tiles in LDS and writes whole
//    16-byte vectors of the destination (optionally bias + leaky ReLU and
//    the slope mask, the fused forward of an unpooled layer).
//
// v_mfma_f32_16x16x32_bf16 lane layout: A lane l holds row l%16 and K
// 8*(l/16)..+7; B lane l holds column l%16, same K; D lane l holds column
// l%16 and rows 4*(l/16)..+3.

#include "cf_common.h"
#include "cf_kernels.h"

#include <algorithm>
#include <cstdio>
#include <cstdlib>

namespace cf {
namespace {

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;
// plain 16-byte vector (a HIP uint4 is a struct, and its copies between
// address spaces stay memcpys through private memory)
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

struct DirParams {
  int nb;
  int sd_, sh_, sw_, sc;  // gathered tensor extent and channels (x forward, dz backward)
  int dd, dh, dw, dc;     // destination extent and channels (z forward, dx backward; GEMM N)
  int kd, kh, kw;         // kernel extent
  int s_d, s_h, s_w;      // conv stride
  int pd, ph, pw;         // padding before
  int wci, wco;           // weight channels W[t][wci][wco]
  int ncls;               // row classes: 1 forward, s_d*s_h*s_w backward-data
  float alpha;
};

// Row geometry of one class along one dimension.
//   forward:        source = j*s + q + u (q = -p),  weight tap = u,          destination = j
//   backward-data:  source = j + q - u,             weight tap = t0 + s*u,   destination = j*s + r
struct DimGeom {
  int j, u, t0, q;
};

template <bool FWD>
__device__ __forceinline__ DimGeom dim_geom(int r, int dst_ext, int k, int s, int pad) {
  DimGeom g;
  if (FWD) {
    g.j = dst_ext;
    g.u = k;
    g.t0 = 0;
    g.q = -pad;
  } else {
    g.j = dst_ext > r ? (dst_ext - r + s - 1) / s : 0;
    g.t0 = (r + pad) % s;
    g.u = g.t0 < k ? (k - g.t0 + s - 1) / s : 0;
    g.q = (r + pad - g.t0) / s;
  }
  return g;
}

// swizzled byte offset of (row, 32-byte chunk) in a wave's 32 x 64 bf16 weight
// slice: rows are 128 B, the chunk index is XORed with bits 1 and 3 of the row
// so that the eight rows a transposing read touches per half-wave land in
// distinct banks
__device__ __forceinline__ int wslice_off(int row, int chunk) {
  const int h = ((row >> 1) & 1) | (((row >> 3) & 1) << 1);
  return row * 128 + ((chunk ^ h) << 5);
}

template <bool FWD, int FM, int FN, int WM, int WK, bool ACT>
__global__ __launch_bounds__(256) void conv_direct_kernel(const uint16_t *__restrict__ src,
                                                          const uint16_t *__restrict__ wt,
                                                          const float *__restrict__ bias,
                                                          uint16_t *__restrict__ dst, uint8_t *__restrict__ mask,
                                                          DirParams p) {
  constexpr int BM = 16 * FM * WM, BN = 16 * FN;
  static_assert(WM * WK == 4, "four waves");
  static_assert(!FWD || FN == 4, "forward weight slices are 64 output channels wide");
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

  // ---- class and row tile of this workgroup --------------------------------
  int b = blockIdx.x, cls = 0;
  DimGeom gd, gh, gw;
  int rd = 0, rh = 0, rw = 0, m = 0;
  for (;;) {
    rd = FWD ? 0 : cls / (p.s_h * p.s_w);
    rh = FWD ? 0 : (cls / p.s_w) % p.s_h;
    rw = FWD ? 0 : cls % p.s_w;
    gd = dim_geom<FWD>(rd, p.dd, p.kd, p.s_d, p.pd);
    gh = dim_geom<FWD>(rh, p.dh, p.kh, p.s_h, p.ph);
    gw = dim_geom<FWD>(rw, p.dw, p.kw, p.s_w, p.pw);
    m = p.nb * gd.j * gh.j * gw.j;
    const int tiles = (m + BM - 1) / BM;
    if (b < tiles || cls + 1 >= p.ncls) break;
    b -= tiles;
    ++cls;
  }
  const int m0 = b * BM;
  if (m0 >= m) return;  // uniform: the whole workgroup leaves
  const int n0 = blockIdx.y * BN;
  const int bs_d = FWD ? p.s_d : 1, bs_h = FWD ? p.s_h : 1, bs_w = FWD ? p.s_w : 1;

  // ---- per-row-fragment source base ----------------------------------------
  int rbd[FM], rbh[FM], rbw[FM];
  const uint16_t *rp[FM];  // row base pointers (never dereferenced for an out-of-range voxel)
  bool rok[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int row = m0 + wm * 16 * FM + 16 * i + r16;
    rok[i] = row < m;
    const int rr = rok[i] ? row : 0;
    const int jw_ = rr % gw.j;
    int t = rr / gw.j;
    const int jh_ = t % gh.j;
    t /= gh.j;
    const int jd_ = t % gd.j;
    const int n = t / gd.j;
    rbd[i] = jd_ * bs_d + gd.q;
    rbh[i] = jh_ * bs_h + gh.q;
    rbw[i] = jw_ * bs_w + gw.q;
    const int rvox = ((n * p.sd_ + rbd[i]) * p.sh_ + rbh[i]) * p.sw_ + rbw[i];
    rp[i] = src + (long long)rvox * p.sc + 8 * g4;
  }

  // ---- this wave's k-steps: taps u = wk, wk + WK, ...; 32 channels per step --
  const int ntap = gd.u * gh.u * gw.u;
  const int nch = p.sc >> 5;
  const int mytaps = ntap > wk ? (ntap - wk + WK - 1) / WK : 0;
  const int nsteps = mytaps * nch;
  int cc = 0, ud = 0, uh = 0, uw = 0;
  if (mytaps > 0) {
    ud = wk / (gh.u * gw.u);
    uh = (wk / gw.u) % gh.u;
    uw = wk % gw.u;
  }
  auto advance = [&]() {
    if (++cc == nch) {
      cc = 0;
      uw += WK;
      while (uw >= gw.u) {
        uw -= gw.u;
        if (++uh == gh.u) {
          uh = 0;
          ++ud;
        }
      }
    }
  };

  u32x4_t a_nx[FM], w_nx[NW];
  auto load = [&]() {
    const int sgn_d = FWD ? ud : -ud, sgn_h = FWD ? uh : -uh, sgn_w = FWD ? uw : -uw;
    const long long soff = (long long)((sgn_d * p.sh_ + sgn_h) * p.sw_ + sgn_w) * p.sc + cc * 32;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const bool ok = rok[i] && (unsigned)(rbd[i] + sgn_d) < (unsigned)p.sd_ &&
                      (unsigned)(rbh[i] + sgn_h) < (unsigned)p.sh_ && (unsigned)(rbw[i] + sgn_w) < (unsigned)p.sw_;
      a_nx[i] = ok ? *reinterpret_cast<const u32x4_t *>(rp[i] + soff) : u32x4_t{0u, 0u, 0u, 0u};
    }
    const int tap = ((gd.t0 + (FWD ? 1 : p.s_d) * ud) * p.kh + (gh.t0 + (FWD ? 1 : p.s_h) * uh)) * p.kw +
                    (gw.t0 + (FWD ? 1 : p.s_w) * uw);
    if constexpr (FWD) {
      // slice W[tap][32 cc .. +32][n0 .. n0 + 64): 256 16-byte vectors, 4 per lane
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int q = lane + 64 * v;
        w_nx[v] = *reinterpret_cast<const u32x4_t *>(wt + ((long long)tap * p.wci + cc * 32 + (q >> 3)) * p.wco + n0 +
                                                   8 * (q & 7));
      }
    } else {
      // B fragment j: column ci = n0 + 16 j + l%16, K = 8 consecutive output channels
#pragma unroll
      for (int j = 0; j < FN; ++j)
        w_nx[j] = *reinterpret_cast<const u32x4_t *>(wt + ((long long)tap * p.wci + n0 + 16 * j + r16) * p.wco +
                                                   cc * 32 + 8 * g4);
    }
  };

  unsigned char *wbuf = smem + wave * 2 * WSLICE;
  // LDS byte offsets of this lane's four 16-byte weight vectors in a slice
  int wst[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int q = lane + 64 * v;
    wst[v] = wslice_off(q >> 3, (q & 7) >> 1) + (q & 1) * 16;
  }
#define CF_STAGE_W(buf)                                                              \
  do {                                                                               \
    _Pragma("unroll") for (int v = 0; v < 4; ++v)                                    \
        *reinterpret_cast<u32x4_t *>(wbuf + (buf) * WSLICE + wst[v]) = w_nx[v];      \
  } while (0)

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if (nsteps > 0) {
    load();
    if constexpr (FWD) CF_STAGE_W(0);
    u32x4_t a_cu[FM], b_cu[FWD ? 1 : NW];
#pragma unroll
    for (int i = 0; i < FM; ++i) a_cu[i] = a_nx[i];
    if constexpr (!FWD) {
#pragma unroll
      for (int j = 0; j < NW; ++j) b_cu[j] = w_nx[j];
    }
    for (int s = 0; s < nsteps; ++s) {
      const bool more = s + 1 < nsteps;
      if (more) {
        advance();
        load();
      }
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
        for (int j = 0; j < FN; ++j) bf[j] = __builtin_bit_cast(bf16x8_t, b_cu[j]);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const bf16x8_t af = __builtin_bit_cast(bf16x8_t, a_cu[i]);
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bf[j], acc[i][j], 0, 0, 0);
      }
      if (more) {
        if constexpr (FWD) CF_STAGE_W((s + 1) & 1);
#pragma unroll
        for (int i = 0; i < FM; ++i) a_cu[i] = a_nx[i];
        if constexpr (!FWD) {
#pragma unroll
          for (int j = 0; j < NW; ++j) b_cu[j] = w_nx[j];
        }
      }
    }
  }

#undef CF_STAGE_W

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
    if (grow >= m) continue;
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
    const int jw_ = grow % gw.j;
    int t = grow / gw.j;
    const int jh_ = t % gh.j;
    t /= gh.j;
    const int jd_ = t % gd.j;
    const int n = t / gd.j;
    const int od_ = FWD ? jd_ : jd_ * p.s_d + rd;
    const int oh_ = FWD ? jh_ : jh_ * p.s_h + rh;
    const int ow_ = FWD ? jw_ : jw_ * p.s_w + rw;
    const long long e0 = ((((long long)n * p.dd + od_) * p.dh + oh_) * p.dw + ow_) * p.dc + n0 + 8 * c8;
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

struct DirCfg {
  int fm, wm, wk;
};

template <bool FWD>
long long dir_tiles(const DirParams &p, int bm) {
  long long t = 0;
  for (int c = 0; c < p.ncls; ++c) {
    const int rd = FWD ? 0 : c / (p.s_h * p.s_w), rh = FWD ? 0 : (c / p.s_w) % p.s_h, rw = FWD ? 0 : c % p.s_w;
    auto J = [&](int r, int ext, int s) { return FWD ? ext : (ext > r ? (ext - r + s - 1) / s : 0); };
    const long long m = (long long)p.nb * J(rd, p.dd, p.s_d) * J(rh, p.dh, p.s_h) * J(rw, p.dw, p.s_w);
    t += (m + bm - 1) / bm;
  }
  return t;
}

template <bool FWD, int FN, bool ACT>
hipError_t launch_dir_t(const DirCfg &c, const DirParams &p, const void *src, const void *w, const float *bias,
                        void *dst, void *mask, hipStream_t st) {
  const int bm = 16 * c.fm * c.wm;
  dim3 grid((unsigned)dir_tiles<FWD>(p, bm), p.dc / (16 * FN), 1);
  if (grid.x == 0 || grid.y == 0) return hipSuccess;  // no destination rows
  const uint16_t *s16 = (const uint16_t *)src, *w16 = (const uint16_t *)w;
  uint16_t *d16 = (uint16_t *)dst;
  uint8_t *m8 = (uint8_t *)mask;
#define CF_DIR_LAUNCH(FM_, WM_, WK_)                                                                       \
  hipLaunchKernelGGL((conv_direct_kernel<FWD, FM_, FN, WM_, WK_, ACT>), grid, dim3(256), 0, st, s16, w16, \
                     bias, d16, m8, p)
  if (c.fm == 4 && c.wm == 2) CF_DIR_LAUNCH(4, 2, 2);
  else if (c.fm == 4 && c.wm == 1) CF_DIR_LAUNCH(4, 1, 4);
  else if (c.fm == 2 && c.wm == 2) CF_DIR_LAUNCH(2, 2, 2);
  else if (c.fm == 2 && c.wm == 1) CF_DIR_LAUNCH(2, 1, 4);
  else CF_DIR_LAUNCH(1, 1, 4);
#undef CF_DIR_LAUNCH
  return hipGetLastError();
}

// Tile choice: the largest row tile that still yields 512 workgroups (two
// per compute unit); more rows per wave amortise the weight stream, waves
// along K keep every wave busy when rows are few.  CF_DIRECT_TILE="fm,wm,wk"
// forces one of the candidates (tests cover every variant this way).
template <bool FWD>
DirCfg choose_cfg(const DirParams &p) {
  static const DirCfg cand[] = {{4, 2, 2}, {2, 2, 2}, {4, 1, 4}, {2, 1, 4}, {1, 1, 4}};
  if (const char *e = getenv("CF_DIRECT_TILE")) {
    int fm = 0, wm = 0, wk = 0;
    if (sscanf(e, "%d,%d,%d", &fm, &wm, &wk) == 3)
      for (const DirCfg &c : cand)
        if (c.fm == fm && c.wm == wm && c.wk == wk) return c;
  }
  const int fn = FWD ? 4 : (p.dc % 64 == 0 ? 4 : 2);
  const long long ny = p.dc / (16 * fn);
  for (const DirCfg &c : cand)
    if (dir_tiles<FWD>(p, 16 * c.fm * c.wm) * ny >= 512) return c;
  return cand[4];
}

}  // namespace

bool direct_supported(const ConvShape &s, bool fwd) {
  if (s.dtype != DT_BF16) return false;
  const int gc = fwd ? s.ci : s.co;  // contracted channels (32 per k-step)
  const int nc = fwd ? s.co : s.ci;  // GEMM columns
  if (gc % 32 != 0 || nc % 32 != 0) return false;
  if (fwd && nc % 64 != 0) return false;
  if (s.sd * s.sh * s.sw > 8) return false;
  // 32-bit voxel indices
  const long long vin = (long long)s.n * s.d * s.h * s.w, vout = (long long)s.n * s.od * s.oh * s.ow;
  if (vin >= (1LL << 31) / 8 || vout >= (1LL << 31) / 8) return false;
  return true;
}

hipError_t launch_conv_fwd_direct(const ConvShape &s, const void *x, const void *w, const float *bias, float alpha,
                                  void *out, void *mask, bool act, hipStream_t st) {
  DirParams p{};
  p.nb = s.n;
  p.sd_ = s.d; p.sh_ = s.h; p.sw_ = s.w; p.sc = s.ci;
  p.dd = s.od; p.dh = s.oh; p.dw = s.ow; p.dc = s.co;
  p.kd = s.kd; p.kh = s.kh; p.kw = s.kw;
  p.s_d = s.sd; p.s_h = s.sh; p.s_w = s.sw;
  p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.wci = s.ci; p.wco = s.co;
  p.ncls = 1;
  p.alpha = alpha;
  const DirCfg c = choose_cfg<true>(p);
  return act ? launch_dir_t<true, 4, true>(c, p, x, w, bias, out, mask, st)
             : launch_dir_t<true, 4, false>(c, p, x, w, nullptr, out, nullptr, st);
}

hipError_t launch_conv_bwd_data_direct(const ConvShape &s, const void *dz, const void *w, void *dx,
                                       hipStream_t st) {
  DirParams p{};
  p.nb = s.n;
  p.sd_ = s.od; p.sh_ = s.oh; p.sw_ = s.ow; p.sc = s.co;
  p.dd = s.d; p.dh = s.h; p.dw = s.w; p.dc = s.ci;
  p.kd = s.kd; p.kh = s.kh; p.kw = s.kw;
  p.s_d = s.sd; p.s_h = s.sh; p.s_w = s.sw;
  p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.wci = s.ci; p.wco = s.co;
  p.ncls = s.sd * s.sh * s.sw;
  p.alpha = 0.f;
  const DirCfg c = choose_cfg<false>(p);
  return p.dc % 64 == 0 ? launch_dir_t<false, 4, false>(c, p, dz, w, nullptr, dx, nullptr, st)
                        : launch_dir_t<false, 2, false>(c, p, dz, w, nullptr, dx, nullptr, st);
}

}  // namespace cf
