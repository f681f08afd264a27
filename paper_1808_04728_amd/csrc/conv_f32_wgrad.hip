// conv_f32_wgrad.hip -- fp32 backward-weights on v_mfma_f32_16x16x4_f32
// (Section III-C: the weight-gradient operator is a forward-like convolution
// with a large reduction and a small output; the paper gives each thread a
// private copy of the output and reduces the copies afterwards).
//
//   dW[t, ci, co] = sum_{n, o} x~[n, o*s + t - p, ci] dz[n, o, co]
//
// is a GEMM with rows (t, ci), columns co and the output voxels as K.  The
// voxels are split into fixed slices (grid z); a slice's partial dW goes to the
// caller's workspace and a fixed-order column sum adds the slices (bitwise
// reproducible, no atomics).  Inside a slice each wave owns RU row units of 64
// rows and FN column fragments of 16 output channels, and steps through the
// slice four voxels at a time (K slot = l/16 for lane l).
//
// One 16-byte load per lane feeds four MFMAs: lane l (m = l%16) loads four
// consecutive channels of one gathered voxel, and register j of the load is
// the A operand of MFMA j, whose row m then stands for
//   * 4^3-wide kernels (unit = (kd, kh, 16 channels from c0)): tap column
//     kw = m/4 and channel c0 + 4 (m%4) + j -- the 16 lanes of a voxel slot
//     read four neighbouring voxels x 64 bytes, one 256-byte run;
//   * 64k-channel layers (unit = (tap, 64 channels from c0)): channel
//     c0 + 4m + j -- 256 contiguous bytes of one voxel.
// The gradient operand (B: output channel l%16 at voxel slot l/16) is shared
// by every row of the wave.  Operands are streamed into registers PF steps
// ahead through range-checked buffer loads (a padding tap or a voxel past the
// slice reads zero).
//
// Fused variants: the gradient operand is rebuilt from the layer's output
// gradient -- pooled layers: from the pooled-output gradient g and the
// forward's slope mask,
//   dz[v, co] = g[pool(v), co] / 8 * (mask bit (v, co) ? 1 : alpha)
// (zero outside complete pooling windows); unpooled layers: from the gradient
// dy of the activation y and y itself,
//   dz[v, co] = dy[v, co] * (y[v, co] > 0 ? 1 : alpha)
// -- the bias gradient db = sum_v dz is summed from the same values in a fixed
// order, and dz can be stored once for the layer's backward-data.

#include "cf_common.h"
#include "cf_kernels.h"
#include "conv_f32_wgrad_kernel.h"
#include "fastdiv.h"

#include <algorithm>
#include <cstdlib>

namespace cf {
namespace {



__device__ __forceinline__ uint32_t ld32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4_t ld128(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}


// xcd_major: workgroup b (on XCD b % 8 by round-robin dispatch) takes grid
// position xcd * per + b / 8 of the (x fastest, then y, z) order, so an XCD
// runs a contiguous run of slices with all their row units and column groups,
// and the input and gradient rows those share meet in that XCD's L2 (the
// grid's size is a multiple of 8 when it is set)
template <int GM, bool KW4, int RU, int FN, int WV, int PF>
__global__ __launch_bounds__(64 * WV) void wgrad_f32_kernel(const float *__restrict__ x,
                                                            const float *__restrict__ g,
                                                            const void *__restrict__ aux,
                                                            float *__restrict__ part_w, float *__restrict__ part_b,
                                                            float *__restrict__ dz_out, const WF32Params p,
                                                            int xcd_major) {
  int bx = blockIdx.x, by = blockIdx.y, bz = blockIdx.z;
  if (xcd_major) {
    const int gx = gridDim.x, gy = gridDim.y;
    const int b = bx + gx * (by + gy * bz);
    const int per = gx * gy * (int)gridDim.z / 8;
    const int j = (b & 7) * per + (b >> 3);
    bx = j % gx;
    const int t = j / gx;
    by = t % gy;
    bz = t / gy;
  }
  wgrad_f32_body<GM, KW4, RU, FN, WV, PF>(x, g, aux, part_w, part_b, dz_out, p, bx, by, bz);
}

// ---------------------------------------------------------------------------
// The single-input-channel first layer (fp32, 16 output channels, fused with
// the pool and lReLU adjoints).  With one input channel every input voxel
// feeds all k^3 taps, so a tap-per-row operand would load each voxel k^3
// times.  Here lane l of fragment kw has row (kd, kh) = (l%16 / k, l%16 % k)
// and K slot l/16 holding four consecutive voxels: the lane loads one window
// of its (kd, kh) input row -- the aligned 16 bytes of its four voxels, the
// voxel before and two after -- and takes the A operands of all k fragments
// (kw = 0 .. k-1) from it by shifting.  Row k^2 of fragment 0 is a row of ones,
// which makes the bias gradient db = sum_v dz a row of the same accumulators.
// The gradient operand (B) is rebuilt per lane from the pooled gradient and
// the mask (a lane's four voxels share two pooling windows along w).  A
// wave walks 16-voxel segments of output rows; the eight waves of a
// workgroup meet in LDS and write one partial row per workgroup.
// ---------------------------------------------------------------------------

struct L1F32Params {
  int n, d, h, w;      // input
  int od, oh, ow;      // conv output
  int pd, ph;          // padding before (d, h)
  int pod, poh, pow_;  // pooled extents
  int total, per;      // 16-voxel row segments; per wave
  FastDiv fs, fh, fd;  // segment decode: segments per row, oh, od
  uint32_t x_bytes, g_bytes, m_bytes;
  float alpha;
};

__device__ __forceinline__ float2 ld64f(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
  const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
  return make_float2(__uint_as_float(v[0]), __uint_as_float(v[1]));
}

template <int KE, int PW, int WV, int PF>
__global__ __launch_bounds__(64 * WV) void l1_wgrad_f32_kernel(const float *__restrict__ x,
                                                               const float *__restrict__ dp,
                                                               const uint16_t *__restrict__ mask16,
                                                               float *__restrict__ part_w,
                                                               float *__restrict__ part_b, const L1F32Params p) {
  constexpr int R = KE * KE;  // (kd, kh) rows of a fragment
  static_assert(R < 16 && PW <= 1 && KE - PW <= 3, "window of the voxel before and two after");
  __shared__ float red[WV][KE][16][16];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g4 = lane >> 4, r16 = lane & 15;
  const bool rv = r16 < R;
  const float ones = r16 == R ? 1.f : 0.f;
  const int kd = rv ? r16 / KE : 0, kh = rv ? r16 % KE : 0;
  const int gw = blockIdx.x * WV + wave;
  const int s0 = gw * p.per, s1 = min(s0 + p.per, p.total);

  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc((void *)x, (short)0, p.x_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t gr = __builtin_amdgcn_make_buffer_rsrc((void *)dp, (short)0, p.g_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t mr = __builtin_amdgcn_make_buffer_rsrc((void *)mask16, (short)0, p.m_bytes, 0x00020000);

  struct Ld {
    u32x4_t cur;
    float left;
    float2 right;
    float g0, g1;
    float2 mk;  // the four voxels' 16-bit mask rows, as raw bits
  };
  constexpr int NS = PF + 1;
  Ld ring[NS];
  auto load = [&](int seg, Ld &L) {
    const bool live = seg < s1;
    const int sg = live ? seg : s0;
    const int t1 = fdiv(sg, p.fs), t2 = fdiv(t1, p.fh), nn = fdiv(t2, p.fd);
    const int ws = sg - t1 * (int)p.fs.div, oh_ = t1 - t2 * (int)p.fh.div, od_ = t2 - nn * (int)p.fd.div;
    const int wv0 = ws * 16 + 4 * g4;  // this lane's first voxel along w
    const int id = od_ + kd - p.pd, ih = oh_ + kh - p.ph;
    const bool rowok = live & rv & ((unsigned)id < (unsigned)p.d) & ((unsigned)ih < (unsigned)p.h);
    const uint32_t rb = (uint32_t)(((nn * p.d + id) * p.h + ih) * p.w + wv0) * 4u;
    // a valid byte offset is below 2^31: bit 31 sends a masked lane past the buffer (zeros)
    L.cur = ld128(xr, rb | ((uint32_t)!(rowok & (wv0 < p.w)) << 31));
    L.left = __uint_as_float(ld32(xr, (rb - 4u) | ((uint32_t)!(rowok & (wv0 >= 1)) << 31)));
    L.right = ld64f(xr, (rb + 16u) | ((uint32_t)!(rowok & (wv0 + 4 < p.w)) << 31));
    const int pd_ = od_ >> 1, ph_ = oh_ >> 1, pw0 = wv0 >> 1;
    const bool win = live & (pd_ < p.pod) & (ph_ < p.poh);
    const uint32_t gb = (uint32_t)(((((nn * p.pod + pd_) * p.poh + ph_) * p.pow_ + pw0) * 16) + r16) * 4u;
    L.g0 = __uint_as_float(ld32(gr, gb | ((uint32_t)!(win & (pw0 < p.pow_)) << 31)));
    L.g1 = __uint_as_float(ld32(gr, (gb + 64u) | ((uint32_t)!(win & (pw0 + 1 < p.pow_)) << 31)));
    const uint32_t mb = (uint32_t)(((nn * p.od + od_) * p.oh + oh_) * p.ow + wv0) * 2u;
    // two 4-byte loads: with an output w extent of 2 mod 4 the four voxels' rows
    // are 4-byte but not 8-byte aligned
    const uint32_t mbad = (uint32_t)!(live & (wv0 < p.ow)) << 31;
    L.mk = make_float2(__uint_as_float(ld32(mr, mb | mbad)), __uint_as_float(ld32(mr, (mb + 4u) | mbad)));
  };

  f32x4_t acc[KE];
#pragma unroll
  for (int k = 0; k < KE; ++k) acc[k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const float s1v = 0.125f, sav = 0.125f * p.alpha;
  const int nsteps = s1 > s0 ? s1 - s0 : 0;
  if (nsteps > 0) {
    const int niter = (nsteps + NS - 1) / NS * NS;
#pragma unroll
    for (int q = 0; q < PF; ++q) load(s0 + q, ring[q]);
    for (int b0 = 0; b0 < niter; b0 += NS) {
#pragma unroll
      for (int q = 0; q < NS; ++q) {
        load(s0 + b0 + q + PF, ring[(q + PF) % NS]);
        // keep this step's prefetch loads ahead of its MFMAs: the scheduler would
        // otherwise sink them, and the wait before the next step's MFMAs would
        // then cover every load in flight
        __builtin_amdgcn_sched_barrier(0);
        const Ld &L = ring[q];
        // window E[k] = x[wv0 - 1 + k], k = 0 .. 6
        const float E[7] = {L.left, __uint_as_float(L.cur[0]), __uint_as_float(L.cur[1]),
                            __uint_as_float(L.cur[2]), __uint_as_float(L.cur[3]), L.right.x, L.right.y};
        const uint32_t m01 = __float_as_uint(L.mk.x), m23 = __float_as_uint(L.mk.y);
        const uint32_t mb[4] = {m01, m01 >> 16, m23, m23 >> 16};
        float dz[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) dz[j] = (j < 2 ? L.g0 : L.g1) * (((mb[j] >> r16) & 1u) ? s1v : sav);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int kw = 0; kw < KE; ++kw) {
            const float a = rv ? E[kw - PW + 1 + j] : (kw == 0 ? ones : 0.f);
            acc[kw] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, dz[j], acc[kw], 0, 0, 0);
          }
      }
    }
  }

  // D row 4 (l/16) + e of fragment kw = (kd, kh) row, or the bias row R; column l%16
#pragma unroll
  for (int kw = 0; kw < KE; ++kw)
#pragma unroll
    for (int e = 0; e < 4; ++e) red[wave][kw][4 * g4 + e][r16] = acc[kw][e];
  __syncthreads();
  constexpr int TAPS = KE * KE * KE;
  for (int i = threadIdx.x; i < (TAPS + 1) * 16; i += 64 * WV) {
    const int row = i >> 4, co = i & 15;
    int kw = 0, rr = R;  // the bias row
    if (row < TAPS) {
      kw = row % KE;
      rr = row / KE;  // (kd, kh) = (row / KE / KE, row / KE % KE): fragment row kd * KE + kh
    }
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < WV; ++w) s += red[w][kw][rr][co];
    if (row < TAPS) part_w[(long long)blockIdx.x * TAPS * 16 + i] = s;
    else part_b[(long long)blockIdx.x * 16 + co] = s;
  }
}


WPlan w_plan(const ConvShape &s, int gm) {
  const bool fused = gm == GM_POOL_MASK;  // 32 channels per workgroup (one mask word)
  WPlan pl{};
  const long long vox = (long long)s.n * s.od * s.oh * s.ow;
  pl.kw4 = s.kw == 4 && s.ci % 16 == 0;
  if (pl.kw4) {
    pl.cunits = s.ci / 16;
    pl.units = s.kd * s.kh * pl.cunits;
  } else {
    pl.cunits = s.ci / 64;
    pl.units = s.kd * s.kh * s.kw * pl.cunits;
  }
  pl.fn = fused ? 2 : (s.co % 64 == 0 ? 4 : (s.co % 32 == 0 ? 2 : 1));
  // CF_F32W_FN=1|2|4 overrides the column groups of an unpooled launch (measurement sweeps)
  if (const char *e = getenv("CF_F32W_FN")) {
    const int f = atoi(e);
    if (!fused && (f == 1 || f == 2 || f == 4) && s.co % (16 * f) == 0) pl.fn = f;
  }
  // Row units per wave and workgroups per launch (measured on the 128^3 stack at
  // batch 1, sums included):
  //  * about one workgroup per compute unit, or per two for short reductions
  //    (below 2^16 voxels, where more slices would write more partials than the
  //    slices read operands);
  //  * pooled layers with short reductions (the stride-2 layer) take one row
  //    unit per wave and one workgroup per compute unit: twice the workgroups
  //    over the same slices (40 -> 31 us);
  //  (with a scalar-heavy step, two workgroups per compute unit measured faster
  //  on the 16 -> 32 layer, 218 -> 200 us; with the row values computed once per
  //  row, one is: 195 against 201 us, and half the partials).
  const bool shortk = vox < (1 << 16);
  // two row units per wave wherever the reduction is long: the A fragment's
  // loads and the gradient operand then feed twice the MFMAs (the 16 -> 32
  // layer's plain weight gradient on a stored dz: 171.5 -> 159.1 us)
  pl.ru = (fused ? !shortk : (!shortk || pl.units >= 64)) ? 2 : 1;
  // CF_F32W_RU=1|2 overrides the row units per wave (measurement sweeps)
  if (const char *e = getenv("CF_F32W_RU")) pl.ru = atoi(e) == 1 ? 1 : 2;
  pl.wv = 8;
  pl.gx = (pl.units + pl.ru * pl.wv - 1) / (pl.ru * pl.wv);
  pl.gy = s.co / (16 * pl.fn);
  const long long tiles = (long long)pl.gx * pl.gy;
  // plain reductions of 2^18 voxels and more: two workgroups per compute unit
  // (four waves per SIMD; the 16 -> 32 layer at 128^3 on a stored dz: step
  // -4.5 us with twice the partials; at the paper's 60^3, 2^17.7 voxels, the
  // doubled partials cost more than the waves gain: +3 us)
  const bool longk = vox >= (1 << 18);
  long long target = shortk ? (fused ? kNumCUs : kNumCUs / 2) : (!fused && longk ? 2 * kNumCUs : kNumCUs);
  // CF_F32W_TARGET overrides the workgroup target (measurement sweeps)
  if (const char *e = getenv("CF_F32W_TARGET")) target = std::max(1, atoi(e));
  long long want = std::max(1LL, (target + tiles - 1) / tiles);
  // CF_F32W_MINSTEPS overrides the shortest slice (measurement sweeps; 8 steps of
  // 4 voxels measured best on the stack's deep layers)
  const char *ms = getenv("CF_F32W_MINSTEPS");
  const long long minsteps = ms ? std::max(1, atoi(ms)) : 8;
  want = std::min(want, std::max(1LL, vox / (4 * minsteps)));
  // slices of whole output rows, at least minsteps steps of 4 voxels each
  const long long rows = (long long)s.n * s.od * s.oh;
  const long long nws = (s.ow + 3) / 4;
  long long per = (rows + want - 1) / want;
  per = std::max(per, (minsteps + nws - 1) / nws);
  pl.rows_per = (int)std::max(1LL, per);
  pl.nsplit = (int)((rows + pl.rows_per - 1) / pl.rows_per);
  return pl;
}

WF32Params w_params(const ConvShape &s, const WPlan &pl, float alpha) {
  WF32Params p{};
  p.n = s.n; p.d = s.d; p.h = s.h; p.w = s.w; p.ci = s.ci;
  p.od = s.od; p.oh = s.oh; p.ow = s.ow; p.co = s.co;
  p.sd = s.sd; p.sh = s.sh; p.sw = s.sw; p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.kh = s.kh; p.kw = s.kw;
  p.m = s.kd * s.kh * s.kw * s.ci;
  p.units = pl.units;
  p.cunits = pl.cunits;
  p.vox = s.n * s.od * s.oh * s.ow;
  p.rows_per = pl.rows_per;
  p.nws = (s.ow + 3) / 4;
  p.fh = make_fastdiv(s.oh);
  p.fd = make_fastdiv(s.od);
  p.x_bytes = (uint32_t)((long long)s.n * s.d * s.h * s.w * s.ci * 4);
  p.alpha = alpha;
  p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
  return p;
}

// CF_F32W_XCD=0 keeps the plain grid order of the weight-gradient workgroups
bool xcd_env() {
  const char *e = getenv("CF_F32W_XCD");
  return !(e && e[0] == '0');
}

template <int GM, bool KW4, int RU, int FN>
hipError_t launch_w(const WPlan &pl, const WF32Params &p, const float *x, const float *g, const void *aux,
                    float *pw, float *pb, float *dz_out, hipStream_t st) {
  dim3 grid(pl.gx, pl.gy, pl.nsplit);
  constexpr int PF = 2;
  const int xm = ((long long)pl.gx * pl.gy * pl.nsplit) % 8 == 0 && xcd_env();
  hipLaunchKernelGGL((wgrad_f32_kernel<GM, KW4, RU, FN, 8, PF>), grid, dim3(512), 0, st, x, g, aux, pw, pb,
                     dz_out, p, xm);
  return hipGetLastError();
}

template <int GM, bool KW4, int FN>
hipError_t launch_wu(const WPlan &pl, const WF32Params &p, const float *x, const float *g, const void *aux,
                     float *pw, float *pb, float *dz_out, hipStream_t st) {
  return pl.ru == 2 ? launch_w<GM, KW4, 2, FN>(pl, p, x, g, aux, pw, pb, dz_out, st)
                    : launch_w<GM, KW4, 1, FN>(pl, p, x, g, aux, pw, pb, dz_out, st);
}

template <int GM>
hipError_t launch_wfn(const WPlan &pl, const WF32Params &p, const float *x, const float *g, const void *aux,
                      float *pw, float *pb, float *dz_out, hipStream_t st) {
  if (pl.kw4)
    return pl.fn == 4 ? launch_wu<GM, true, 4>(pl, p, x, g, aux, pw, pb, dz_out, st)
         : pl.fn == 2 ? launch_wu<GM, true, 2>(pl, p, x, g, aux, pw, pb, dz_out, st)
                      : launch_wu<GM, true, 1>(pl, p, x, g, aux, pw, pb, dz_out, st);
  return pl.fn == 4 ? launch_wu<GM, false, 4>(pl, p, x, g, aux, pw, pb, dz_out, st)
       : pl.fn == 2 ? launch_wu<GM, false, 2>(pl, p, x, g, aux, pw, pb, dz_out, st)
                    : launch_wu<GM, false, 1>(pl, p, x, g, aux, pw, pb, dz_out, st);
}

}  // namespace

WPlan f32w_plan(const ConvShape &s, int gm) { return w_plan(s, gm); }
WF32Params f32w_params(const ConvShape &s, const WPlan &pl, float alpha) { return w_params(s, pl, alpha); }

namespace {
// two workgroups of eight waves per compute unit (four waves per SIMD; 62 -> 58
// us against one at 128^3); CF_L1F32_BLOCKS overrides the count (measurement
// sweeps)
int l1_blocks() {
  const char *e = getenv("CF_L1F32_BLOCKS");
  return e ? std::max(1, std::min(8 * kNumCUs, atoi(e))) : 2 * kNumCUs;
}

L1F32Params l1_params(const ConvShape &s, float alpha) {
  L1F32Params p{};
  p.n = s.n; p.d = s.d; p.h = s.h; p.w = s.w;
  p.od = s.od; p.oh = s.oh; p.ow = s.ow;
  p.pd = s.pd; p.ph = s.ph;
  p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
  const int nseg = (s.ow + 15) / 16;
  p.total = s.n * s.od * s.oh * nseg;
  p.per = (p.total + l1_blocks() * 8 - 1) / (l1_blocks() * 8);
  p.fs = make_fastdiv(nseg);
  p.fh = make_fastdiv(s.oh);
  p.fd = make_fastdiv(s.od);
  p.x_bytes = (uint32_t)((long long)s.n * s.d * s.h * s.w * 4);
  p.g_bytes = (uint32_t)((long long)s.n * p.pod * p.poh * p.pow_ * 16 * 4);
  p.m_bytes = (uint32_t)((long long)s.n * s.od * s.oh * s.ow * 2);
  p.alpha = alpha;
  return p;
}
}  // namespace

bool l1f32_wgrad_supported(const ConvShape &s) {
  const long long xin = (long long)s.n * s.d * s.h * s.w, vout = (long long)s.n * s.od * s.oh * s.ow;
  return s.dtype == DT_F32 && s.ci == 1 && s.co == 16 && s.sd == 1 && s.sh == 1 && s.sw == 1 && s.kd == s.kh &&
         s.kd == s.kw && (s.kd == 2 || s.kd == 3) && s.pw <= 1 && s.kd - s.pw <= 3 && s.w % 4 == 0 &&
         s.ow % 2 == 0 && s.od >= 2 && s.oh >= 2 && xin * 4 < (1LL << 31) && vout * 64 < (1LL << 31);
}

size_t l1f32_wgrad_workspace(const ConvShape &s) {
  return (size_t)l1_blocks() * (s.kd * s.kh * s.kw + 1) * 16 * sizeof(float);
}

hipError_t launch_l1_wgrad_f32(const ConvShape &s, const float *x, const float *dp, const uint16_t *mask,
                               float alpha, float *dw, float *db, void *ws, hipStream_t st) {
  const L1F32Params p = l1_params(s, alpha);
  const int nb = l1_blocks();
  const int taps = s.kd * s.kh * s.kw;
  float *pw = (float *)ws;
  float *pb = pw + (size_t)nb * taps * 16;
  if (s.kd == 2)
    hipLaunchKernelGGL((l1_wgrad_f32_kernel<2, 0, 8, 2>), dim3(nb), dim3(512), 0, st, x, dp, mask, pw, pb, p);
  else if (s.pw == 0)
    hipLaunchKernelGGL((l1_wgrad_f32_kernel<3, 0, 8, 2>), dim3(nb), dim3(512), 0, st, x, dp, mask, pw, pb, p);
  else
    hipLaunchKernelGGL((l1_wgrad_f32_kernel<3, 1, 8, 2>), dim3(nb), dim3(512), 0, st, x, dp, mask, pw, pb, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_sum_rows(pw, dw, nb, taps * 16, st);
  if (e != hipSuccess) return e;
  return launch_sum_rows(pb, db, nb, 16, st);
}

bool f32wgrad_supported(const ConvShape &s) {
  if (s.dtype != DT_F32 || s.co % 16 != 0) return false;
  if (!((s.kw == 4 && s.ci % 16 == 0) || s.ci % 64 == 0)) return false;
  const long long xin = (long long)s.n * s.d * s.h * s.w * s.ci, zout = (long long)s.n * s.od * s.oh * s.ow * s.co;
  const long long m = (long long)s.kd * s.kh * s.kw * s.ci;
  return xin * 4 < (1LL << 31) && zout * 4 < (1LL << 31) && m * s.co < (1LL << 31) && zout > 0;
}

bool f32wgrad_fused_supported(const ConvShape &s) {
  // 32 output channels per workgroup (one mask word per voxel and workgroup), any stride
  return f32wgrad_supported(s) && s.co % 32 == 0 && s.od >= 2 && s.oh >= 2 && s.ow >= 2;
}

size_t f32wgrad_workspace(const ConvShape &s, int gm) {
  const WPlan pl = w_plan(s, gm);
  return (size_t)pl.nsplit * ((size_t)s.kd * s.kh * s.kw * s.ci * s.co + (gm != GM_DZ ? s.co : 0)) * sizeof(float);
}

hipError_t launch_conv_bwd_weight_f32(const ConvShape &s, const float *x, const float *g, const void *aux,
                                      float alpha, float *dw, float *db, void *ws, int gm, float *dz_out,
                                      hipStream_t st) {
  const WPlan pl = w_plan(s, gm);
  WF32Params p = w_params(s, pl, alpha);
  float *pw = (float *)ws;
  const int m = p.m;
  float *pb = pw + (size_t)pl.nsplit * m * s.co;
  hipError_t e;
  if (gm == GM_POOL_MASK) {
    p.g_bytes = (uint32_t)((long long)s.n * p.pod * p.poh * p.pow_ * s.co * 4);
    p.m_bytes = (uint32_t)(((long long)p.vox * s.co + 31) / 32 * 4);
    e = pl.kw4 ? launch_wu<GM_POOL_MASK, true, 2>(pl, p, x, g, aux, pw, pb, dz_out, st)
               : launch_wu<GM_POOL_MASK, false, 2>(pl, p, x, g, aux, pw, pb, dz_out, st);
  } else if (gm == GM_DY_Y) {
    p.g_bytes = p.m_bytes = (uint32_t)((long long)p.vox * s.co * 4);
    e = launch_wfn<GM_DY_Y>(pl, p, x, g, aux, pw, pb, dz_out, st);
  } else {
    p.g_bytes = (uint32_t)((long long)p.vox * s.co * 4);
    e = launch_wfn<GM_DZ>(pl, p, x, g, nullptr, pw, nullptr, nullptr, st);
  }
  if (e != hipSuccess) return e;
  e = launch_sum_rows(pw, dw, pl.nsplit, m * s.co, st);
  if (e != hipSuccess || gm == GM_DZ) return e;
  return launch_sum_rows(pb, db, pl.nsplit, s.co, st);
}

}  // namespace cf
