// conv_direct_wgrad.hip -- weight gradient of the deep layers of the stack
// (bf16, input channels a multiple of 8, output channels a multiple of 64).
//
// The weight gradient (Section III-C, Algorithm 1) is the contraction over
// every output voxel v = (n, o):
//   dW[t, ci, co] = sum_v x~[n, o*s + t - p, ci] dz[v, co]
// i.e. a GEMM with rows (t, ci) (the flattened [kd][kh][kw][ci] index of the
// weight, M = k^3 ci), columns co and reduction K = output voxels.  At a few
// thousand to a few tens of thousands of voxels per layer the reduction is
// split over K (slices of whole k-steps); every slice writes a fp32 partial
// of the whole gradient and a fixed-order column sum (reduce.hip) adds the
// slices, so the result bits depend on the shape and the data alone.
//
// Data movement (same scheme as the LDS-staged forward kernel):
//  * a workgroup owns a (64 WM) x (64 WN) block of dW (WM x WN = 4 waves, a
//    64 x 64 block per wave) and one K slice; per k-step of 32 voxels it
//    stages, by buffer -> LDS DMA, a [32 voxels][64 rows] tile for each of
//    its WM row blocks (8 consecutive rows = 8 channels of one tap, gathered
//    from the voxel's tap neighbour in NDHWC; padding voxels and voxels past
//    the slice read as zero through the range check) and a [32 voxels][64
//    co] tile of dz for each of its WN column blocks;
//  * both MFMA operands want 8 consecutive voxels per lane, so both tiles are
//    read back with the transposing read ds_read_b64_tr_b16; the DMA applies
//    the bank swizzle of those reads on the global side (each lane's 16
//    bytes land at a fixed LDS slot);
//  * LNS = 4 stages in separate LDS arrays visited by an unrolled ring, one
//    barrier per k-step, whole rounds of four steps (the steps past the end
//    load zeros): the compiler then tracks which stage each DMA fills and the
//    only wait is the explicit one;
//  * the partial block leaves straight from the accumulators (16 lanes write
//    64 contiguous bytes of a dW row).
//
// Fused variants (the gradient operand rebuilt, never read from a stored dz):
// pooled layers take the pooled-output gradient g and the forward's slope mask,
//   dz[v, co] = g[pool(v), co] / 8 * (mask bit (v, co) ? 1 : alpha)
// (zero outside complete pooling windows); unpooled layers take the gradient
// dy of the activation y and y itself,
//   dz[v, co] = dy[v, co] * (y[v, co] > 0 ? 1 : alpha).
// Each thread loads its slot's sources into registers with the same lead as
// the DMA, forms dz in fp32, rounds it to bf16 into the LDS slot the DMA
// would have filled, and adds the fp32 values to its share of the bias
// gradient db = sum_v dz; the shares of a slice meet in a fixed order (lane
// butterfly, then the four waves) and the workgroups of the slice's first
// row block write them as one partial row of db.

#include "cf_common.h"
#include "cf_kernels.h"
#include "fastdiv.h"

#include <algorithm>
#include <cstdlib>

namespace cf {
namespace {

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef short v8i16_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr uint32_t DW_OOB = 0x80000000u;  // past every buffer: the load returns zeros
constexpr int DW_LNS = 4;                 // pipeline stages

struct DwParams {
  int d, h, w, ci;        // input extent and channels
  int co;                 // output channels
  int kh, kw;             // kernel extent (kd follows from the row count)
  int sd, sh, sw;         // strides
  int pd, ph, pw;         // padding before
  int m;                  // GEMM rows: kd kh kw ci
  int pvox;               // output voxels n od oh ow (the reduction)
  int chunk;              // voxels per K slice (a multiple of 32)
  int mt, nt, jobs;       // row blocks, column blocks, mt nt slices
  int per;                // jobs per XCD
  int x_bytes, g_bytes;   // extents of the range-checked buffers (g: dz, pooled gradient or dy)
  int aux_bytes;          // fused: extent of the slope mask or of y
  int pod, poh, pow_;     // pooled extents (pooled gradient)
  float alpha;            // fused: leaky-ReLU slope
  FastDiv fow, foh, fod;  // output extent divisors
};

// gradient operand of the weight-gradient kernel
enum : int { DW_DZ = GRAD_DZ, DW_POOL = GRAD_POOL, DW_DYY = GRAD_DYY };

// byte offset of (row, 32-byte chunk) in a [32][64] bf16 tile with 128-byte
// rows: the chunk index is XORed with bits 1 and 3 of the row so that the
// rows one transposing read touches per half-wave fall in distinct banks
__device__ __forceinline__ int tile_off(int row, int chunk) {
  const int h = ((row >> 1) & 1) | (((row >> 3) & 1) << 1);
  return row * 128 + ((chunk ^ h) << 5);
}

template <int N>
struct Stage {
  static constexpr int v = N;
};

__device__ __forceinline__ u32x4_t ld128(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

template <int WN, int GM>
__global__ __launch_bounds__(256, GM == GRAD_DZ ? 2 : 1) void dw_lds_kernel(const uint16_t *__restrict__ x,
                                                        const uint16_t *__restrict__ g,
                                                        const void *__restrict__ aux, float *__restrict__ part,
                                                        float *__restrict__ part_b, const DwParams p) {
  constexpr int WM = 4 / WN;
  constexpr bool FUSED = GM != DW_DZ;
  // vector-memory instructions per thread and k-step: one DMA per 4 KB tile,
  // plus (fused) the two register loads of each gradient tile
  constexpr int NBLK = WM + (FUSED ? 2 * WN : WN);
  // x and dz tiles of each stage in arrays of their own: every fragment read
  // then matches exactly one array the DMA fills
  __shared__ __attribute__((aligned(16))) unsigned char sa0[WM * 4096], sb0[WN * 4096];
  __shared__ __attribute__((aligned(16))) unsigned char sa1[WM * 4096], sb1[WN * 4096];
  __shared__ __attribute__((aligned(16))) unsigned char sa2[WM * 4096], sb2[WN * 4096];
  __shared__ __attribute__((aligned(16))) unsigned char sa3[WM * 4096], sb3[WN * 4096];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int g4 = lane >> 4, r16 = lane & 15;
  // jobs in slice-major order, XCD x (workgroups b with b % 8 == x) taking
  // the contiguous run [x per, (x + 1) per): consecutive slices, i.e. one
  // contiguous range of voxels whose x and dz stay in that XCD's L2
  const int job = (blockIdx.x & 7) * p.per + (blockIdx.x >> 3);
  if (job >= p.jobs) return;
  const int split = job / (p.mt * p.nt), tile = job - split * (p.mt * p.nt);
  const int mrow0 = (tile % p.mt) * 64 * WM, n0 = (tile / p.mt) * 64 * WN;
  const int vbeg = split * p.chunk;
  const int vend = min(p.pvox, vbeg + p.chunk);
  const int nsteps = vend > vbeg ? (vend - vbeg + 31) >> 5 : 0;

  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc((void *)x, (short)0, p.x_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t zr = __builtin_amdgcn_make_buffer_rsrc((void *)g, (short)0, p.g_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t ar =
      __builtin_amdgcn_make_buffer_rsrc((void *)aux, (short)0, FUSED ? p.aux_bytes : 0, 0x00020000);
  (void)ar;

  // this thread's DMA slot in every tile: voxel row vr of the k-step, 16-byte
  // slot j, which holds logical 8-element chunk lj (the swizzle of tile_off)
  const int vr = tid >> 3, j = tid & 7;
  const int hsw = ((vr >> 1) & 1) | (((vr >> 3) & 1) << 1);
  const int lj = 2 * ((j >> 1) ^ hsw) + (j & 1);
  // A tiles: rows mrow0 + 64 k + 8 lj .. +7 are channels c.. of tap (td, th, tw)
  int a_d[WM], a_h[WM], a_w[WM], a_c[WM];
#pragma unroll
  for (int k = 0; k < WM; ++k) {
    const int m = mrow0 + 64 * k + 8 * lj;
    const int tap = m / p.ci, c = m - tap * p.ci;
    const int tw = tap % p.kw, t1 = tap / p.kw, th = t1 % p.kh, td = t1 / p.kh;
    a_d[k] = m < p.m ? td - p.pd : -(1 << 20);  // rows past the gradient fail every bounds check
    a_h[k] = th - p.ph;
    a_w[k] = tw - p.pw;
    a_c[k] = c;
  }
  // dz tiles: output channels n0 + 64 k + 8 lj .. +7
  int b_col[WN];
#pragma unroll
  for (int k = 0; k < WN; ++k) b_col[k] = n0 + 64 * k + 8 * lj;

  auto stage_a = [&](auto ix) -> unsigned char * {
    constexpr int S = decltype(ix)::v;
    if constexpr (S == 0) return sa0;
    else if constexpr (S == 1) return sa1;
    else if constexpr (S == 2) return sa2;
    else return sa3;
  };
  auto stage_b = [&](auto ix) -> unsigned char * {
    constexpr int S = decltype(ix)::v;
    if constexpr (S == 0) return sb0;
    else if constexpr (S == 1) return sb1;
    else if constexpr (S == 2) return sb2;
    else return sb3;
  };

  // fused: the gradient sources of the LNS steps in flight (register ring,
  // one slot per stage) and this thread's share of db
  u32x4_t gsrc[DW_LNS][WN], asrc[DW_LNS][WN];
  float dbs[WN][8];
#pragma unroll
  for (int k = 0; k < WN; ++k)
#pragma unroll
    for (int e = 0; e < 8; ++e) dbs[k][e] = 0.f;

  int vnext = vbeg + vr;  // this thread's voxel in the next step to load
  auto issue = [&](auto ix) {
    constexpr int S = decltype(ix)::v;
    unsigned char *sa = stage_a(ix), *sb = stage_b(ix);
    const int vg = vnext;
    vnext += 32;
    const bool live = vg < vend;
    const int vv = live ? vg : 0;
    const int t1 = fdiv(vv, p.fow), t2 = fdiv(t1, p.foh), n = fdiv(t2, p.fod);
    const int ow0 = vv - t1 * (int)p.fow.div, oh0 = t1 - t2 * (int)p.foh.div, od0 = t2 - n * (int)p.fod.div;
    const int bw = ow0 * p.sw, bh = oh0 * p.sh, bd = od0 * p.sd;
    if constexpr (GM == DW_DYY) {
#pragma unroll
      for (int k = 0; k < WN; ++k) {
        uint32_t off = live ? (uint32_t)(vv * p.co + b_col[k]) * 2u : DW_OOB;
        asm volatile("" : "+v"(off));
        gsrc[S][k] = ld128(zr, off);
        asrc[S][k] = ld128(ar, off);
      }
    } else if constexpr (GM == DW_POOL) {
      // outside complete pooling windows the gradient reads as zero
      const bool inp = live & (od0 < 2 * p.pod) & (oh0 < 2 * p.poh) & (ow0 < 2 * p.pow_);
      const int pv = ((n * p.pod + (od0 >> 1)) * p.poh + (oh0 >> 1)) * p.pow_ + (ow0 >> 1);
#pragma unroll
      for (int k = 0; k < WN; ++k) {
        uint32_t off = inp ? (uint32_t)(pv * p.co + b_col[k]) * 2u : DW_OOB;
        uint32_t moff = live ? (uint32_t)(vv * p.co + b_col[k]) >> 3 : DW_OOB;
        asm volatile("" : "+v"(off), "+v"(moff));
        gsrc[S][k] = ld128(zr, off);
        asrc[S][k][0] = __builtin_amdgcn_raw_buffer_load_b8(ar, moff, 0, 0);
      }
    }
#pragma unroll
    for (int k = 0; k < WM; ++k) {
      const int id = bd + a_d[k], ih = bh + a_h[k], iw = bw + a_w[k];
      const bool ok = live & ((unsigned)id < (unsigned)p.d) & ((unsigned)ih < (unsigned)p.h) &
                      ((unsigned)iw < (unsigned)p.w);
      uint32_t off = ok ? (uint32_t)((((n * p.d + id) * p.h + ih) * p.w + iw) * p.ci + a_c[k]) * 2u : DW_OOB;
      asm volatile("" : "+v"(off));  // a select, not two predicated copies of the load
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t *)(sa + k * 4096 + wave * 1024), 16, off, 0, 0, 0);
    }
    if constexpr (!FUSED) {
#pragma unroll
      for (int k = 0; k < WN; ++k) {
        uint32_t off = live ? (uint32_t)(vv * p.co + b_col[k]) * 2u : DW_OOB;
        asm volatile("" : "+v"(off));
        __builtin_amdgcn_raw_ptr_buffer_load_lds(zr, (lds_void_t *)(sb + k * 4096 + wave * 1024), 16, off, 0,
                                                 0, 0);
      }
    }
  };

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) acc[i][jn] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // fragment of 16 tile columns (chunk cc): 8 consecutive voxels per lane
  auto frag = [&](const unsigned char *tile, int cc) {
    const int row = 8 * g4 + (r16 >> 2);
    const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(tile + tile_off(row, cc) + (r16 & 3) * 8));
    const v4i16_t hi =
        __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(tile + tile_off(row + 4, cc) + (r16 & 3) * 8));
    const v8i16_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8_t, v);
  };

  // one k-step on stage ix: wait for this thread's loads of the step (the next
  // LNS - 2 steps may stay in flight) and its fragment reads of the previous
  // step, (fused: form this step's dz into its slots of the stage), barrier,
  // refill the previous step's stage, MFMAs of this step.  Vector-memory
  // loads complete in issue order, so vmcnt(VMC) covers this step's loads.
  auto kstep = [&](auto ix) {
    constexpr int S = decltype(ix)::v;
    constexpr int VMC = (DW_LNS - 2) * NBLK;
    __builtin_amdgcn_s_waitcnt(0x0070 | (VMC & 15) | ((VMC >> 4) << 14));  // vmcnt(VMC) lgkmcnt(0)
    if constexpr (FUSED) {
#pragma unroll
      for (int k = 0; k < WN; ++k) {
        float f[8];
        form_dz8<GM>(gsrc[S][k], asrc[S][k], p.alpha, f);
#pragma unroll
        for (int e = 0; e < 8; ++e) dbs[k][e] += f[e];
        const u32x4_t v = pack_bf16x8(f);
        *reinterpret_cast<u32x4_t *>(stage_b(ix) + k * 4096 + tid * 16) = v;
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the slots are written
    }
    asm volatile("s_barrier" ::: "memory");
    issue(Stage<(S + DW_LNS - 1) % DW_LNS>{});
    bf16x8_t af[4], bf[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = frag(stage_a(ix) + wm * 4096, i);
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) bf[jn] = frag(stage_b(ix) + wn * 4096, jn);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jn = 0; jn < 4; ++jn) acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[jn], acc[i][jn], 0, 0, 0);
  };

  if (nsteps > 0) {
    issue(Stage<0>{});
    issue(Stage<1>{});
    issue(Stage<2>{});
    for (int s = 0; s < nsteps; s += DW_LNS) {
      kstep(Stage<0>{});
      kstep(Stage<1>{});
      kstep(Stage<2>{});
      kstep(Stage<3>{});
    }
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): no DMA outlives the workgroup
  }

  // every partial element of the block is written (zeros for an empty slice)
  float *dst = part + (long long)split * p.m * p.co;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = mrow0 + 64 * wm + 16 * i + 4 * g4 + e;
      if (m >= p.m) continue;
#pragma unroll
      for (int jn = 0; jn < 4; ++jn) dst[(long long)m * p.co + n0 + 64 * wn + 16 * jn + r16] = acc[i][jn][e];
    }

  if constexpr (FUSED) {
    // db shares: a wave's voxel rows with the same logical chunk (lane bits 3
    // and 5; bit 4 selects a swizzle, i.e. another chunk) by a butterfly, then
    // the eight partial rows in order; the slice's first row block writes
    if (mrow0 != 0) return;  // uniform
#pragma unroll
    for (int k = 0; k < WN; ++k)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float v = dbs[k][e];
        v += __shfl_xor(v, 8);
        v += __shfl_xor(v, 32);
        dbs[k][e] = v;
      }
    __syncthreads();  // every wave is done with the stage arrays
    float *red = reinterpret_cast<float *>(sa0);  // [8 partial rows][64 WN channels]
    if ((lane & 0x28) == 0) {
      const int r = 2 * wave + ((lane >> 4) & 1);
#pragma unroll
      for (int k = 0; k < WN; ++k)
#pragma unroll
        for (int e = 0; e < 8; ++e) red[r * 64 * WN + 64 * k + 8 * lj + e] = dbs[k][e];
    }
    __syncthreads();
    if (tid < 64 * WN) {
      float v = 0.f;
#pragma unroll
      for (int r = 0; r < 8; ++r) v += red[r * 64 * WN + tid];
      part_b[(long long)split * p.co + n0 + tid] = v;
    }
  }
}

struct DwPlan {
  int wn, mt, nt, chunk, nsplit;
};

// Column blocks of 128 when the output channels allow (two waves share each
// gathered tile), else 64.  K slices: enough workgroups for two per compute
// unit (CF_DWGRAD_WGS overrides the target), but at least 8 k-steps each.
DwPlan plan(const ConvShape &s) {
  DwPlan pl;
  pl.wn = s.co % 128 == 0 ? 2 : 1;
  const int m = s.kd * s.kh * s.kw * s.ci;
  pl.mt = (m + 64 * (4 / pl.wn) - 1) / (64 * (4 / pl.wn));
  pl.nt = s.co / (64 * pl.wn);
  int target = 512;
  if (const char *e = getenv("CF_DWGRAD_WGS")) target = std::max(1, atoi(e));
  const long long pvox = (long long)s.n * s.od * s.oh * s.ow;
  const long long tiles = (long long)pl.mt * pl.nt;
  const long long want = std::max(1LL, (target + tiles - 1) / tiles);
  long long chunk = (pvox + want - 1) / want;
  chunk = std::max(256LL, (chunk + 31) / 32 * 32);
  pl.chunk = (int)chunk;
  pl.nsplit = (int)std::max(1LL, (pvox + chunk - 1) / chunk);
  return pl;
}

}  // namespace

bool direct_wgrad_supported(const ConvShape &s) {
  if (s.dtype != DT_BF16) return false;
  if (s.ci % 8 != 0 || s.co % 64 != 0) return false;
  const long long xin = (long long)s.n * s.d * s.h * s.w * s.ci;
  const long long pvox = (long long)s.n * s.od * s.oh * s.ow;
  const long long m = (long long)s.kd * s.kh * s.kw * s.ci;
  if (xin * 2 >= (1LL << 31) || pvox * s.co * 2 >= (1LL << 31) || m * s.co >= (1LL << 31)) return false;
  return pvox > 0;
}

size_t direct_wgrad_workspace(const ConvShape &s, bool fused) {
  const DwPlan pl = plan(s);
  return (size_t)pl.nsplit * ((size_t)s.kd * s.kh * s.kw * s.ci * s.co + (fused ? s.co : 0)) * sizeof(float);
}

template <int GM>
static hipError_t launch_dw(int wn, dim3 grid, const DwParams &p, const void *x, const void *g, const void *aux,
                            float *pw, float *pb, hipStream_t st) {
  const uint16_t *x16 = (const uint16_t *)x, *g16 = (const uint16_t *)g;
  if (wn == 2)
    hipLaunchKernelGGL((dw_lds_kernel<2, GM>), grid, dim3(256), 0, st, x16, g16, aux, pw, pb, p);
  else
    hipLaunchKernelGGL((dw_lds_kernel<1, GM>), grid, dim3(256), 0, st, x16, g16, aux, pw, pb, p);
  return hipGetLastError();
}

hipError_t launch_conv_bwd_weight_direct(const ConvShape &s, const void *x, const void *g, const void *aux, int gm,
                                         float alpha, float *dw, float *db, void *ws, hipStream_t st) {
  const DwPlan pl = plan(s);
  DwParams p{};
  p.d = s.d; p.h = s.h; p.w = s.w; p.ci = s.ci; p.co = s.co;
  p.kh = s.kh; p.kw = s.kw;
  p.sd = s.sd; p.sh = s.sh; p.sw = s.sw;
  p.pd = s.pd; p.ph = s.ph; p.pw = s.pw;
  p.m = s.kd * s.kh * s.kw * s.ci;
  p.pvox = s.n * s.od * s.oh * s.ow;
  p.chunk = pl.chunk;
  p.x_bytes = (int)((long long)s.n * s.d * s.h * s.w * s.ci * 2);
  p.pod = s.od / 2; p.poh = s.oh / 2; p.pow_ = s.ow / 2;
  p.alpha = alpha;
  const long long zb = (long long)p.pvox * s.co * 2;
  if (gm == DWG_POOL) {
    p.g_bytes = (int)((long long)s.n * p.pod * p.poh * p.pow_ * s.co * 2);
    p.aux_bytes = (int)(((long long)p.pvox * s.co + 31) / 32 * 4);
  } else {
    p.g_bytes = p.aux_bytes = (int)zb;
  }
  p.fow = make_fastdiv(s.ow);
  p.foh = make_fastdiv(s.oh);
  p.fod = make_fastdiv(s.od);
  p.mt = pl.mt;
  p.nt = pl.nt;
  p.jobs = pl.mt * pl.nt * pl.nsplit;
  p.per = (p.jobs + 7) / 8;
  float *pw = (float *)ws;
  float *pb = pw + (size_t)pl.nsplit * p.m * s.co;
  const dim3 grid((unsigned)(8 * p.per));
  hipError_t e;
  if (gm == DWG_POOL) e = launch_dw<DW_POOL>(pl.wn, grid, p, x, g, aux, pw, pb, st);
  else if (gm == DWG_DYY) e = launch_dw<DW_DYY>(pl.wn, grid, p, x, g, aux, pw, pb, st);
  else e = launch_dw<DW_DZ>(pl.wn, grid, p, x, g, nullptr, pw, nullptr, st);
  if (e != hipSuccess) return e;
  e = launch_sum_rows(pw, dw, pl.nsplit, p.m * s.co, st);
  if (e != hipSuccess || gm == DWG_DZ) return e;
  return launch_sum_rows(pb, db, pl.nsplit, s.co, st);
}

}  // namespace cf
