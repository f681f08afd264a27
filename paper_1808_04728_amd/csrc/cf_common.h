// cf_common.h -- device helpers shared by the gfx950 kernels of this library.
//
// Storage types: fp32 tensors are `float`, bf16 tensors are raw `uint16_t`
// (IEEE bfloat16 bit patterns).  Arithmetic is always fp32; every bf16 store
// rounds to nearest even.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cf {

enum : int { DT_F32 = 0, DT_BF16 = 1 };

template <int DT> struct Store;
template <> struct Store<DT_F32> { using T = float; static constexpr int VEC = 4; };
template <> struct Store<DT_BF16> { using T = uint16_t; static constexpr int VEC = 8; };

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t u) { return __uint_as_float(((uint32_t)u) << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) {
  __bf16 b = (__bf16)f;  // round to nearest even (v_cvt_pk_bf16_f32 on gfx950)
  return __builtin_bit_cast(uint16_t, b);
}

// two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32, lo in bits 0..15
__device__ __forceinline__ uint32_t f2bf2(float lo, float hi) {
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t b = __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t);
  return __builtin_bit_cast(uint32_t, b);
}

template <int DT> __device__ __forceinline__ float to_f32(typename Store<DT>::T v);
template <> __device__ __forceinline__ float to_f32<DT_F32>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<DT_BF16>(uint16_t v) { return bf2f(v); }

template <int DT> __device__ __forceinline__ typename Store<DT>::T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<DT_F32>(float v) { return v; }
template <> __device__ __forceinline__ uint16_t from_f32<DT_BF16>(float v) { return f2bf(v); }

// 16-byte vector of storage elements, viewed either as raw words or elements.
template <int DT> union Vec16 {
  uint4 u;
  typename Store<DT>::T e[Store<DT>::VEC];
};

// 16-byte global load / store; NT = non-temporal (streaming) access for
// tensors read or written once and larger than the last-level cache, so they
// do not displace lines that other data still needs.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
template <bool NT> __device__ __forceinline__ uint4 ld16(const void *p) {
  if constexpr (NT) {
    const u32x4_t a = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    return make_uint4(a.x, a.y, a.z, a.w);
  } else {
    return *reinterpret_cast<const uint4 *>(p);
  }
}
template <bool NT> __device__ __forceinline__ void st16(void *p, uint4 v) {
  if constexpr (NT) {
    const u32x4_t a = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(a, reinterpret_cast<u32x4_t *>(p));
  } else {
    *reinterpret_cast<uint4 *>(p) = v;
  }
}

// Gradient operand of a fused backward kernel: dz rebuilt from what the layer
// kept instead of a stored dz.  GRAD_POOL: from the pooled-output gradient g
// and the forward's slope mask, dz = g / 8 * (bit ? 1 : alpha); GRAD_DYY: from
// the activation gradient dy and the activation y, dz = dy * (y > 0 ? 1 : alpha).
enum : int { GRAD_DZ = 0, GRAD_POOL = 1, GRAD_DYY = 3 };

// dz of eight bf16 channels in fp32: GRAD_POOL gv = g, bits 0..7 of av[0] = the
// mask bits of the eight channels; GRAD_DYY gv = dy, av = y
template <int GM>
__device__ __forceinline__ void form_dz8(const u32x4_t &gv, const u32x4_t &av, float alpha, float (&f)[8]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float lo = __uint_as_float(gv[q] << 16), hi = __uint_as_float(gv[q] & 0xffff0000u);
    if constexpr (GM == GRAD_POOL) {
      const uint32_t bits = av[0] >> (2 * q);
      f[2 * q] = lo * ((bits & 1u) ? 0.125f : 0.125f * alpha);
      f[2 * q + 1] = hi * ((bits & 2u) ? 0.125f : 0.125f * alpha);
    } else {
      // y > 0 for a bf16 value: its 32-bit widening compared as a signed integer
      const bool plo = (int)(av[q] << 16) > 0, phi = (int)(av[q] & 0xffff0000u) > 0;
      f[2 * q] = lo * (plo ? 1.f : alpha);
      f[2 * q + 1] = hi * (phi ? 1.f : alpha);
    }
  }
}

// Split form of the same dz for kernels that multiply it into a matrix product:
// dz = s1 * src + s2 * (src & sel) with sel = 0xffff on the bf16 halves where
// the slope is 1 (GRAD_POOL: s1 = alpha / 8, s2 = (1 - alpha) / 8, sel = the mask
// bits; GRAD_DYY: s1 = alpha, s2 = 1 - alpha, sel = y > 0).  src and src & sel are
// exact bf16 values, so two products of them, scaled and added in fp32, give
// dz times the other operand without rounding dz itself.
// sel of eight channels from their eight mask bits (word q: bits 2q, 2q + 1)
__device__ __forceinline__ u32x4_t sel_of_bits8(uint32_t bits) {
  u32x4_t m;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t lo = (uint32_t)((int)(bits << (31 - 2 * q)) >> 31);  // 0 or all ones
    const uint32_t hi = (uint32_t)((int)(bits << (30 - 2 * q)) >> 31);
    m[q] = (lo & 0xffffu) | (hi & 0xffff0000u);
  }
  return m;
}

// sel of eight channels from their bf16 activations: 0xffff where y > 0 (as a
// signed 16-bit integer a bf16 value is positive exactly when it is > 0)
__device__ __forceinline__ u32x4_t sel_of_pos8(const u32x4_t &y) {
  typedef short s16x2_t __attribute__((ext_vector_type(2)));
  typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));
  u32x4_t m;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t yq = y[q];  // (a bit cast of the element expression itself would read element 0)
    const s16x2_t v = __builtin_bit_cast(s16x2_t, yq);
    const u16x2_t pos = __builtin_bit_cast(u16x2_t, __builtin_elementwise_max(v, (s16x2_t){0, 0}));
    const u16x2_t one = __builtin_elementwise_min(pos, (u16x2_t){1, 1});  // 1 where y > 0
    m[q] = __builtin_bit_cast(uint32_t, (u16x2_t){0, 0} - one);
  }
  return m;
}

// eight fp32 values rounded (to nearest even) into eight packed bf16
__device__ __forceinline__ u32x4_t pack_bf16x8(const float (&f)[8]) {
  return u32x4_t{f2bf2(f[0], f[1]), f2bf2(f[2], f[3]), f2bf2(f[4], f[5]), f2bf2(f[6], f[7])};
}

// tensors of at least this many bytes take the non-temporal forms in the
// streaming elementwise and pooling passes (the last-level cache is 256 MiB)
constexpr long long kStreamBytes = 1LL << 28;

}  // namespace cf
