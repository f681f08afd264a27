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

// tensors of at least this many bytes take the non-temporal forms in the
// streaming elementwise and pooling passes (the last-level cache is 256 MiB)
constexpr long long kStreamBytes = 1LL << 28;

}  // namespace cf
