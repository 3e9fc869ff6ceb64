// Device side of the fused entry point's prologue: a bf16 input element x of
// channel c becomes RNE_bf16(SiLU(x * scale[n][c] + shift[n][c])), with
// SiLU(u) = u / (1 + e^-u) in fp32 (hardware exponential and reciprocal,
// a few ulp of fp32, far below one bf16 step) and one round-to-nearest-even
// conversion.  Included by the kernel translation units only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace c3c {

typedef uint32_t fuse_u32x4 __attribute__((ext_vector_type(4)));
typedef float fuse_f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 fuse_bf16x2 __attribute__((ext_vector_type(2)));

__device__ inline float fuse_silu(float u) {
  // e^-u overflows to +inf for u < -88: the reciprocal is then 0 and the
  // result -0, the limit of SiLU
  return u * __builtin_amdgcn_rcpf(1.f + __expf(-u));
}

// two bf16 elements packed in one dword, both of the same channel; lo_ok /
// hi_ok false keeps that element's bits (the zero of a padding position)
__device__ inline uint32_t fuse_pair(uint32_t v, float s, float t, bool lo_ok, bool hi_ok) {
  const float a = fuse_silu(__builtin_fmaf(__uint_as_float(v << 16), s, t));
  const float b = fuse_silu(__builtin_fmaf(__uint_as_float(v & 0xffff0000u), s, t));
  const uint32_t r = __builtin_bit_cast(uint32_t, __builtin_convertvector((fuse_f32x2{a, b}), fuse_bf16x2));
  return (lo_ok ? (r & 0xffffu) : (v & 0xffffu)) | (hi_ok ? (r & 0xffff0000u) : (v & 0xffff0000u));
}

// 8 consecutive elements of one channel, all valid or all kept
__device__ inline fuse_u32x4 fuse_seg8(fuse_u32x4 v, float s, float t, bool ok) {
  fuse_u32x4 o;
#pragma unroll
  for (int r = 0; r < 4; ++r) o[r] = fuse_pair(v[r], s, t, ok, ok);
  return o;
}

// one element (low 16 bits of v)
__device__ inline uint16_t fuse_one(uint32_t v, float s, float t, bool ok) {
  return static_cast<uint16_t>(fuse_pair(v & 0xffffu, s, t, ok, false));
}

// the prologue of one widened bf16 value, returned widened again
__device__ inline float fuse_value(float x, float s, float t) {
  const float u = fuse_silu(__builtin_fmaf(x, s, t));
  const uint32_t r = __builtin_bit_cast(uint32_t, __builtin_convertvector((fuse_f32x2{u, 0.f}), fuse_bf16x2));
  return __uint_as_float(r << 16);
}

// bf16 bits -> fp32
__device__ inline float fuse_widen(uint32_t b16) { return __uint_as_float(b16 << 16); }

}  // namespace c3c
