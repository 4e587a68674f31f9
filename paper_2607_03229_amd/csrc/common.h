// Device-side helpers shared by the gfx950 kernels of libmpipe.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpipe {

typedef __bf16 bf16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <class T> __device__ __forceinline__ float to_f(T v) { return (float)v; }
template <class T> __device__ __forceinline__ T from_f(float v) { return (T)v; }

// 16-byte chunk index swizzle for LDS tiles whose rows are 128 bytes (8 chunks).
// XOR-ing the chunk with bits 0-2 and 3-5 of the row makes both the 16-row
// MFMA fragment reads and the row-wise tile stores bank-conflict free.
__device__ __forceinline__ int swz(int row, int chunk) {
  return row * 8 + (chunk ^ ((row ^ (row >> 3)) & 7));
}

// exact GELU (erf form) and its derivative
__device__ __forceinline__ float gelu_f(float u) {
  return 0.5f * u * (1.0f + erff(u * 0.7071067811865476f));
}
__device__ __forceinline__ float gelu_grad_f(float u) {
  const float Phi = 0.5f * (1.0f + erff(u * 0.7071067811865476f));
  const float phi = 0.3989422804014327f * __expf(-0.5f * u * u);
  return Phi + u * phi;
}

// bf16 pair packing helpers on 32-bit words (low half = first element)
__device__ __forceinline__ uint32_t pack_lo(uint32_t a, uint32_t b) {  // a.lo | b.lo << 16
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ __forceinline__ uint32_t pack_hi(uint32_t a, uint32_t b) {  // a.hi | b.hi << 16
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

__device__ __forceinline__ float warp_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float warp_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

}  // namespace mpipe
