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

// bf16 GELU: standard normal CDF Phi(u) and density phi(u) sharing one
// exp(-u^2/2): erfc(x) = y(t) exp(-x^2), t = 1 / (1 + p x), x = |u| / sqrt(2), with the
// five-term polynomial y of Abramowitz & Stegun 7.1.26 (|error in erf| <= 1.5e-7, far
// below the bf16 rounding of the outputs).  Every bf16 GEMM epilogue uses these, so a
// token's result never depends on which kernel (tile size) computed it; fp32 uses erff.
__device__ __forceinline__ void phi_pair(float u, float& Phi, float& dens) {
  const float x = fabsf(u) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
  const float y = t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f),
                               -0.284496736f), 0.254829592f);
  const float e = __builtin_amdgcn_exp2f(-x * x * 1.4426950408889634f);   // exp(-u^2/2)
  const float tail = 0.5f * y * e;                                           // Phi(-|u|)
  Phi = u >= 0.f ? 1.0f - tail : tail;
  dens = e * 0.3989422804014327f;
}
__device__ __forceinline__ float gelu_fast(float u) {
  float P, d;
  phi_pair(u, P, d);
  return u * P;
}
__device__ __forceinline__ float gelu_grad_fast(float u) {
  float P, d;
  phi_pair(u, P, d);
  return fmaf(u, d, P);
}

// ---- 2D rotary position on pair-interleaved q / k columns ----------------------------
// The encoder stores the q and k columns of every head pair-interleaved: stored column 2j
// of a head holds rotary component j and stored column 2j + 1 holds component j + d/2,
// the two components one rotation mixes.  q and k are permuted alike, so attention
// scores are unchanged, and a rotation needs only adjacent values.  pos[row] packs the
// patch position as y << 16 | x; tab[p * d/4 + k] = (cos, sin) of p * theta^(-4k/d).
// Component j < d/4 turns by the angle of y, the others by that of x.

// original head-local component of stored head-local column s
__host__ __device__ __forceinline__ int rope_component(int s, int d) {
  return (s & 1) ? (s >> 1) + (d >> 1) : (s >> 1);
}
// (cos, sin) of rotary pair j (< d/2) of packed row `row`
__device__ __forceinline__ float2 rope_cs(const int32_t* pos, const float2* tab, int d,
                                          int64_t row, int j) {
  const uint32_t pp = (uint32_t)pos[row];
  const int q4 = d >> 2;
  const bool along_y = j < q4;
  const int coord = (int)(along_y ? (pp >> 16) : (pp & 0xFFFFu));
  return tab[coord * q4 + (along_y ? j : j - q4)];
}
// Forward rotation of (a, b) = (x_j, x_{j+d/2}); the backward applies the inverse.
// Written with explicit fmaf so that every kernel and every unrolled copy rounds the
// same way (a row's result must not depend on the tile or lane that computes it):
//   rotate:   a' = fma(a, c, -(b s)),  b' = fma(b, c, a s)
//   unrotate: a' = fma(a, c, b s),     b' = fma(b, c, -(a s))
__device__ __forceinline__ float rope_first(float a, float b, float2 cs, bool inverse) {
  const float bs = b * cs.y;
  return fmaf(a, cs.x, inverse ? bs : -bs);
}
__device__ __forceinline__ float rope_second(float a, float b, float2 cs, bool inverse) {
  const float as = a * cs.y;
  return fmaf(b, cs.x, inverse ? -as : as);
}
__device__ __forceinline__ void rope_rotate(float& a, float& b, float2 cs) {
  const float a0 = a;
  a = rope_first(a0, b, cs, false);
  b = rope_second(a0, b, cs, false);
}
__device__ __forceinline__ void rope_unrotate(float& a, float& b, float2 cs) {
  const float a0 = a;
  a = rope_first(a0, b, cs, true);
  b = rope_second(a0, b, cs, true);
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
