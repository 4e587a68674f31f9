// GEMM family for the encoder: C[M,N] = sum_k A(m,k) B(n,k), with fused epilogues.
//
// One kernel template covers the three operand layouts the encoder needs:
//   forward Linear      Y  = X W^T       A [M][K],  B [N][K]   (both K-contiguous)
//   input gradient      dX = dY W        A [M][K],  B [K][N]   (B K-major)
//   weight gradient     dW = dY^T X      A [K][M],  B [K][N]   (both K-major)
// K-major tiles are transposed in registers on their way into LDS, so the
// MFMA fragment reads are always 16-byte, K-contiguous and bank-conflict free.
//
// Tiling (gfx950): 256 threads = 4 wave64 in a 2x2 grid, block tile 128x128,
// K step 64 (bf16) / 32 (fp32), each wave owns a 64x64 tile of 4x4 16x16
// accumulators.  bf16 uses v_mfma_f32_16x16x32_bf16; fp32 uses
// v_mfma_f32_16x16x4_f32 (eight per 32-wide K step).  LDS is double-buffered
// (64 KB); the next tile's global loads are in flight during the MFMAs.
// Blocks are remapped so that consecutive tiles land on the same XCD and walk
// the output in groups of 8 tile-rows (L2 reuse of A rows and B columns).
#include "common.h"
#include "internal.h"

namespace mpipe {
namespace {

constexpr int BM = 128, BN = 128, NTHR = 256, GROUP_M = 8;

template <class T> struct KStep;
template <> struct KStep<bf16> { static constexpr int BK = 64; static constexpr int VEC = 8; };
template <> struct KStep<float> { static constexpr int BK = 32; static constexpr int VEC = 4; };

struct Regs4 { uint4 v[4]; };

// ---- global -> registers ----------------------------------------------------

// K-contiguous operand X[rows][ld]: tile rows r0..r0+127, k in [k0, k0+BK).
// Thread t loads chunk (t & 7) of rows (t >> 3) + 32 i.
template <class T>
__device__ __forceinline__ void load_kcontig(Regs4& R, const T* X, int64_t ld, int rows, int r0,
                                             int k0, int kend) {
  constexpr int VEC = KStep<T>::VEC;
  const int t = threadIdx.x;
  const int c = t & 7;
  const int k = k0 + c * VEC;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int row = r0 + (t >> 3) + 32 * i;
    row = row < rows ? row : rows - 1;
    if (k < kend)
      R.v[i] = *reinterpret_cast<const uint4*>(X + (int64_t)row * ld + k);
    else
      R.v[i] = make_uint4(0, 0, 0, 0);
  }
}

// K-major operand X[k][ld] (columns contiguous): tile cols c0..c0+127, k in
// [k0, k0+BK).  bf16: thread t loads 4 k-rows x 8 cols (cb = t & 15, kq = t >> 4);
// fp32: 4 k-rows x 4 cols (cb = t & 31, kq = t >> 5).
template <class T>
__device__ __forceinline__ void load_kmajor(Regs4& R, const T* X, int64_t ld, int cols, int c0,
                                            int k0, int kend) {
  constexpr int VEC = KStep<T>::VEC;
  constexpr int NCB = 128 / VEC;
  const int t = threadIdx.x;
  const int cb = t % NCB, kq = t / NCB;
  const int col = c0 + cb * VEC;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int k = k0 + 4 * kq + j;
    if (k < kend && col < cols)
      R.v[j] = *reinterpret_cast<const uint4*>(X + (int64_t)k * ld + col);
    else
      R.v[j] = make_uint4(0, 0, 0, 0);
  }
}

// ---- registers -> LDS ([row][BK] tiles, 128-byte rows, swizzled chunks) -------

__device__ __forceinline__ void store_kcontig(uint4* lds, const Regs4& R) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 4; ++i) lds[swz((t >> 3) + 32 * i, t & 7)] = R.v[i];
}

template <class T> __device__ __forceinline__ void store_kmajor(uint4* lds, const Regs4& R);

template <> __device__ __forceinline__ void store_kmajor<bf16>(uint4* lds, const Regs4& R) {
  // 4 k-rows x 8 cols -> 8 rows (one per col) of 4 k values (8 bytes each)
  const int t = threadIdx.x;
  const int cb = t & 15, kq = t >> 4;
  uint2* l2 = reinterpret_cast<uint2*>(lds);
  const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&R.v[0]);
  const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&R.v[1]);
  const uint32_t* r2 = reinterpret_cast<const uint32_t*>(&R.v[2]);
  const uint32_t* r3 = reinterpret_cast<const uint32_t*>(&R.v[3]);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int p = i >> 1;
    uint2 v;
    if (i & 1) {
      v.x = pack_hi(r0[p], r1[p]);
      v.y = pack_hi(r2[p], r3[p]);
    } else {
      v.x = pack_lo(r0[p], r1[p]);
      v.y = pack_lo(r2[p], r3[p]);
    }
    const int row = cb * 8 + i;
    l2[swz(row, kq >> 1) * 2 + (kq & 1)] = v;
  }
}

template <> __device__ __forceinline__ void store_kmajor<float>(uint4* lds, const Regs4& R) {
  // 4 k-rows x 4 cols -> 4 rows (one per col) of 4 k values (one 16-byte chunk)
  const int t = threadIdx.x;
  const int cb = t & 31, kq = t >> 5;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint4 v;
    v.x = (&R.v[0].x)[i];
    v.y = (&R.v[1].x)[i];
    v.z = (&R.v[2].x)[i];
    v.w = (&R.v[3].x)[i];
    lds[swz(cb * 4 + i, kq)] = v;
  }
}

// ---- MFMA on one LDS stage -------------------------------------------------------

template <class T> struct Mma;

template <> struct Mma<bf16> {
  // two 32-wide K steps per 64-wide stage
  static __device__ __forceinline__ void run(const uint4* As, const uint4* Bs, int wm, int wn,
                                             f32x4 (&acc)[4][4]) {
    const int l = threadIdx.x & 63;
    const int g = l >> 4, r = l & 15;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      bf16x8 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint4 va = As[swz(wm * 64 + 16 * i + r, kk * 4 + g)];
        uint4 vb = Bs[swz(wn * 64 + 16 * i + r, kk * 4 + g)];
        a[i] = *reinterpret_cast<bf16x8*>(&va);
        b[i] = *reinterpret_cast<bf16x8*>(&vb);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
};

template <> struct Mma<float> {
  // one 32-wide K step: lane group g holds k = 8g..8g+7 (two chunks); the eight
  // 16x16x4 MFMAs take slot s = those k's in order (same mapping for A and B).
  static __device__ __forceinline__ void run(const uint4* As, const uint4* Bs, int wm, int wn,
                                             f32x4 (&acc)[4][4]) {
    const int l = threadIdx.x & 63;
    const int g = l >> 4, r = l & 15;
    float a[4][8], b[4][8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ra = wm * 64 + 16 * i + r, rb = wn * 64 + 16 * i + r;
      uint4 a0 = As[swz(ra, 2 * g)], a1 = As[swz(ra, 2 * g + 1)];
      uint4 b0 = Bs[swz(rb, 2 * g)], b1 = Bs[swz(rb, 2 * g + 1)];
      const float* pa0 = reinterpret_cast<const float*>(&a0);
      const float* pa1 = reinterpret_cast<const float*>(&a1);
      const float* pb0 = reinterpret_cast<const float*>(&b0);
      const float* pb1 = reinterpret_cast<const float*>(&b1);
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        a[i][s] = pa0[s];
        a[i][s + 4] = pa1[s];
        b[i][s] = pb0[s];
        b[i][s + 4] = pb1[s];
      }
    }
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][s], b[j][s], acc[i][j], 0, 0, 0);
  }
};

// ---- epilogues -------------------------------------------------------------------

template <class T, int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs& p, int split, int m0, int n0,
                                         f32x4 (&acc)[4][4]) {
  const int l = threadIdx.x & 63;
  const int g = l >> 4, r = l & 15;
  const T* bias = reinterpret_cast<const T*>(p.bias);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = n0 + 16 * j + r;
    if (n >= p.N) continue;
    const float bv = (bias != nullptr && split == 0) ? to_f(bias[n]) : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = m0 + 16 * i + 4 * g + v;
        if (m >= p.M) continue;
        const float x = acc[i][j][v] + bv;
        if constexpr (EPI == EPI_STORE) {
          reinterpret_cast<T*>(p.C)[(int64_t)m * p.ldc + n] = from_f<T>(x);
        } else if constexpr (EPI == EPI_GELU) {
          if (p.C2) reinterpret_cast<T*>(p.C2)[(int64_t)m * p.ldc2 + n] = from_f<T>(x);
          // GELU of the stored (rounded) pre-activation, so the backward sees the
          // same value the forward used
          const float u = to_f(from_f<T>(x));
          reinterpret_cast<T*>(p.C)[(int64_t)m * p.ldc + n] = from_f<T>(gelu_f(u));
        } else if constexpr (EPI == EPI_RESID) {
          const float* R = reinterpret_cast<const float*>(p.aux);
          const float base = R ? R[(int64_t)m * p.ld_aux + n] : 0.0f;
          reinterpret_cast<float*>(p.C)[(int64_t)m * p.ldc + n] = base + x;
        } else if constexpr (EPI == EPI_GELU_BWD) {
          const float u = to_f(reinterpret_cast<const T*>(p.aux)[(int64_t)m * p.ld_aux + n]);
          reinterpret_cast<T*>(p.C)[(int64_t)m * p.ldc + n] = from_f<T>(x * gelu_grad_f(u));
        } else {  // EPI_F32: fp32 output (split-K partial slice, or accumulate)
          float* C = reinterpret_cast<float*>(p.C) + (int64_t)split * p.split_stride;
          const int64_t o = (int64_t)m * p.ldc + n;
          C[o] = p.beta ? C[o] + x : x;
        }
      }
    }
  }
}

// ---- the kernel ------------------------------------------------------------------

template <class T, bool AK, bool BKM, int EPI>
__global__ __launch_bounds__(NTHR, 2) void gemm_kernel(GemmArgs p) {
  constexpr int BK = KStep<T>::BK;
  __shared__ uint4 lds_a[2][BM * 8];
  __shared__ uint4 lds_b[2][BN * 8];

  // XCD-aware block order: the hardware deals consecutive block ids round-robin
  // to the 8 XCDs; undo that so each XCD works on a contiguous run of tiles.
  const int ntiles = p.tiles_m * p.tiles_n;
  const int nb = gridDim.x;  // multiple of 8
  const int b = blockIdx.x;
  const int pid = (b % 8) * (nb / 8) + (b / 8);
  if (pid >= ntiles) return;
  const int group = pid / (GROUP_M * p.tiles_n);
  const int first_m = group * GROUP_M;
  const int gsize = min(p.tiles_m - first_m, GROUP_M);
  const int tm = first_m + (pid % gsize);
  const int tn = (pid % (GROUP_M * p.tiles_n)) / gsize;
  const int split = blockIdx.y;

  const int m0 = tm * BM, n0 = tn * BN;
  const int kbeg = split * p.kps;
  const int kend = min(p.K, kbeg + p.kps);
  const int nk = (kend - kbeg + BK - 1) / BK;

  const T* A = reinterpret_cast<const T*>(p.A);
  const T* B = reinterpret_cast<const T*>(p.B);
  const int w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  Regs4 ra, rb;
  auto gload = [&](int k0) {
    if constexpr (AK) load_kmajor<T>(ra, A, p.lda, p.M, m0, k0, kend);
    else load_kcontig<T>(ra, A, p.lda, p.M, m0, k0, kend);
    if constexpr (BKM) load_kmajor<T>(rb, B, p.ldb, p.N, n0, k0, kend);
    else load_kcontig<T>(rb, B, p.ldb, p.N, n0, k0, kend);
  };
  auto lstore = [&](int buf) {
    if constexpr (AK) store_kmajor<T>(lds_a[buf], ra);
    else store_kcontig(lds_a[buf], ra);
    if constexpr (BKM) store_kmajor<T>(lds_b[buf], rb);
    else store_kcontig(lds_b[buf], rb);
  };

  if (nk > 0) {
    gload(kbeg);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int cur = kt & 1;
      if (kt + 1 < nk) gload(kbeg + (kt + 1) * BK);
      Mma<T>::run(lds_a[cur], lds_b[cur], wm, wn, acc);
      if (kt + 1 < nk) lstore(cur ^ 1);
      __syncthreads();
    }
  }
  epilogue<T, EPI>(p, split, m0 + wm * 64, n0 + wn * 64, acc);
}

// =====================================================================================
// Large-tile bf16 kernel: 256 threads = 4 wave64 (2x2), block tile 256x256, K step 64,
// each wave owns a 128x128 tile of 4x4 v_mfma_f32_32x32x16_bf16 accumulators (in
// AGPRs).  A 128x128 wave tile needs ~94 B/clk/CU of LDS reads+writes at the full
// MFMA rate, under what the LDS delivers; 64x64 wave tiles would need ~128 B/clk.
// LDS: two stages of two 256x64 tiles (128 KB).  The epilogue stages each wave's
// accumulators through LDS, 32 rows at a time, so every global access of the
// epilogue (bias, residual, GELU aux, outputs) is a 16-byte coalesced vector.
// =====================================================================================
namespace big {

constexpr int BM = 256, BN = 256, BK = 64, NTHR = 256;
constexpr int SP = 136;   // staging row pitch in floats: rows 4 apart land 32 banks apart

struct Regs8 { uint4 v[8]; };

__device__ __forceinline__ void load_kc(Regs8& R, const bf16* X, int64_t ld, int rows, int r0,
                                        int k0, int kend) {
  // branch-free: the address is clamped into the operand and a K tail is zeroed
  const int t = threadIdx.x;
  const int k = k0 + (t & 7) * 8;
  const bool ok = k < kend;
  const int kc = ok ? k : kend - 8;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    int row = r0 + (t >> 3) + 32 * i;
    row = row < rows ? row : rows - 1;
    const uint4 v = *reinterpret_cast<const uint4*>(X + (int64_t)row * ld + kc);
    R.v[i] = ok ? v : make_uint4(0, 0, 0, 0);
  }
}
__device__ __forceinline__ void store_kc(uint4* lds, const Regs8& R) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 8; ++i) lds[swz((t >> 3) + 32 * i, t & 7)] = R.v[i];
}
// K-major [k][cols]: sub-blocks of 4 k-rows x 8 columns; cb = t & 31, kq = (t >> 5) + 8 i.
// Branch-free: rows past kend and columns past `cols` read a clamped address and are zeroed.
__device__ __forceinline__ void load_km(Regs8& R, const bf16* X, int64_t ld, int cols, int c0,
                                        int k0, int kend) {
  const int t = threadIdx.x;
  const int col = c0 + (t & 31) * 8;
  const bool cok = col < cols;
  const int cc = cok ? col : 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int kq = (t >> 5) + 8 * i;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = k0 + 4 * kq + j;
      const bool ok = cok && k < kend;
      const int kk = k < kend ? k : kend - 1;
      const uint4 v = *reinterpret_cast<const uint4*>(X + (int64_t)kk * ld + cc);
      R.v[4 * i + j] = ok ? v : make_uint4(0, 0, 0, 0);
    }
  }
}
__device__ __forceinline__ void store_km(uint4* lds, const Regs8& R) {
  const int t = threadIdx.x;
  const int cb = t & 31;
  uint2* l2 = reinterpret_cast<uint2*>(lds);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int kq = (t >> 5) + 8 * i;
    const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&R.v[4 * i + 0]);
    const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&R.v[4 * i + 1]);
    const uint32_t* r2 = reinterpret_cast<const uint32_t*>(&R.v[4 * i + 2]);
    const uint32_t* r3 = reinterpret_cast<const uint32_t*>(&R.v[4 * i + 3]);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int pw = e >> 1;
      uint2 v;
      if (e & 1) {
        v.x = pack_hi(r0[pw], r1[pw]);
        v.y = pack_hi(r2[pw], r3[pw]);
      } else {
        v.x = pack_lo(r0[pw], r1[pw]);
        v.y = pack_lo(r2[pw], r3[pw]);
      }
      l2[swz(cb * 8 + e, kq >> 1) * 2 + (kq & 1)] = v;
    }
  }
}

typedef __attribute__((ext_vector_type(16))) float f32x16;

// 8 consecutive outputs (m, n..n+7) through the epilogue, vectorised
template <int EPI>
__device__ __forceinline__ void epi8(const GemmArgs& p, int split, int m, int n, float* v,
                                     bool vec) {
  const bf16* bias = reinterpret_cast<const bf16*>(p.bias);
  if (vec) {
    if (bias != nullptr && split == 0) {
      const uint4 bb = *reinterpret_cast<const uint4*>(bias + n);
      const bf16* b8 = reinterpret_cast<const bf16*>(&bb);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += (float)b8[e];
    }
    if constexpr (EPI == EPI_STORE || EPI == EPI_GELU || EPI == EPI_GELU_BWD) {
      bf16 o[8];
      if constexpr (EPI == EPI_STORE) {
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (bf16)v[e];
      } else if constexpr (EPI == EPI_GELU) {
        bf16 pre[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          pre[e] = (bf16)v[e];
          o[e] = (bf16)gelu_f((float)pre[e]);
        }
        if (p.C2)
          *reinterpret_cast<uint4*>(reinterpret_cast<bf16*>(p.C2) + (int64_t)m * p.ldc2 + n) =
              *reinterpret_cast<const uint4*>(pre);
      } else {
        const uint4 uu = *reinterpret_cast<const uint4*>(reinterpret_cast<const bf16*>(p.aux) +
                                                         (int64_t)m * p.ld_aux + n);
        const bf16* u8 = reinterpret_cast<const bf16*>(&uu);
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (bf16)(v[e] * gelu_grad_f((float)u8[e]));
      }
      *reinterpret_cast<uint4*>(reinterpret_cast<bf16*>(p.C) + (int64_t)m * p.ldc + n) =
          *reinterpret_cast<const uint4*>(o);
    } else if constexpr (EPI == EPI_RESID) {
      const float* R = reinterpret_cast<const float*>(p.aux);
      float4 r0 = make_float4(0.f, 0.f, 0.f, 0.f), r1 = r0;
      if (R) {
        r0 = *reinterpret_cast<const float4*>(R + (int64_t)m * p.ld_aux + n);
        r1 = *reinterpret_cast<const float4*>(R + (int64_t)m * p.ld_aux + n + 4);
      }
      float* C = reinterpret_cast<float*>(p.C) + (int64_t)m * p.ldc + n;
      *reinterpret_cast<float4*>(C) = make_float4(r0.x + v[0], r0.y + v[1], r0.z + v[2], r0.w + v[3]);
      *reinterpret_cast<float4*>(C + 4) = make_float4(r1.x + v[4], r1.y + v[5], r1.z + v[6], r1.w + v[7]);
    } else {  // EPI_F32
      float* C = reinterpret_cast<float*>(p.C) + (int64_t)split * p.split_stride +
                 (int64_t)m * p.ldc + n;
      float4 a = make_float4(v[0], v[1], v[2], v[3]), b = make_float4(v[4], v[5], v[6], v[7]);
      if (p.beta) {
        const float4 c0 = *reinterpret_cast<const float4*>(C);
        const float4 c1 = *reinterpret_cast<const float4*>(C + 4);
        a.x += c0.x; a.y += c0.y; a.z += c0.z; a.w += c0.w;
        b.x += c1.x; b.y += c1.y; b.z += c1.z; b.w += c1.w;
      }
      *reinterpret_cast<float4*>(C) = a;
      *reinterpret_cast<float4*>(C + 4) = b;
    }
    return;
  }
  // scalar tail (ragged N or unaligned strides)
  for (int e = 0; e < 8; ++e) {
    const int nn = n + e;
    if (nn >= p.N) break;
    float x = v[e] + ((bias != nullptr && split == 0) ? (float)bias[nn] : 0.f);
    if constexpr (EPI == EPI_STORE) {
      reinterpret_cast<bf16*>(p.C)[(int64_t)m * p.ldc + nn] = (bf16)x;
    } else if constexpr (EPI == EPI_GELU) {
      const bf16 pre = (bf16)x;
      if (p.C2) reinterpret_cast<bf16*>(p.C2)[(int64_t)m * p.ldc2 + nn] = pre;
      reinterpret_cast<bf16*>(p.C)[(int64_t)m * p.ldc + nn] = (bf16)gelu_f((float)pre);
    } else if constexpr (EPI == EPI_RESID) {
      const float* R = reinterpret_cast<const float*>(p.aux);
      const float base = R ? R[(int64_t)m * p.ld_aux + nn] : 0.f;
      reinterpret_cast<float*>(p.C)[(int64_t)m * p.ldc + nn] = base + x;
    } else if constexpr (EPI == EPI_GELU_BWD) {
      const float u = (float)reinterpret_cast<const bf16*>(p.aux)[(int64_t)m * p.ld_aux + nn];
      reinterpret_cast<bf16*>(p.C)[(int64_t)m * p.ldc + nn] = (bf16)(x * gelu_grad_f(u));
    } else {
      float* C = reinterpret_cast<float*>(p.C) + (int64_t)split * p.split_stride;
      const int64_t o = (int64_t)m * p.ldc + nn;
      C[o] = p.beta ? C[o] + x : x;
    }
  }
}

template <bool AK, bool BKM, int EPI>
__global__ __launch_bounds__(NTHR, 1) void gemm_big_kernel(GemmArgs p) {
  // one 128 KB array: stages [A0 | A1 | B0 | B1], reused by the epilogue staging
  __shared__ uint4 smem[2 * (BM + BN) * 8];
  auto lds_a = [&](int buf) { return smem + buf * (BM * 8); };
  auto lds_b = [&](int buf) { return smem + 2 * BM * 8 + buf * (BN * 8); };
  const int ntiles = p.tiles_m * p.tiles_n;
  const int nb = gridDim.x;
  const int b = blockIdx.x;
  const int pid = (b % 8) * (nb / 8) + (b / 8);
  if (pid >= ntiles) return;
  const int group = pid / (GROUP_M * p.tiles_n);
  const int first_m = group * GROUP_M;
  const int gsize = min(p.tiles_m - first_m, GROUP_M);
  const int tm = first_m + (pid % gsize);
  const int tn = (pid % (GROUP_M * p.tiles_n)) / gsize;
  const int split = blockIdx.y;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kbeg = split * p.kps;
  const int kend = min(p.K, kbeg + p.kps);
  const int nk = (kend - kbeg + BK - 1) / BK;
  const bf16* A = reinterpret_cast<const bf16*>(p.A);
  const bf16* B = reinterpret_cast<const bf16*>(p.B);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int wm = w >> 1, wn = w & 1;

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  Regs8 ra, rb;
  auto gload = [&](int k0) {
    if constexpr (AK) load_km(ra, A, p.lda, p.M, m0, k0, kend);
    else load_kc(ra, A, p.lda, p.M, m0, k0, kend);
    if constexpr (BKM) load_km(rb, B, p.ldb, p.N, n0, k0, kend);
    else load_kc(rb, B, p.ldb, p.N, n0, k0, kend);
  };
  auto lstore = [&](int buf) {
    if constexpr (AK) store_km(lds_a(buf), ra);
    else store_kc(lds_a(buf), ra);
    if constexpr (BKM) store_km(lds_b(buf), rb);
    else store_kc(lds_b(buf), rb);
  };
  // fragments of one 16-wide K sub-step: rows wm*128 + 32i + (l & 31), chunk 2s + (l >> 5)
  auto frags = [&](const uint4* As, const uint4* Bs, int s, bf16x8 (&fa)[4], bf16x8 (&fb)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint4 va = As[swz(wm * 128 + 32 * i + (l & 31), 2 * s + (l >> 5))];
      uint4 vb = Bs[swz(wn * 128 + 32 * i + (l & 31), 2 * s + (l >> 5))];
      fa[i] = *reinterpret_cast<bf16x8*>(&va);
      fb[i] = *reinterpret_cast<bf16x8*>(&vb);
    }
  };
  if (nk > 0) {
    gload(kbeg);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int cur = kt & 1;
      const bool more = kt + 1 < nk;
      const uint4* As = lds_a(cur);
      const uint4* Bs = lds_b(cur);
      bf16x8 fa[2][4], fb[2][4];
      frags(As, Bs, 0, fa[0], fb[0]);
      if (more) gload(kbeg + (kt + 1) * BK);
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        if (s < 3) frags(As, Bs, s + 1, fa[(s + 1) & 1], fb[(s + 1) & 1]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s & 1][i], fb[s & 1][j],
                                                                acc[i][j], 0, 0, 0);
        // interleave the next sub-step's LDS reads with this sub-step's 16 MFMAs
        if (s < 3) {
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);   // MFMA
          }
        }
      }
      if (more) lstore(cur ^ 1);
      __syncthreads();
    }
  }
  // epilogue: per m-subtile i, stage the wave's 32x128 block through LDS
  static_assert(4 * 32 * SP * 4 <= 2 * (BM + BN) * 8 * 16, "epilogue staging must fit in LDS");
  float* stage = reinterpret_cast<float*>(smem) + w * (32 * SP);
#pragma unroll
  for (int i = 0; i < 4; ++i) {   // (acc[i] must be indexed statically)
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int rr = 8 * (e >> 2) + 4 * (l >> 5) + (e & 3);
        stage[rr * SP + 32 * j + (l & 31)] = acc[i][j][e];
      }
    __syncthreads();
    const int cg = l & 15;
#pragma unroll 1
    for (int u = 0; u < 8; ++u) {
      const int rr = (l >> 4) + 4 * u;
      const int m = m0 + wm * 128 + 32 * i + rr;
      const int n = n0 + wn * 128 + 8 * cg;
      if (m >= p.M || n >= p.N) continue;
      float v[8];
      const float4 x0 = *reinterpret_cast<const float4*>(stage + rr * SP + 8 * cg);
      const float4 x1 = *reinterpret_cast<const float4*>(stage + rr * SP + 8 * cg + 4);
      v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w;
      v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
      epi8<EPI>(p, split, m, n, v, p.vec && n + 8 <= p.N);
    }
  }
}

template <bool AK, bool BKM, int EPI>
hipError_t launch_big(const GemmArgs& a0, hipStream_t s) {
  GemmArgs a = a0;
  a.tiles_m = (a.M + BM - 1) / BM;
  a.tiles_n = (a.N + BN - 1) / BN;
  const int nt = a.tiles_m * a.tiles_n;
  const int nb = (nt + 7) / 8 * 8;
  int splits = a.kps > 0 ? (a.K + a.kps - 1) / a.kps : 1;
  if (a.kps <= 0) a.kps = a.K;
  if (splits < 1) splits = 1;
  hipLaunchKernelGGL((gemm_big_kernel<AK, BKM, EPI>), dim3(nb, splits), dim3(NTHR), 0, s, a);
  return hipGetLastError();
}

template <bool AK, bool BKM>
hipError_t dispatch_big(const GemmArgs& a, int epi, hipStream_t s) {
  switch (epi) {
    case EPI_STORE: return launch_big<AK, BKM, EPI_STORE>(a, s);
    case EPI_GELU: return launch_big<AK, BKM, EPI_GELU>(a, s);
    case EPI_RESID: return launch_big<AK, BKM, EPI_RESID>(a, s);
    case EPI_GELU_BWD: return launch_big<AK, BKM, EPI_GELU_BWD>(a, s);
    case EPI_F32: return launch_big<AK, BKM, EPI_F32>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace big

template <class T, bool AK, bool BKM, int EPI>
hipError_t launch(const GemmArgs& a0, hipStream_t s) {
  GemmArgs a = a0;
  a.tiles_m = (a.M + BM - 1) / BM;
  a.tiles_n = (a.N + BN - 1) / BN;
  int nt = a.tiles_m * a.tiles_n;
  int nb = (nt + 7) / 8 * 8;
  int splits = a.kps > 0 ? (a.K + a.kps - 1) / a.kps : 1;
  if (a.kps <= 0) a.kps = a.K;
  if (splits < 1) splits = 1;
  hipLaunchKernelGGL((gemm_kernel<T, AK, BKM, EPI>), dim3(nb, splits), dim3(NTHR), 0, s, a);
  return hipGetLastError();
}

template <class T, bool AK, bool BKM>
hipError_t dispatch_epi(const GemmArgs& a, int epi, hipStream_t s) {
  switch (epi) {
    case EPI_STORE: return launch<T, AK, BKM, EPI_STORE>(a, s);
    case EPI_GELU: return launch<T, AK, BKM, EPI_GELU>(a, s);
    case EPI_RESID: return launch<T, AK, BKM, EPI_RESID>(a, s);
    case EPI_GELU_BWD: return launch<T, AK, BKM, EPI_GELU_BWD>(a, s);
    case EPI_F32: return launch<T, AK, BKM, EPI_F32>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

// Host entry: layout = NT (fwd), NN (dX) or TN (dW); requirements checked by the caller:
// K-contiguous operands need K % VEC == 0 and ld % VEC == 0; K-major operands need
// their column count and ld to be multiples of VEC; all pointers 16-byte aligned.
hipError_t gemm(int dtype, int layout, int epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (dtype == DT_BF16 && a.M >= 512 && a.N >= 256) {
    GemmArgs b = a;
    // 16-byte vector epilogue when every output/aux row stride keeps 16-byte alignment
    auto al16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
    const bool f32out = epi == EPI_RESID || epi == EPI_F32;
    const int64_t vq = f32out ? 4 : 8;
    b.vec = al16(a.C) && a.ldc % vq == 0 && (a.bias == nullptr || al16(a.bias)) &&
            (a.aux == nullptr || (al16(a.aux) && a.ld_aux % (epi == EPI_RESID ? 4 : 8) == 0)) &&
            (a.C2 == nullptr || (al16(a.C2) && a.ldc2 % 8 == 0));
    switch (layout) {
      case GEMM_NT: return big::dispatch_big<false, false>(b, epi, s);
      case GEMM_NN: return big::dispatch_big<false, true>(b, epi, s);
      case GEMM_TN: return big::dispatch_big<true, true>(b, epi, s);
    }
  }
  if (dtype == DT_BF16) {
    switch (layout) {
      case GEMM_NT: return dispatch_epi<bf16, false, false>(a, epi, s);
      case GEMM_NN: return dispatch_epi<bf16, false, true>(a, epi, s);
      case GEMM_TN: return dispatch_epi<bf16, true, true>(a, epi, s);
    }
  } else {
    switch (layout) {
      case GEMM_NT: return dispatch_epi<float, false, false>(a, epi, s);
      case GEMM_NN: return dispatch_epi<float, false, true>(a, epi, s);
      case GEMM_TN: return dispatch_epi<float, true, true>(a, epi, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace mpipe
