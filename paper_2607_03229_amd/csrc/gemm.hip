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
#include <type_traits>

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
    // rotary columns (q, k) are stored pair-interleaved: bias of the original column
    const bool rot = EPI == EPI_STORE_ROPE && n < p.rope_cols;
    const int nb = rot ? n - n % p.rope_d + rope_component(n % p.rope_d, p.rope_d) : n;
    const float bv = (bias != nullptr && split == 0) ? to_f(bias[nb]) : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = m0 + 16 * i + 4 * g + v;
        if (m >= p.M) continue;
        float x = acc[i][j][v] + bv;
        if constexpr (EPI == EPI_STORE || EPI == EPI_STORE_ROPE) {
          if (rot) {   // the pair partner (column n ^ 1, same row) is in lane l ^ 1
            const float y = __shfl_xor(x, 1);
            const float2 cs = rope_cs(p.rope_pos, p.rope_tab, p.rope_d, m, (n % p.rope_d) >> 1);
            x = (n & 1) ? rope_second(y, x, cs, false) : rope_first(x, y, cs, false);
          }
          reinterpret_cast<T*>(p.C)[(int64_t)m * p.ldc + n] = from_f<T>(x);
        } else if constexpr (EPI == EPI_GELU) {
          // GELU and GELU' at the rounded pre-activation u; the backward multiplies by
          // the stored GELU'(u)
          const float u = to_f(from_f<T>(x));
          const bool fast = std::is_same<T, bf16>::value;
          const float gv = fast ? gelu_fast(u) : gelu_f(u);
          if (p.C2)
            reinterpret_cast<T*>(p.C2)[(int64_t)m * p.ldc2 + n] =
                from_f<T>(fast ? gelu_grad_fast(u) : gelu_grad_f(u));
          reinterpret_cast<T*>(p.C)[(int64_t)m * p.ldc + n] = from_f<T>(gv);
        } else if constexpr (EPI == EPI_RESID) {
          const float* R = reinterpret_cast<const float*>(p.aux);
          const float base = R ? R[(int64_t)m * p.ld_aux + n] : 0.0f;
          reinterpret_cast<float*>(p.C)[(int64_t)m * p.ldc + n] = base + x;
        } else if constexpr (EPI == EPI_GELU_BWD) {
          const float gg = to_f(reinterpret_cast<const T*>(p.aux)[(int64_t)m * p.ld_aux + n]);
          reinterpret_cast<T*>(p.C)[(int64_t)m * p.ldc + n] = from_f<T>(x * gg);
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
    case EPI_STORE_ROPE: return launch<T, AK, BKM, EPI_STORE_ROPE>(a, s);
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
namespace {
// The big kernels (bf16, M >= 512, N >= 256) have 16-byte vector epilogues only: every
// output/aux row stride must keep 16-byte alignment, else the general kernel takes the
// problem.
bool takes_big(int dtype, int epi, const GemmArgs& a) {
  if (!(dtype == DT_BF16 && a.M >= 512 && a.N >= 256 && a.N % 8 == 0)) return false;
  auto al16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
  const bool f32out = epi == EPI_RESID || epi == EPI_F32;
  const int64_t vq = f32out ? 4 : 8;
  return al16(a.C) && a.ldc % vq == 0 && (a.bias == nullptr || al16(a.bias)) &&
         (a.aux == nullptr || (al16(a.aux) && a.ld_aux % (epi == EPI_RESID ? 4 : 8) == 0)) &&
         (a.C2 == nullptr || (al16(a.C2) && a.ldc2 % 8 == 0)) &&
         (epi != EPI_F32 || a.split_stride % 4 == 0);
}
}  // namespace

bool gemm_fused_colsum(int dtype, int layout, int epi, const GemmArgs& a) {
  return layout == GEMM_NN && epi == EPI_GELU_BWD && a.kps <= 0 && takes_big(dtype, epi, a);
}

hipError_t gemm(int dtype, int layout, int epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.colsum && !gemm_fused_colsum(dtype, layout, epi, a)) return hipErrorInvalidValue;
  if (takes_big(dtype, epi, a)) return gemm_big(layout, epi, a, s);
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
