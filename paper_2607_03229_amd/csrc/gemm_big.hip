// Large-tile bf16 GEMMs for gfx950: the encoder's Linear layers at full size.
//
// C[M,N] = sum_k A(m,k) B(n,k) with the same operand layouts and epilogues as the
// general kernel (NT forward, NN input gradient, TN weight gradient).
//
// Three kernels, all 256 threads = 4 wave64 in a 2x2 grid of v_mfma_f32_32x32x16_bf16
// accumulators with the same K order, so a given output element gets bitwise the same
// value from any of them:
//   gemm_big_kernel (TN): block tile 256x256, each wave 128x128 (4x4 accumulators,
//     256 AGPRs), a 4-stage ring (128 KB of LDS), one block per CU.  A 128x128 wave tile
//     keeps the LDS traffic (fragment reads + tile fills) well under what the LDS
//     delivers at the full MFMA rate.
//   gemm_nt64_kernel (NT, described with it below): the same block with 64-deep K stages.
//   gemm_nn_kernel (NN, described with it below): block tile 128x256, two blocks per CU.
//
// Operand tiles (rows x 32 k) are filled by 16-byte global->LDS DMA (global_load_lds)
// in a ring, so the next tiles are in flight while tile t is multiplied and no tile
// data passes through VGPRs.  Each lane of a DMA instruction owns one fixed LDS slot and
// picks the source element of that slot, which is how the tiles get their
// bank-conflict-free XOR swizzles:
//   K-contiguous operand ([rows][k]): 64-byte rows, chunk c of row r at c ^ fkc(r);
//      fragment reads are 16-byte ds_read_b128.
//   K-major operand ([k][cols], 256 cols): 512-byte k-rows, chunk c of k-row k at
//      c ^ gkm(k); fragments come straight from the raw tile through
//      ds_read_b64_tr_b16, so no operand is ever transposed in registers.
// Both swizzles keep every fragment read conflict-free whether the LDS serves 128
// or 256 bytes per cycle.
//
// Pipeline per K tile t: the fragments of its first 16-wide K half are already in
// registers; the second half's fragments are read while the first half's MFMAs run;
// then one barrier (tile t+1 landed for every wave, stage t no longer read), the DMA
// of tile t+NST into stage t, and tile t+1's first fragments are read while the second
// half's MFMAs run.  Ragged M/N edges read clamped (valid) rows; a ragged K tail reads
// clamped rows and zeroes the A fragments past the end.  The epilogue stages each
// wave's accumulators through its own LDS region, 16 rows at a time, so all epilogue
// global accesses are 16-byte vectors (the dispatcher sends ragged-N or misaligned
// problems to the general kernel); the operands it reads (GELU' factor, residual,
// accumulate target) are fetched one staging pass ahead.
#include <type_traits>

#include "common.h"
#include "internal.h"

// (the DMA assembly declares the reserved register M0 clobbered, which clang reports)
#pragma clang diagnostic ignored "-Winline-asm"

namespace mpipe {
namespace {

constexpr int BN = 256, BK = 32, NTHR = 256, GROUP_M = 8;
constexpr int B_U4 = BN * BK * 2 / 16;      // 16-byte slots of a B operand tile (1024)
constexpr int SP = 136;                     // epilogue staging pitch in floats

typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// chunk swizzle of a K-contiguous tile (4 chunks per 64-byte row): bit1 = r2, bit0 = r1^r3
__device__ __forceinline__ int fkc(int r) { return ((r >> 1) & 2) | (((r >> 1) ^ (r >> 3)) & 1); }
// chunk swizzle of a K-major tile (32 chunks per 512-byte k-row), by k mod 4: 0, 10, 4, 14
__device__ __forceinline__ int gkm(int k) { return ((k & 1) ? 10 : 0) ^ ((k & 2) ? 4 : 0); }

// The DMAs, and the waits for them, are issued as inline assembly that the compiler
// does not track: it then inserts no waits of its own for them (its conservative
// vmcnt(0) before fragment reads would drain the ring once per pass of the loop).
// This is safe because the main loop has no other vector-memory instructions and
// every DMA is waited for (wait_vm<0>) before the epilogue's loads.
template <int n>
__device__ __forceinline__ void wait_vm() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(n) : "memory");
}
// Barrier after this wave's LDS reads have completed; no fence for the DMAs in flight.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
// Orders this wave's LDS writes before its later LDS reads (a wave's LDS operations
// execute in issue order; the clobber keeps the compiler from moving accesses across).
__device__ __forceinline__ void lds_wave_fence() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(size_t)(lds_void*)p;
}

// ---- DMA sources ---------------------------------------------------------------------
// DMA instruction q of an operand tile fills LDS slots 64q..64q+63, lane l slot 64q + l;
// wave w issues instructions q = n*w .. n*w + n-1 of a tile that takes 4n instructions.

// K-contiguous operand X[rows][ld], tile rows r0.., k from k0: slot (row 16q + l/4,
// physical chunk l%4) holds logical chunk (l%4) ^ fkc(row).
__device__ __forceinline__ const bf16* src_kc(const bf16* X, int64_t ld, int rows, int r0, int k0,
                                              int kend, int q) {
  const int l = threadIdx.x & 63;
  const int row = 16 * q + (l >> 2);
  int k = k0 + 8 * ((l & 3) ^ fkc(row));
  k = k < kend ? k : kend - 8;
  int gr = r0 + row;
  gr = gr < rows ? gr : rows - 1;
  return X + (int64_t)gr * ld + k;
}
// K-major operand X[k][ld], 256-col tile from c0, k-rows from k0: slot (k-row 2q + l/32,
// physical chunk l%32) holds logical chunk (l%32) ^ gkm(k-row).
__device__ __forceinline__ const bf16* src_km(const bf16* X, int64_t ld, int cols, int c0, int k0,
                                              int kend, int q) {
  const int l = threadIdx.x & 63;
  const int kr = 2 * q + (l >> 5);
  int col = c0 + 8 * ((l & 31) ^ gkm(kr));
  col = col < cols ? col : cols - 8;
  int k = k0 + kr;
  k = k < kend ? k : kend - 1;
  return X + (int64_t)k * ld + col;
}
// 16-byte global->LDS DMA of instruction q: lane l writes LDS byte tile + 1024 q + 16 l
// (M0 holds the wave-uniform base).
// M0 is declared clobbered; nothing else in these kernels keeps a value in it.
__device__ __forceinline__ void dma16(const bf16* src, const uint4* tile, int q) {
  const uint32_t base = lds_addr(tile) + 1024u * q;
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               ::"v"(src), "s"(__builtin_amdgcn_readfirstlane(base)) : "memory", "m0");
}

// ---- epilogue ------------------------------------------------------------------------

// The vector epilogue works on 8 consecutive outputs (m, n..n+7) of a lane.  Its global
// operands (GELU' factor, residual, accumulate target) are fetched one staging pass
// ahead, so their latency overlaps the previous pass instead of stalling each store.
struct AuxV { uint4 v[2]; };

template <int EPI>
__device__ __forceinline__ void aux_fetch(const GemmArgs& p, int split, int m, int n, AuxV& a) {
  if constexpr (EPI == EPI_GELU_BWD) {
    a.v[0] = *reinterpret_cast<const uint4*>(reinterpret_cast<const bf16*>(p.aux) +
                                             (int64_t)m * p.ld_aux + n);
  } else if constexpr (EPI == EPI_RESID) {
    if (p.aux) {
      const float* R = reinterpret_cast<const float*>(p.aux) + (int64_t)m * p.ld_aux + n;
      a.v[0] = *reinterpret_cast<const uint4*>(R);
      a.v[1] = *reinterpret_cast<const uint4*>(R + 4);
    }
  } else if constexpr (EPI == EPI_F32) {
    if (p.beta) {
      const float* C = reinterpret_cast<const float*>(p.C) + (int64_t)split * p.split_stride +
                       (int64_t)m * p.ldc + n;
      a.v[0] = *reinterpret_cast<const uint4*>(C);
      a.v[1] = *reinterpret_cast<const uint4*>(C + 4);
    }
  } else if constexpr (EPI == EPI_STORE_ROPE) {
    // (cos, sin) of the four rotary pairs of columns n..n+7 at row m: consecutive table
    // entries (a head's d/4 pairs per axis are a multiple of 4, so they share an axis)
    if (n < p.rope_cols) {
      const int q4 = p.rope_d >> 2, j0 = (n % p.rope_d) >> 1;
      const uint32_t pp = (uint32_t)p.rope_pos[m];
      const int coord = (int)(j0 < q4 ? (pp >> 16) : (pp & 0xFFFFu));
      const float2* t = p.rope_tab + coord * q4 + (j0 < q4 ? j0 : j0 - q4);
      a.v[0] = *reinterpret_cast<const uint4*>(t);
      a.v[1] = *reinterpret_cast<const uint4*>(t + 2);
    }
  }
}

// The bias of a lane's eight columns n..n+7 (zeros when `take` is false).  Columns that
// get the fused rotary position are stored pair-interleaved, so their bias entries come
// from the original columns.
__device__ __forceinline__ void load_bias8(const GemmArgs& p, bool take, int n, float* bias8) {
#pragma unroll
  for (int e = 0; e < 8; ++e) bias8[e] = 0.f;
  if (!take || p.bias == nullptr) return;
  const bf16* bias = reinterpret_cast<const bf16*>(p.bias);
  if (p.rope_pos != nullptr && n < p.rope_cols) {   // EPI_STORE_ROPE's q, k columns
    const int base = n - n % p.rope_d, s0 = n % p.rope_d;   // eight columns of one head
#pragma unroll
    for (int e = 0; e < 8; ++e) bias8[e] = (float)bias[base + rope_component(s0 + e, p.rope_d)];
    return;
  }
  const uint4 bb = *reinterpret_cast<const uint4*>(bias + n);
  const bf16* b8 = reinterpret_cast<const bf16*>(&bb);
#pragma unroll
  for (int e = 0; e < 8; ++e) bias8[e] = (float)b8[e];
}

template <int EPI>
__device__ __forceinline__ void epi8_vec(const GemmArgs& p, int split, int m, int n, float* v,
                                         const float* bias8, const AuxV& ax,
                                         float* sum8 = nullptr) {
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] += bias8[e];
  if constexpr (EPI == EPI_STORE || EPI == EPI_STORE_ROPE || EPI == EPI_GELU ||
                EPI == EPI_GELU_BWD) {
    bf16 o[8];
    if constexpr (EPI == EPI_STORE || EPI == EPI_STORE_ROPE) {
      if constexpr (EPI == EPI_STORE_ROPE) {
        if (n < p.rope_cols) {   // q, k: rotate the four pairs by the prefetched angles
          const float2* cs = reinterpret_cast<const float2*>(&ax.v[0]);
#pragma unroll
          for (int e = 0; e < 8; e += 2) rope_rotate(v[e], v[e + 1], cs[e / 2]);
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (bf16)v[e];
    } else if constexpr (EPI == EPI_GELU) {
      // GELU and its derivative at the bf16-rounded pre-activation u, from one Phi/phi
      // evaluation; the derivative is what the backward needs of u
      bf16 gd[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float u = (float)(bf16)v[e];
        float P, dens;
        phi_pair(u, P, dens);
        o[e] = (bf16)(u * P);
        gd[e] = (bf16)fmaf(u, dens, P);
      }
      if (p.C2)
        *reinterpret_cast<uint4*>(reinterpret_cast<bf16*>(p.C2) + (int64_t)m * p.ldc2 + n) =
            *reinterpret_cast<const uint4*>(gd);
    } else {   // EPI_GELU_BWD: aux holds GELU'(u) from the forward
      const bf16* g8 = reinterpret_cast<const bf16*>(&ax.v[0]);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (bf16)(v[e] * (float)g8[e]);
      if (sum8) {   // column sums of what is stored (the next bias gradient)
#pragma unroll
        for (int e = 0; e < 8; ++e) sum8[e] += (float)o[e];
      }
    }
    *reinterpret_cast<uint4*>(reinterpret_cast<bf16*>(p.C) + (int64_t)m * p.ldc + n) =
        *reinterpret_cast<const uint4*>(o);
  } else {   // EPI_RESID, EPI_F32: fp32 out, plus the fetched residual / previous value
    float* C = reinterpret_cast<float*>(p.C) +
               (EPI == EPI_F32 ? (int64_t)split * p.split_stride : 0) + (int64_t)m * p.ldc + n;
    const bool add = EPI == EPI_RESID ? p.aux != nullptr : p.beta != 0;
    const float* r8 = reinterpret_cast<const float*>(&ax.v[0]);
    float4 a = make_float4(v[0], v[1], v[2], v[3]), b = make_float4(v[4], v[5], v[6], v[7]);
    if (add) {
      a.x += r8[0]; a.y += r8[1]; a.z += r8[2]; a.w += r8[3];
      b.x += r8[4]; b.y += r8[5]; b.z += r8[6]; b.w += r8[7];
    }
    *reinterpret_cast<float4*>(C) = a;
    *reinterpret_cast<float4*>(C + 4) = b;
  }
}

// ---- the kernel ----------------------------------------------------------------------

// 256x256 tiles: MT 32-row MFMA tiles per wave in M, NST ring stages, IA / IPT DMA
// instructions per wave for an A tile / a whole K tile.
constexpr int BM = 256, MT = 4, NST = 4;
constexpr int A_U4 = BM * BK * 2 / 16;   // 16-byte slots of an A tile (1024)
constexpr int IA = 4, IPT = IA + 4;
constexpr int BIG_LDS_U4 = NST * (A_U4 + B_U4);

template <bool AK, bool BKM, int EPI>
__global__ __launch_bounds__(NTHR, 1) void gemm_big_kernel(GemmArgs p) {
  // the ring: stage s of A at smem + s*A_U4, of B at smem + NST*A_U4 + s*B_U4.  The DMAs
  // are assembly with a memory clobber, so no fragment read moves across one.
  __shared__ uint4 smem[BIG_LDS_U4];
  static_assert(4 * 16 * SP * 4 <= BIG_LDS_U4 * 16, "epilogue staging must fit in the ring");

  // XCD-aware block order (consecutive block ids go round-robin to the 8 XCDs), then
  // groups of GROUP_M tile-rows for L2 reuse
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
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  const bf16* A = reinterpret_cast<const bf16*>(p.A);
  const bf16* B = reinterpret_cast<const bf16*>(p.B);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int wm = w >> 1, wn = w & 1;

  f32x16 acc[MT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  auto stage_a = [&](int s) { return smem + s * A_U4; };
  auto stage_b = [&](int s) { return smem + NST * A_U4 + s * B_U4; };

  // per-lane DMA sources of the first K tile; a full tile t adds t*BK (K-contiguous)
  // or t*BK*ld (K-major) elements
  auto srcA = [&](int k0, int i) {
    return AK ? src_km(A, p.lda, p.M, m0, k0, kend, IA * w + i)
              : src_kc(A, p.lda, p.M, m0, k0, kend, IA * w + i);
  };
  auto srcB = [&](int k0, int i) {
    return BKM ? src_km(B, p.ldb, p.N, n0, k0, kend, 4 * w + i)
               : src_kc(B, p.ldb, p.N, n0, k0, kend, 4 * w + i);
  };
  const bf16* sA[IA];
  const bf16* sB[4];
#pragma unroll
  for (int i = 0; i < IA; ++i) sA[i] = srcA(kbeg, i);
#pragma unroll
  for (int i = 0; i < 4; ++i) sB[i] = srcB(kbeg, i);
  const int64_t stepA = AK ? (int64_t)BK * p.lda : BK;
  const int64_t stepB = BKM ? (int64_t)BK * p.ldb : BK;

  auto dma_tile = [&](int s, int t) __attribute__((always_inline)) {
    const int k0 = kbeg + t * BK;
    if (k0 + BK <= kend) {
#pragma unroll
      for (int i = 0; i < IA; ++i) dma16(sA[i] + t * stepA, stage_a(s), IA * w + i);
#pragma unroll
      for (int i = 0; i < 4; ++i) dma16(sB[i] + t * stepB, stage_b(s), 4 * w + i);
    } else {   // ragged last tile: clamped sources
#pragma unroll
      for (int i = 0; i < IA; ++i) dma16(srcA(k0, i), stage_a(s), IA * w + i);
#pragma unroll
      for (int i = 0; i < 4; ++i) dma16(srcB(k0, i), stage_b(s), 4 * w + i);
    }
  };

  // Per-lane fragment offsets (bytes).  K-contiguous block of 32 rows at row base rb:
  // lane reads row rb + l%32, logical chunk 2h + l/32 -> rb*64 + (koff ^ 32h), since
  // fkc depends only on the row bits below 32.
  const int kc_off = 64 * (l & 31) + 16 * ((l >> 5) ^ fkc(l & 31));
  // K-major block of 32 cols at col base cb = 128 wv + 32 i: 16-lane group G = l/16
  // reads k-rows 8(G/2) + (l%16)/4 (+4 for the second read, +16 for the second K half)
  // at col cb + 16(G%2) + 4(l%4); the swizzle makes the chunk depend on i.
  int km_off[4];
  {
    const int G = l >> 4, j = l & 15;
    const int kr = 8 * (G >> 1) + (j >> 2);
    const int gg = gkm(j >> 2);
    const int lo = 2 * (G & 1) + ((j & 3) >> 1);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      km_off[i] = kr * 512 + 16 * ((4 * (i ^ (gg >> 2))) + (lo ^ (gg & 3))) + 8 * (j & 1);
  }

  // fragments of K half h (16 k) of a stage: operand rows/cols of wave (wm, wn)
  auto frag_kc = [&](const uint4* t, int rb, int h) __attribute__((always_inline)) -> bf16x8 {
    const char* base = reinterpret_cast<const char*>(t) + rb * 64;
    const uint4 v = *reinterpret_cast<const uint4*>(base + (kc_off ^ (32 * h)));
    return *reinterpret_cast<const bf16x8*>(&v);
  };
  auto frag_km = [&](const uint4* t, int wv, int i, int h) __attribute__((always_inline)) -> bf16x8 {
    const char* base = reinterpret_cast<const char*>(t) + 16 * 16 * wv + h * 16 * 512 + km_off[i];
    const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base));
    const s16x4 c = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + 4 * 512));
    bf16x8 v;
    const bf16* pa = reinterpret_cast<const bf16*>(&a);
    const bf16* pc = reinterpret_cast<const bf16*>(&c);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] = pa[e];
      v[4 + e] = pc[e];
    }
    return v;
  };
  auto frag_a = [&](int s, int i, int h) __attribute__((always_inline)) -> bf16x8 {
    return AK ? frag_km(stage_a(s), wm, i, h) : frag_kc(stage_a(s), wm * (32 * MT) + 32 * i, h);
  };
  auto frag_b = [&](int s, int j, int h) __attribute__((always_inline)) -> bf16x8 {
    return BKM ? frag_km(stage_b(s), wn, j, h) : frag_kc(stage_b(s), wn * 128 + 32 * j, h);
  };
  bf16x8 fa[2][MT], fb[2][4];
  auto read_frags = [&](int s, int h, int t, bf16x8 (&a)[MT], bf16x8 (&bb)[4])
      __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < MT; ++i) a[i] = frag_a(s, i, h);
#pragma unroll
    for (int j = 0; j < 4; ++j) bb[j] = frag_b(s, j, h);
    // ragged K tail: zero the A elements past kend (B there holds clamped, finite data)
    const int kr = kend - (kbeg + t * BK) - 16 * h - 8 * (l >> 5);
    if (kend - (kbeg + t * BK) < BK) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (e >= kr) a[i][e] = (bf16)0.f;
    }
  };
  auto mma = [&](const bf16x8 (&a)[MT], const bf16x8 (&bb)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], bb[j], acc[i][j], 0, 0, 0);
  };
  // wait until tile t+1 has landed for this wave: only DMAs of later tiles (at most
  // NST-2 of them, issued before tile t+NST) may stay pending
  auto wait_next = [&](int t) __attribute__((always_inline)) {
    const int later = nk - 2 - t;
    if (later >= 2) wait_vm<2 * IPT>();
    else if (later == 1) wait_vm<IPT>();
    else wait_vm<0>();
  };

  // one K tile t in stage S = t % NST; fa[0]/fb[0] hold its first half on entry and the
  // next tile's first half on exit
  auto body = [&](auto S, int t) __attribute__((always_inline)) {
    constexpr int s = decltype(S)::value;
    constexpr int sn = (s + 1) % NST;
    read_frags(s, 1, t, fa[1], fb[1]);
    mma(fa[0], fb[0]);
    wait_next(t);
    lds_barrier();
    if (t + NST < nk) dma_tile(s, t + NST);
    if (t + 1 < nk) read_frags(sn, 0, t + 1, fa[0], fb[0]);
    mma(fa[1], fb[1]);
  };

  // Steady-state tile (every tile read or DMA'd precedes the last, possibly ragged,
  // tile): the same work as body(), with each fragment read and DMA placed between two
  // MFMAs in a fixed order (sched_barrier fences), so the MFMA pipe never waits behind a
  // burst of memory instructions.  Fragment reads go in the order the MFMAs (i-major)
  // first use them: A0, B0..B3, A1..
  constexpr int NMF = 4 * MT;      // MFMAs per K half
  constexpr int NRD = MT + 4;      // fragment reads per K half
  auto rd1 = [&](int s, int h, int k, bf16x8 (&a)[MT], bf16x8 (&bb)[4])
      __attribute__((always_inline)) {
    const bool isb = k >= 1 && k <= 4;
    const int i = k == 0 ? 0 : isb ? k - 1 : k - 4;
    if (isb) bb[i] = frag_b(s, i, h);
    else a[i] = frag_a(s, i, h);
  };
  auto mf1 = [&](int n, const bf16x8 (&a)[MT], const bf16x8 (&bb)[4]) __attribute__((always_inline)) {
    acc[n >> 2][n & 3] =
        __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[n >> 2], bb[n & 3], acc[n >> 2][n & 3], 0, 0, 0);
  };
  auto dm1 = [&](int s, int t, int q) __attribute__((always_inline)) {
    if (q < IA) dma16(sA[q] + t * stepA, stage_a(s), IA * w + q);
    else dma16(sB[q - IA] + t * stepB, stage_b(s), 4 * w + (q - IA));
  };
  auto body_full = [&](auto S, int t) __attribute__((always_inline)) {
    constexpr int s = decltype(S)::value;
    constexpr int sn = (s + 1) % NST;
    // first half: second-half reads of this tile, read r before MFMA r*NMF/NRD
#pragma unroll
    for (int n = 0; n < NMF; ++n) {
#pragma unroll
      for (int r = 0; r < NRD; ++r)
        if (r * NMF / NRD == n) {
          rd1(s, 1, r, fa[1], fb[1]);
          __builtin_amdgcn_sched_barrier(0);
        }
      mf1(n, fa[0], fb[0]);
      __builtin_amdgcn_sched_barrier(0);
    }
    wait_vm<(NST - 2) * IPT>();
    lds_barrier();
    // second half: DMA d of tile t+NST before MFMA d*NMF/IPT, read r of the next tile's
    // first half right after MFMA r*NMF/NRD
#pragma unroll
    for (int n = 0; n < NMF; ++n) {
#pragma unroll
      for (int d = 0; d < IPT; ++d)
        if (d * NMF / IPT == n) {
          dm1(s, t + NST, d);
          __builtin_amdgcn_sched_barrier(0);
        }
      mf1(n, fa[1], fb[1]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int r = 0; r < NRD; ++r)
        if (r * NMF / NRD == n) {
          rd1(sn, 0, r, fa[0], fb[0]);
          __builtin_amdgcn_sched_barrier(0);
        }
    }
  };

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  using S3 = std::integral_constant<int, 3>;
  if (nk > 0) {
#pragma unroll
    for (int s = 0; s < NST; ++s)
      if (s < nk) dma_tile(s, s);
    // tile 0 landed: the prologue's later tiles may stay pending
    if (nk > 3) wait_vm<3 * IPT>();
    else if (nk == 3) wait_vm<2 * IPT>();
    else if (nk == 2) wait_vm<IPT>();
    else wait_vm<0>();
    lds_barrier();
    read_frags(0, 0, 0, fa[0], fb[0]);
    int t = 0;
    // steady state: the tiles read (<= t+NST) and the tiles DMA'd (<= t+2NST-1) all
    // precede the last, possibly ragged, tile, so every source is unclamped and in bounds
    for (; t + 2 * NST + 1 <= nk; t += NST) {
      body_full(S0{}, t);
      body_full(S1{}, t + 1);
      body_full(S2{}, t + 2);
      body_full(S3{}, t + 3);
    }
    for (; t < nk; t += NST) {
      body(S0{}, t);
      if (t + 1 < nk) body(S1{}, t + 1);
      if (t + 2 < nk) body(S2{}, t + 2);
      if (t + 3 < nk) body(S3{}, t + 3);
    }
  }

  // epilogue: each wave stages 16x128 accumulator rows at a time in its own LDS region
  // (after the barrier below no wave reads the ring any more).  Pass pi = 2i + hh covers
  // rows 32i + 16hh .. +15 of the wave tile; lane (u, cg) takes row (l/16) + 4u, columns
  // 8cg..8cg+7.
  __syncthreads();
  float* stage = reinterpret_cast<float*>(smem) + w * 16 * SP;
  const int cg = l & 15;
  const int n = n0 + wn * 128 + 8 * cg;   // N % 8 == 0: all eight columns or none in range
  const bool vec = n < p.N;
  float bias8[8];
  load_bias8(p, vec && split == 0, n, bias8);
  auto row_of = [&](int pi, int u) { return m0 + wm * (32 * MT) + 16 * pi + (l >> 4) + 4 * u; };
  constexpr bool kAux = EPI == EPI_GELU_BWD || EPI == EPI_RESID || EPI == EPI_F32 ||
                        EPI == EPI_STORE_ROPE;
  AuxV ax[2][4];
  auto fetch = [&](int pi, AuxV (&dst)[4]) __attribute__((always_inline)) {
    if constexpr (kAux) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int m = row_of(pi, u);
        if (vec && m < p.M) aux_fetch<EPI>(p, split, m, n, dst[u]);
      }
    }
  };
  fetch(0, ax[0]);
#pragma unroll
  for (int i = 0; i < MT; ++i) {     // (acc[i] must be indexed statically)
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int pi = 2 * i + hh;
      if (pi + 1 < 2 * MT) fetch(pi + 1, ax[(pi + 1) & 1]);
      lds_wave_fence();   // the previous pass's staging reads are done
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 8 * hh; e < 8 * hh + 8; ++e) {
          const int rr = 8 * ((e >> 2) & 1) + 4 * (l >> 5) + (e & 3);
          stage[rr * SP + 32 * j + (l & 31)] = acc[i][j][e];
        }
      lds_wave_fence();   // this pass's staging writes are visible to the whole wave
      auto out_row = [&](int u, const AuxV& a) __attribute__((always_inline)) {
        const int rr = (l >> 4) + 4 * u;
        const int m = row_of(pi, u);
        if (m >= p.M || n >= p.N) return;
        float v[8];
        const float4 x0 = *reinterpret_cast<const float4*>(stage + rr * SP + 8 * cg);
        const float4 x1 = *reinterpret_cast<const float4*>(stage + rr * SP + 8 * cg + 4);
        v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w;
        v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
        epi8_vec<EPI>(p, split, m, n, v, bias8, a);
      };
      if constexpr (kAux) {   // static u: the prefetched operands live in registers
#pragma unroll
        for (int u = 0; u < 4; ++u) out_row(u, ax[pi & 1][u]);
      } else {                // no operands to prefetch: a rolled loop keeps the code small
#pragma unroll 1
        for (int u = 0; u < 4; ++u) out_row(u, ax[0][0]);
      }
    }
  }
}

// ---- NT kernel: 256x256 tiles, 64-deep K stages ---------------------------------------
//
// Both operands K-contiguous ([M][K] activations, [N][K] weight).  A K tile is 64 deep, so
// every operand row of a stage is one whole 128-byte line: DMA instruction q of a 32 KB
// operand tile fetches rows 8q..8q+7, lane l row 8q + l/8 at physical chunk l%8, which
// holds logical chunk (l%8) ^ f8(row), f8(row) = (row >> 1) & 7.  A fragment read (32
// rows at one logical chunk per lane half) then covers 16 distinct 16-byte bank groups in
// every 16-lane group.  Two stages (2 x 64 KB): the DMA of tile t+2 goes out right after
// the barrier in the middle of tile t (stage t%2 fully read by then), so at every wait
// the only DMAs pending are tile t+1's, and one barrier covers 2048 MFMA cycles per wave.
// Waves 2x2 of 128x128 with 4x4 32x32x16 accumulators in the same K order as the other
// kernels, so an output element gets bitwise the same value from any of them.
constexpr int BK64 = 64;
constexpr int T64_U4 = 256 * BK64 * 2 / 16;   // 16-byte slots of a 256 x 64 operand tile (2048)
constexpr int I64 = 8;                        // DMA instructions per wave per operand tile
constexpr int NT64_LDS_U4 = 2 * 2 * T64_U4;   // two stages of A and B: 128 KB

__device__ __forceinline__ int f8(int r) { return (r >> 1) & 7; }
// source of instruction q of a 256-row, 64-deep K-contiguous tile (rows r0.., k from k0)
__device__ __forceinline__ const bf16* src_kc64(const bf16* X, int64_t ld, int rows, int r0,
                                                int k0, int kend, int q) {
  const int l = threadIdx.x & 63;
  const int row = 8 * q + (l >> 3);
  int k = k0 + 8 * ((l & 7) ^ f8(row));
  k = k < kend ? k : kend - 8;
  int gr = r0 + row;
  gr = gr < rows ? gr : rows - 1;
  return X + (int64_t)gr * ld + k;
}

template <int EPI>
__global__ __launch_bounds__(NTHR, 1) void gemm_nt64_kernel(GemmArgs p) {
  __shared__ uint4 smem[NT64_LDS_U4];
  static_assert(4 * 16 * SP * 4 <= NT64_LDS_U4 * 16, "epilogue staging must fit in the ring");

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
  const int m0 = tm * 256, n0 = tn * 256;
  const int kbeg = split * p.kps;
  const int kend = min(p.K, kbeg + p.kps);
  const int nk = kend > kbeg ? (kend - kbeg + BK64 - 1) / BK64 : 0;
  const int nfull = kend > kbeg ? (kend - kbeg) / BK64 : 0;   // tiles t < nfull are whole
  const bf16* A = reinterpret_cast<const bf16*>(p.A);
  const bf16* B = reinterpret_cast<const bf16*>(p.B);
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), l = threadIdx.x & 63;
  const int wm = w >> 1, wn = w & 1;

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  auto stage_a = [&](int s) { return smem + s * T64_U4; };
  auto stage_b = [&](int s) { return smem + (2 + s) * T64_U4; };
  const bf16* sA[I64];
  const bf16* sB[I64];
#pragma unroll
  for (int i = 0; i < I64; ++i) {
    sA[i] = src_kc64(A, p.lda, p.M, m0, kbeg, kend, I64 * w + i);
    sB[i] = src_kc64(B, p.ldb, p.N, n0, kbeg, kend, I64 * w + i);
  }
  // DMA d (0..15: A instructions, then B) of tile t into stage s; a whole tile adds t*64
  auto dm1 = [&](int s, int t, int d) __attribute__((always_inline)) {
    if (d < I64) dma16(sA[d] + t * BK64, stage_a(s), I64 * w + d);
    else dma16(sB[d - I64] + t * BK64, stage_b(s), I64 * w + (d - I64));
  };
  auto dma_tile = [&](int s, int t) __attribute__((always_inline)) {
    if (t < nfull) {
#pragma unroll
      for (int d = 0; d < 2 * I64; ++d) dm1(s, t, d);
    } else {   // ragged last tile: clamped sources
      const int k0 = kbeg + t * BK64;
#pragma unroll
      for (int i = 0; i < I64; ++i) {
        dma16(src_kc64(A, p.lda, p.M, m0, k0, kend, I64 * w + i), stage_a(s), I64 * w + i);
        dma16(src_kc64(B, p.ldb, p.N, n0, k0, kend, I64 * w + i), stage_b(s), I64 * w + i);
      }
    }
  };

  // lane offset of a fragment read in a 32-row block: row l%32, logical chunk 2h + l/32 of
  // K step h at physical chunk (2h + l/32) ^ f8(l%32) -> kc ^ 32h
  const int kc = 128 * (l & 31) + 16 * ((l >> 5) ^ f8(l & 31));
  auto frag = [&](const uint4* t, int rb, int h) __attribute__((always_inline)) -> bf16x8 {
    const char* base = reinterpret_cast<const char*>(t) + rb * 128;
    const uint4 v = *reinterpret_cast<const uint4*>(base + (kc ^ (32 * h)));
    return *reinterpret_cast<const bf16x8*>(&v);
  };
  // fragment read k (0..7) of K step h, in first-use order A0, B0..B3, A1..A3
  auto rd1 = [&](int s, int h, int k, bf16x8 (&a)[4], bf16x8 (&bb)[4]) __attribute__((always_inline)) {
    const bool isb = k >= 1 && k <= 4;
    const int i = k == 0 ? 0 : isb ? k - 1 : k - 4;
    if (isb) bb[i] = frag(stage_b(s), wn * 128 + 32 * i, h);
    else a[i] = frag(stage_a(s), wm * 128 + 32 * i, h);
  };
  // ragged tile t: zero this lane's A elements of K step h past kend
  auto mask_a = [&](int t, int h, bf16x8 (&a)[4]) __attribute__((always_inline)) {
    if (t >= nfull) {
      const int kr = kend - (kbeg + t * BK64) - 16 * h - 8 * (l >> 5);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (e >= kr) a[i][e] = (bf16)0.f;
    }
  };
  auto mf1 = [&](int n, const bf16x8 (&a)[4], const bf16x8 (&bb)[4]) __attribute__((always_inline)) {
    acc[n >> 2][n & 3] =
        __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[n >> 2], bb[n & 3], acc[n >> 2][n & 3], 0, 0, 0);
  };
  bf16x8 fa[2][4], fb[2][4];
  // tile t in stage S = t % 2; fa[0] / fb[0] hold its K step 0 on entry and tile t+1's on
  // exit.  FULL: tiles t, t+1 and t+2 whole (no guard splits the fenced schedule).
  auto body = [&](auto S, auto FULL, int t) __attribute__((always_inline)) {
    constexpr int s = decltype(S)::value, sn = 1 - s;
    constexpr bool full = decltype(FULL)::value;
#pragma unroll
    for (int h = 0; h < 3; ++h) {
      bf16x8 (&an)[4] = fa[(h + 1) & 1];
      bf16x8 (&bn)[4] = fb[(h + 1) & 1];
#pragma unroll
      for (int n = 0; n < 16; ++n) {
        if ((n & 1) == 0) {
          rd1(s, h + 1, n >> 1, an, bn);
          __builtin_amdgcn_sched_barrier(0);
        }
        mf1(n, fa[h & 1], fb[h & 1]);
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (!full) mask_a(t, h + 1, an);
    }
    wait_vm<0>();   // tile t+1 landed (the only DMAs pending)
    lds_barrier();  // every wave is done with stage s
    if constexpr (full) {
#pragma unroll
      for (int n = 0; n < 16; ++n) {
        dm1(s, t + 2, n);
        __builtin_amdgcn_sched_barrier(0);
        mf1(n, fa[1], fb[1]);
        __builtin_amdgcn_sched_barrier(0);
        if ((n & 1) == 0) {
          rd1(sn, 0, n >> 1, fa[0], fb[0]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    } else {
      if (t + 2 < nk) dma_tile(s, t + 2);
#pragma unroll
      for (int n = 0; n < 16; ++n) mf1(n, fa[1], fb[1]);
      if (t + 1 < nk) {
#pragma unroll
        for (int k = 0; k < 8; ++k) rd1(sn, 0, k, fa[0], fb[0]);
        mask_a(t + 1, 0, fa[0]);
      }
    }
  };

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using F0 = std::integral_constant<bool, false>;
  using F1 = std::integral_constant<bool, true>;
  if (nk > 0) {
    dma_tile(0, 0);
    if (nk > 1) {
      dma_tile(1, 1);
      wait_vm<2 * I64>();   // tile 0 landed; tile 1 may stay pending
    } else {
      wait_vm<0>();
    }
    lds_barrier();
#pragma unroll
    for (int k = 0; k < 8; ++k) rd1(0, 0, k, fa[0], fb[0]);
    mask_a(0, 0, fa[0]);
    int t = 0;
    // steady state: tiles t, t+1 and the DMA'd tile t+2 all whole
    for (; t + 4 <= nfull; t += 2) {
      body(S0{}, F1{}, t);
      body(S1{}, F1{}, t + 1);
    }
    for (; t < nk; t += 2) {   // the last (at most five) tiles, guarded
      body(S0{}, F0{}, t);
      if (t + 1 < nk) body(S1{}, F0{}, t + 1);
    }
  }
  wait_vm<0>();

  // epilogue (as in the 256x256 kernel above)
  __syncthreads();
  float* stage = reinterpret_cast<float*>(smem) + w * 16 * SP;
  const int cg = l & 15;
  const int n = n0 + wn * 128 + 8 * cg;
  const bool vec = n < p.N;
  float bias8[8];
  load_bias8(p, vec && split == 0, n, bias8);
  auto row_of = [&](int pi, int u) { return m0 + wm * 128 + 16 * pi + (l >> 4) + 4 * u; };
  constexpr bool kAux = EPI == EPI_GELU_BWD || EPI == EPI_RESID || EPI == EPI_F32 ||
                        EPI == EPI_STORE_ROPE;
  AuxV ax[2][4];
  auto fetch = [&](int pi, AuxV (&dst)[4]) __attribute__((always_inline)) {
    if constexpr (kAux) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int m = row_of(pi, u);
        if (vec && m < p.M) aux_fetch<EPI>(p, split, m, n, dst[u]);
      }
    }
  };
  fetch(0, ax[0]);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int pi = 2 * i + hh;
      if (pi + 1 < 8) fetch(pi + 1, ax[(pi + 1) & 1]);
      lds_wave_fence();
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 8 * hh; e < 8 * hh + 8; ++e) {
          const int rr = 8 * ((e >> 2) & 1) + 4 * (l >> 5) + (e & 3);
          stage[rr * SP + 32 * j + (l & 31)] = acc[i][j][e];
        }
      lds_wave_fence();
      auto out_row = [&](int u, const AuxV& a) __attribute__((always_inline)) {
        const int rr = (l >> 4) + 4 * u;
        const int m = row_of(pi, u);
        if (m >= p.M || n >= p.N) return;
        float v[8];
        const float4 x0 = *reinterpret_cast<const float4*>(stage + rr * SP + 8 * cg);
        const float4 x1 = *reinterpret_cast<const float4*>(stage + rr * SP + 8 * cg + 4);
        v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w;
        v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
        epi8_vec<EPI>(p, split, m, n, v, bias8, a);
      };
      if constexpr (kAux) {
#pragma unroll
        for (int u = 0; u < 4; ++u) out_row(u, ax[pi & 1][u]);
      } else {
#pragma unroll 1
        for (int u = 0; u < 4; ++u) out_row(u, ax[0][0]);
      }
    }
  }
}

// ---- NN kernel: 128x256 tiles, paired A stages ---------------------------------------
//
// The input-gradient and forward products (A = activations [M][K], B = weight [K][N]).  A
// is filled two K tiles at a time: each DMA instruction fetches 8 rows x 64 k, whole
// 128-byte lines of A (64-byte rows would send half-line requests, which the memory
// pipeline serves at a markedly lower rate).  Its 1 KB of LDS holds the 8 rows' first 32 k
// (tile 2P) and then their second 32 k (tile 2P+1), each as 64-byte rows with the same
// chunk swizzle as the 256x256 kernel, so a tile's fragments sit at a fixed offset in the
// pair stage.  Two pair stages (2 x 16 KB) and three B stages (3 x 16 KB of 512-byte
// K-major rows) make 80 KB, so two blocks share a CU and each one's barriers and epilogue
// overlap the other's main loop.  Waves 2x2, each a 64x128 tile of 2x4 32x32 accumulators.
//
// body(t): the second half's fragments of tile t are read beside the first half's
// MFMAs; wait until tile t+1 has landed; barrier; DMA of B tile t+3 into tile t's B stage
// and, after the second tile of a pair, of A pair (t+3, t+4) into the pair stage just
// consumed; tile t+1's first-half fragments are read beside tile t's second-half MFMAs.
// In issue order the DMAs are B(0) A(0,1) B(1) B(2) A(2,3) B(3) B(4) A(4,5) ..., so when
// tile t+1 is needed the later DMAs still allowed in flight are B(t+2) and, for even t,
// A(t+2, t+3).  Pair stages repeat every 4 tiles: the steady loop is unrolled over that
// period, so A fragment addresses are constant offsets; the B stage rotates at run time.

constexpr int NN_BM = 128;
constexpr int NN_A_U4 = NN_BM * 2 * BK * 2 / 16;   // 16-byte slots of an A pair stage (1024)
constexpr int NN_LDS_U4 = 2 * NN_A_U4 + 3 * B_U4;  // 80 KB
constexpr int NN_IA = 4;                           // A pair DMA instructions per wave
constexpr int NN_IB = 4;                           // B tile DMA instructions per wave
constexpr int NN_PERIOD = 4;

// A pair source of instruction q: lane l fetches row 8q + (l%32)/4, tile half l/32,
// physical chunk l%4, which holds logical chunk (l%4) ^ fkc(row): k = k0 + 32 (l/32) +
// 8 ((l%4) ^ fkc(row)) of the pair's 64-wide K range.
__device__ __forceinline__ const bf16* src_pair(const bf16* X, int64_t ld, int rows, int r0, int k0,
                                                int kend, int q) {
  const int l = threadIdx.x & 63;
  const int row = 8 * q + ((l & 31) >> 2);
  int k = k0 + 32 * (l >> 5) + 8 * ((l & 3) ^ fkc(row));
  k = k < kend ? k : kend - 8;
  int gr = r0 + row;
  gr = gr < rows ? gr : rows - 1;
  return X + (int64_t)gr * ld + k;
}

template <int EPI>
__global__ __launch_bounds__(NTHR, 2) void gemm_nn_kernel(GemmArgs p) {
  __shared__ uint4 smem[NN_LDS_U4];
  static_assert(4 * 16 * SP * 4 <= NN_LDS_U4 * 16, "epilogue staging must fit in the ring");

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
  const int m0 = tm * NN_BM, n0 = tn * BN;
  const int kbeg = split * p.kps;
  const int kend = min(p.K, kbeg + p.kps);
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  const bf16* A = reinterpret_cast<const bf16*>(p.A);
  const bf16* B = reinterpret_cast<const bf16*>(p.B);
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), l = threadIdx.x & 63;
  const int wm = w >> 1, wn = w & 1;

  f32x16 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const char* const lds = reinterpret_cast<const char*>(smem);
  // B stages first, so B fragment offsets fit the 16-bit LDS immediate
  auto pair_stage = [&](int pa) { return smem + 3 * B_U4 + pa * NN_A_U4; };
  auto b_stage = [&](int sb) { return smem + sb * B_U4; };

  // DMA sources of the first A pair / B tile (a full pair P adds 64P elements, a full
  // B tile t adds t*BK rows)
  const bf16* sA[NN_IA];
  const bf16* sB[NN_IB];
#pragma unroll
  for (int i = 0; i < NN_IA; ++i) sA[i] = src_pair(A, p.lda, p.M, m0, kbeg, kend, NN_IA * w + i);
#pragma unroll
  for (int i = 0; i < NN_IB; ++i) sB[i] = src_km(B, p.ldb, p.N, n0, kbeg, kend, NN_IB * w + i);
  const int64_t stepB = (int64_t)BK * p.ldb;
  auto dma_b = [&](int sb, int t) __attribute__((always_inline)) {
    const int k0 = kbeg + t * BK;
    if (k0 + BK <= kend) {
#pragma unroll
      for (int i = 0; i < NN_IB; ++i) dma16(sB[i] + t * stepB, b_stage(sb), NN_IB * w + i);
    } else {
#pragma unroll
      for (int i = 0; i < NN_IB; ++i)
        dma16(src_km(B, p.ldb, p.N, n0, k0, kend, NN_IB * w + i), b_stage(sb), NN_IB * w + i);
    }
  };
  auto dma_a = [&](int pa, int t) __attribute__((always_inline)) {   // pair (t, t+1), t even
    const int k0 = kbeg + t * BK;
    if (k0 + 2 * BK <= kend) {
#pragma unroll
      for (int i = 0; i < NN_IA; ++i) dma16(sA[i] + (t >> 1) * (2 * BK), pair_stage(pa), NN_IA * w + i);
    } else {
#pragma unroll
      for (int i = 0; i < NN_IA; ++i)
        dma16(src_pair(A, p.lda, p.M, m0, k0, kend, NN_IA * w + i), pair_stage(pa), NN_IA * w + i);
    }
  };

  // A fragment i of K half h of the tile with parity par in pair stage pa: rows
  // rb = wm*64 + 32i + l%32 live in instruction slots rb/8 (1 KB each), half par, 64-byte
  // row rb%8, logical chunk 2h + l/32 at physical chunk (2h + l/32) ^ fkc(rb).
  const int kcA = 1024 * ((l & 31) >> 3) + 64 * (l & 7) + 16 * ((l >> 5) ^ fkc(l & 31));
  // B (K-major, as in the 256x256 kernel)
  int km_off[4];
  {
    const int G = l >> 4, j = l & 15;
    const int kr = 8 * (G >> 1) + (j >> 2);
    const int gg = gkm(j >> 2);
    const int lo = 2 * (G & 1) + ((j & 3) >> 1);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      km_off[i] = kr * 512 + 16 * ((4 * (i ^ (gg >> 2))) + (lo ^ (gg & 3))) + 8 * (j & 1);
  }
  auto frag_a = [&](int pa, int par, int i, int h) __attribute__((always_inline)) -> bf16x8 {
    const char* base = lds + (3 * B_U4 + pa * NN_A_U4) * 16 + par * 512 + (wm * 64 + 32 * i) * 128;
    const uint4 v = *reinterpret_cast<const uint4*>(base + (kcA ^ (32 * h)));
    return *reinterpret_cast<const bf16x8*>(&v);
  };
  auto frag_b = [&](int sb, int j, int h) __attribute__((always_inline)) -> bf16x8 {
    const char* base = lds + sb * B_U4 * 16 + 16 * 16 * wn + h * 16 * 512 + km_off[j];
    const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base));
    const s16x4 c = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + 4 * 512));
    bf16x8 v;
    const bf16* pa_ = reinterpret_cast<const bf16*>(&a);
    const bf16* pc = reinterpret_cast<const bf16*>(&c);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] = pa_[e];
      v[4 + e] = pc[e];
    }
    return v;
  };
  bf16x8 fa[2][2], fb[2][4];
  // fragments of K half h of tile t = period slot I (ragged last tile: A zeroed past kend)
  auto read_frags = [&](auto II, int t, int h, bf16x8 (&a)[2], bf16x8 (&bb)[4])
      __attribute__((always_inline)) {
    constexpr int I = decltype(II)::value;
    constexpr int pa = (I >> 1) & 1, par = I & 1;
    const int sb = t % 3;
#pragma unroll
    for (int i = 0; i < 2; ++i) a[i] = frag_a(pa, par, i, h);
#pragma unroll
    for (int j = 0; j < 4; ++j) bb[j] = frag_b(sb, j, h);
    const int rem = kend - (kbeg + t * BK);
    if (rem < BK) {
      const int kr = rem - 16 * h - 8 * (l >> 5);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (e >= kr) a[i][e] = (bf16)0.f;
    }
  };
  auto mma = [&](const bf16x8 (&a)[2], const bf16x8 (&bb)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], bb[j], acc[i][j], 0, 0, 0);
  };
  auto mf1 = [&](int n, const bf16x8 (&a)[2], const bf16x8 (&bb)[4]) __attribute__((always_inline)) {
    acc[n >> 2][n & 3] =
        __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[n >> 2], bb[n & 3], acc[n >> 2][n & 3], 0, 0, 0);
  };
  // read k (0..5) of a half in first-use order A0, B0..B3, A1
  auto rd1 = [&](int pa, int par, int sb, int h, int k, bf16x8 (&a)[2], bf16x8 (&bb)[4])
      __attribute__((always_inline)) {
    if (k >= 1 && k <= 4) bb[k - 1] = frag_b(sb, k - 1, h);
    else a[k == 0 ? 0 : 1] = frag_a(pa, par, k == 0 ? 0 : 1, h);
  };

  // steady-state tile t = period slot I (t + 6 <= nk), B stage sb = t % 3, next sbn:
  // every DMA full, no ragged read
  auto body_fast = [&](auto II, int t, int sb, int sbn) __attribute__((always_inline)) {
    constexpr int I = decltype(II)::value;
    constexpr int P = I & 1, pa = (I >> 1) & 1;
    constexpr int In = (I + 1) % NN_PERIOD;
    constexpr int pan = (In >> 1) & 1, parn = In & 1;
    constexpr int ND = P ? NN_IA + NN_IB : NN_IB;   // DMA instructions after the barrier
#pragma unroll
    for (int n = 0; n < 8; ++n) {
#pragma unroll
      for (int r = 0; r < 6; ++r)
        if (r * 8 / 6 == n) {
          rd1(pa, P, sb, 1, r, fa[1], fb[1]);
          __builtin_amdgcn_sched_barrier(0);
        }
      mf1(n, fa[0], fb[0]);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (P == 0) wait_vm<NN_IB + NN_IA>();
    else wait_vm<NN_IB>();
    lds_barrier();
#pragma unroll
    for (int n = 0; n < 8; ++n) {
#pragma unroll
      for (int d = 0; d < ND; ++d)
        if (d * 8 / ND == n) {
          if (d < NN_IB) dma16(sB[d] + (t + 3) * stepB, b_stage(sb), NN_IB * w + d);
          else dma16(sA[d - NN_IB] + ((t + 3) >> 1) * (2 * BK), pair_stage(pa), NN_IA * w + (d - NN_IB));
          __builtin_amdgcn_sched_barrier(0);
        }
      mf1(n, fa[1], fb[1]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int r = 0; r < 6; ++r)
        if (r * 8 / 6 == n) {
          rd1(pan, parn, sbn, 0, r, fa[0], fb[0]);
          __builtin_amdgcn_sched_barrier(0);
        }
    }
  };
  // tile t = period slot I near the end: guarded DMAs, masked reads
  auto body_slow = [&](auto II, int t) __attribute__((always_inline)) {
    constexpr int I = decltype(II)::value;
    constexpr int pa = (I >> 1) & 1;
    using INext = std::integral_constant<int, (I + 1) % NN_PERIOD>;
    read_frags(II, t, 1, fa[1], fb[1]);
    mma(fa[0], fb[0]);
    if (t + 2 < nk) {
      if constexpr (I & 1) wait_vm<NN_IB>();
      else wait_vm<NN_IB + NN_IA>();
    } else {
      wait_vm<0>();
    }
    lds_barrier();
    if (t + 3 < nk) {
      dma_b(t % 3, t + 3);
      if constexpr (I & 1) dma_a(pa, t + 3);
    }
    if (t + 1 < nk) read_frags(INext{}, t + 1, 0, fa[0], fb[0]);
    mma(fa[1], fb[1]);
  };

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  using S3 = std::integral_constant<int, 3>;
  if (nk > 0) {
    dma_b(0, 0);
    dma_a(0, 0);
    if (nk > 1) dma_b(1, 1);
    if (nk > 2) {
      dma_b(2, 2);
      dma_a(1, 2);
    }
    if (nk > 2) wait_vm<2 * NN_IB + NN_IA>();
    else if (nk == 2) wait_vm<NN_IB>();
    else wait_vm<0>();
    lds_barrier();
    read_frags(S0{}, 0, 0, fa[0], fb[0]);
    // steady state: tiles t with t + 6 <= nk, four at a time (t % 4 == slot); then the
    // last tiles (at most 8)
    const int nfast = nk >= 6 ? (nk - 5) / 4 * 4 : 0;
    int t = 0;
    for (; t < nfast; t += 4) {
      const int s0 = t % 3;
      const int s1 = s0 == 2 ? 0 : s0 + 1;
      const int s2 = s1 == 2 ? 0 : s1 + 1;
      body_fast(S0{}, t, s0, s1);
      body_fast(S1{}, t + 1, s1, s2);
      body_fast(S2{}, t + 2, s2, s0);
      body_fast(S3{}, t + 3, s0, s1);
    }
    for (; t < nk; t += 4) {
      body_slow(S0{}, t);
      if (t + 1 < nk) body_slow(S1{}, t + 1);
      if (t + 2 < nk) body_slow(S2{}, t + 2);
      if (t + 3 < nk) body_slow(S3{}, t + 3);
    }
  }

  // epilogue (as in the 256x256 kernel, 64-row wave tiles)
  __syncthreads();
  float* stage = reinterpret_cast<float*>(smem) + w * 16 * SP;
  const int cg = l & 15;
  const int n = n0 + wn * 128 + 8 * cg;
  const bool vec = n < p.N;
  float bias8[8];
  load_bias8(p, vec && split == 0, n, bias8);
  auto row_of = [&](int pi, int u) { return m0 + wm * 64 + 16 * pi + (l >> 4) + 4 * u; };
  // GELU-backward column sums over this wave's 64-row band (p.colsum is grid-uniform)
  const bool kSum = EPI == EPI_GELU_BWD && p.colsum != nullptr;
  float cs[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) cs[e] = 0.f;
  constexpr bool kAux = EPI == EPI_GELU_BWD || EPI == EPI_RESID || EPI == EPI_F32 ||
                        EPI == EPI_STORE_ROPE;
  AuxV ax[2][4];
  auto fetch = [&](int pi, AuxV (&dst)[4]) __attribute__((always_inline)) {
    if constexpr (kAux) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int m = row_of(pi, u);
        if (vec && m < p.M) aux_fetch<EPI>(p, split, m, n, dst[u]);
      }
    }
  };
  fetch(0, ax[0]);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int pi = 2 * i + hh;
      if (pi + 1 < 4) fetch(pi + 1, ax[(pi + 1) & 1]);
      lds_wave_fence();
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 8 * hh; e < 8 * hh + 8; ++e) {
          const int rr = 8 * ((e >> 2) & 1) + 4 * (l >> 5) + (e & 3);
          stage[rr * SP + 32 * j + (l & 31)] = acc[i][j][e];
        }
      lds_wave_fence();
      auto out_row = [&](int u, const AuxV& a) __attribute__((always_inline)) {
        const int rr = (l >> 4) + 4 * u;
        const int m = row_of(pi, u);
        if (m >= p.M || n >= p.N) return;
        float v[8];
        const float4 x0 = *reinterpret_cast<const float4*>(stage + rr * SP + 8 * cg);
        const float4 x1 = *reinterpret_cast<const float4*>(stage + rr * SP + 8 * cg + 4);
        v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w;
        v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
        epi8_vec<EPI>(p, split, m, n, v, bias8, a, kSum ? cs : nullptr);
      };
      if constexpr (kAux) {
#pragma unroll
        for (int u = 0; u < 4; ++u) out_row(u, ax[pi & 1][u]);
      } else {
#pragma unroll 1
        for (int u = 0; u < 4; ++u) out_row(u, ax[0][0]);
      }
    }
  }
  if (kSum) {
    // the four lanes of a column group hold rows l >> 4 = 0..3 of each staged quad:
    // add them in a fixed order, then one lane writes the band's eight sums
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      cs[e] += __shfl_xor(cs[e], 16);
      cs[e] += __shfl_xor(cs[e], 32);
    }
    const int band0 = m0 + wm * 64;
    if ((l >> 4) == 0 && vec && band0 < p.M) {
      float* dst = p.colsum + (int64_t)(band0 / 64) * p.N + n;
      *reinterpret_cast<float4*>(dst) = make_float4(cs[0], cs[1], cs[2], cs[3]);
      *reinterpret_cast<float4*>(dst + 4) = make_float4(cs[4], cs[5], cs[6], cs[7]);
    }
  }
}

template <int EPI>
hipError_t launch_nn(const GemmArgs& a0, hipStream_t s) {
  GemmArgs a = a0;
  a.tiles_m = (a.M + NN_BM - 1) / NN_BM;
  a.tiles_n = (a.N + BN - 1) / BN;
  const int nt = a.tiles_m * a.tiles_n;
  const int nb = (nt + 7) / 8 * 8;
  int splits = a.kps > 0 ? (a.K + a.kps - 1) / a.kps : 1;
  if (a.kps <= 0) a.kps = a.K;
  if (splits < 1) splits = 1;
  hipLaunchKernelGGL((gemm_nn_kernel<EPI>), dim3(nb, splits), dim3(NTHR), 0, s, a);
  return hipGetLastError();
}

hipError_t dispatch_nn(const GemmArgs& a, int epi, hipStream_t s) {
  switch (epi) {
    case EPI_STORE: return launch_nn<EPI_STORE>(a, s);
    case EPI_STORE_ROPE: return launch_nn<EPI_STORE_ROPE>(a, s);
    case EPI_GELU: return launch_nn<EPI_GELU>(a, s);
    case EPI_RESID: return launch_nn<EPI_RESID>(a, s);
    case EPI_GELU_BWD: return launch_nn<EPI_GELU_BWD>(a, s);
    case EPI_F32: return launch_nn<EPI_F32>(a, s);
  }
  return hipErrorInvalidValue;
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

template <int EPI>
hipError_t launch_nt64(const GemmArgs& a0, hipStream_t s) {
  GemmArgs a = a0;
  a.tiles_m = (a.M + 255) / 256;
  a.tiles_n = (a.N + 255) / 256;
  const int nt = a.tiles_m * a.tiles_n;
  const int nb = (nt + 7) / 8 * 8;
  int splits = a.kps > 0 ? (a.K + a.kps - 1) / a.kps : 1;
  if (a.kps <= 0) a.kps = a.K;
  if (splits < 1) splits = 1;
  hipLaunchKernelGGL((gemm_nt64_kernel<EPI>), dim3(nb, splits), dim3(NTHR), 0, s, a);
  return hipGetLastError();
}

hipError_t dispatch_nt64(const GemmArgs& a, int epi, hipStream_t s) {
  switch (epi) {
    case EPI_STORE: return launch_nt64<EPI_STORE>(a, s);
    case EPI_STORE_ROPE: return launch_nt64<EPI_STORE_ROPE>(a, s);
    case EPI_GELU: return launch_nt64<EPI_GELU>(a, s);
    case EPI_RESID: return launch_nt64<EPI_RESID>(a, s);
    case EPI_GELU_BWD: return launch_nt64<EPI_GELU_BWD>(a, s);
    case EPI_F32: return launch_nt64<EPI_F32>(a, s);
  }
  return hipErrorInvalidValue;
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

}  // namespace

// Kernel per layout, from timings of the encoder's products on MI355X: NN (the forward
// with transposed weights, and the input gradient) runs faster on the 128x256 kernel at
// every encoder shape; NT takes the 256x256 kernel with 64-deep stages (a few per cent
// faster than with 32-deep ones) and the weight gradient (TN, split over K to fill the
// chip) the 256x256 kernel.
hipError_t gemm_big(int layout, int epi, const GemmArgs& a, hipStream_t s) {
  switch (layout) {
    case GEMM_NT: return dispatch_nt64(a, epi, s);
    case GEMM_NN: return dispatch_nn(a, epi, s);
    case GEMM_TN: return dispatch_big<true, true>(a, epi, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpipe
