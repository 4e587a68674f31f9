// Block-diagonal variable-length attention for the packed patch sequence.
//
// Each item (or temporal slice) of the micro-batch is one attention segment
// [s0, s1) of the packed rows; a query attends to every key of its own segment
// and to no other (non-causal softmax attention, scale 1/sqrt(d)).  Segment
// tables and tile work lists come from the host planner, longest segments
// first, heads innermost, so that the longest-running blocks start first.
//
// bf16 kernels (gfx950 MFMA):
//   forward  S^T = K Q^T, online softmax in fp32 (exp2 domain), O^T += V^T P^T.
//            Working on S^T puts one query per lane column, so the per-query
//            max/sum need only a 4-lane reduction and the P^T fragment is
//            already in B-operand layout for the PV product (keys are taken in
//            the permuted order {4g..4g+3, 16+4g..16+4g+3} on both operands).
//   backward two deterministic kernels that recompute P from Q, K and the LSE:
//            dK/dV per 128-key tile looping over query tiles, and dQ per
//            128-query tile looping over key tiles.  No atomics.
// head_dim 80 = three 32-wide MFMA K-steps, the last zero-padded in the register
// operand; output d-tiles of 16.
// fp32 kernels (the small fp32 configuration): plain per-row loops.
#include "common.h"
#include "internal.h"

namespace mpipe {
namespace {

// 16-row sub-tiles per wave (NS) of the bf16 kernels; a 128-row work tile takes 8 / NS
// waves.  NS = 4 reuses each LDS fragment over four MFMAs (half the LDS traffic of NS = 2)
// at one wave per SIMD; NS = 2 runs several blocks of four waves per CU: three for the
// forward and dQ kernels (two-stage tile rings, 48 KB of LDS and at most 168 registers per
// wave; measured 7.5 % and 1 % faster than two blocks with three-stage rings), two for
// dK/dV (three-stage ring, over 200 registers).
constexpr int FWD_NS = 2, DQ_NS = 2, DKDV_NS = 2;

template <int D> struct AD {
  static constexpr int NC = D / 8;                          // 16-byte chunks per row
  // d = 80: rows of 10 chunks with chunk c of row R stored at c ^ ((R >> 3) & 1), which
  // keeps both the 16-row row-fragment reads and the 8-row transposing reads on distinct
  // banks; other widths: an odd pitch (conflict-free row-fragment reads)
  static constexpr bool SWZ = (D == 80);
  static constexpr int PC = SWZ ? NC : (NC % 2 == 0) ? NC + 1 : NC;
  static constexpr int NF = D / 32;                         // full 32-wide K steps over d
  static constexpr bool REM = (D % 32) != 0;                // a last, partial 32-wide step
  static constexpr int NS32 = (D + 31) / 32;                // 32-wide K steps, padded
  static constexpr int NDT = D / 16;                        // 16-wide output d tiles
};

// ---- LDS tile helpers ------------------------------------------------------------

// Stored position of chunk c of tile row `row` (see AD::SWZ).  The same XOR maps a stored
// position back to its chunk.
template <int D>
__device__ __forceinline__ int tile_chunk(int row, int c) {
  return AD<D>::SWZ ? (c ^ ((row >> 3) & 1)) : c;
}
// A/B fragment of a 16x16x32 MFMA from a row tile: row rbase + r (rbase a multiple of 16,
// r < 16), d in [32f + 8g, +8).  The swizzle bit of such a row is bit 3 of r, so only
// the lane's own base moves and every fragment keeps a constant offset from it.
template <int D>
__device__ __forceinline__ bf16x8 frag_row(const uint4* rowt, int rbase, int r, int f, int g) {
  const int sb = AD<D>::SWZ ? (r >> 3) & 1 : 0;
  uint4 v = rowt[(rbase + r) * AD<D>::PC + 4 * f + (g ^ sb)];
  return *reinterpret_cast<bf16x8*>(&v);
}
// Register fragments of one row (query/key) straight from global memory, as 32-wide K
// steps over d.  For d = 80 the third step is padded: lane groups 0-1 hold d 64..79 and
// groups 2-3 hold zeros, so the matching LDS operand may read any finite data there (the
// first chunks of the next row, or the tile's filled pad slots past row 63), and every
// product over d is one chain of 16x16x32 MFMAs.
template <int D> struct RowFrag {
  bf16x8 f[AD<D>::NS32];
};
template <int D>
__device__ __forceinline__ void load_rowfrag(RowFrag<D>& R, const bf16* X, int64_t ld, int row,
                                             int g) {
  const bf16* base = X + (int64_t)row * ld;
#pragma unroll
  for (int f = 0; f < AD<D>::NS32; ++f) {
    const int col = 32 * f + 8 * g;
    if (col < D) {
      uint4 v = *reinterpret_cast<const uint4*>(base + col);
      R.f[f] = *reinterpret_cast<bf16x8*>(&v);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) R.f[f][e] = (bf16)0.f;
    }
  }
}

// acc += A(row tile, rows rbase + 0..15) x B(register fragment) over d
template <int D>
__device__ __forceinline__ f32x4 dot_d(const uint4* rowt, int rbase, int r, const RowFrag<D>& B,
                                       int g, f32x4 acc) {
#pragma unroll
  for (int f = 0; f < AD<D>::NS32; ++f)
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(frag_row<D>(rowt, rbase, r, f, g), B.f[f], acc,
                                                  0, 0, 0);
  return acc;
}

// 2^x on the transcendental unit (v_exp_f32).  Inputs here are <= 0 (or -inf); results
// below the normal range flush to zero, which cannot change a softmax weight in bf16.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bf16x8 pack8(const f32x4& a, const f32x4& b) {
  bf16x8 r;
  r[0] = (bf16)a[0]; r[1] = (bf16)a[1]; r[2] = (bf16)a[2]; r[3] = (bf16)a[3];
  r[4] = (bf16)b[0]; r[5] = (bf16)b[1]; r[6] = (bf16)b[2]; r[7] = (bf16)b[3];
  return r;
}

// ---- asynchronous tile pipeline ------------------------------------------------------
// A tile is 64 rows x D of one head, stored row-major in LDS with a pitch of PC 16-byte
// chunks (tile_chunk gives a chunk's stored position).  It is filled by 16-byte
// global->LDS DMA (global_load_lds): lane l of a wave instruction writes LDS slot
// base + l, so each lane picks the source of its slot; pad slots duplicate chunk 0
// and rows past the segment read a clamped (valid) row.  Transposed operands come
// from the same raw tile through ds_read_b64_tr_b16.
template <int D, int NW> struct TG {
  static constexpr int PC = AD<D>::PC;
  static constexpr int SLOTS = (64 * PC + 64 * NW - 1) / (64 * NW) * (64 * NW);   // whole
  static constexpr int NI = SLOTS / (64 * NW);   // wave instructions; instructions per wave
};
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// UW: take the wave index as a uniform (scalar) value; which choice gives the better
// code differs by kernel (measured: the forward and dQ kernels prefer it, dK/dV does not).
template <int D, int NW, bool UW = true>
__device__ __forceinline__ void dma_tile(uint4* tile, const bf16* X, int64_t ld, int r0,
                                         int rlast) {
  constexpr int PC = AD<D>::PC, NC = AD<D>::NC;
  const int w = UW ? __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) : threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < TG<D, NW>::NI; ++i) {
    const int inst = i * NW + w;
    const int slot = inst * 64 + lane;
    int row = slot / PC, ch = tile_chunk<D>(row, slot % PC);
    ch = ch < NC ? ch : 0;
    row = row < 64 ? row : 63;   // slots past the 64 rows repeat the last row
    int grow = r0 + row;
    grow = grow < rlast ? grow : rlast;
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(X + (int64_t)grow * ld + 8 * ch),
                                     (lds_void*)(tile + inst * 64), 16, 0, 0);
  }
}
// The same DMA for a full tile (r0 + 63 <= rlast), from per-lane source offsets computed
// once per kernel: one 64-bit add per instruction instead of the clamp and multiply.
template <int D, int NW> struct TileSrc {
  int64_t off[TG<D, NW>::NI];
};
template <int D, int NW>
__device__ __forceinline__ void tile_src_init(TileSrc<D, NW>& S, int64_t ld) {
  constexpr int PC = AD<D>::PC, NC = AD<D>::NC;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < TG<D, NW>::NI; ++i) {
    const int slot = (i * NW + w) * 64 + lane;
    int row = slot / PC, ch = tile_chunk<D>(row, slot % PC);
    ch = ch < NC ? ch : 0;
    row = row < 64 ? row : 63;
    S.off[i] = (int64_t)row * ld + 8 * ch;
  }
}
template <int D, int NW>
__device__ __forceinline__ void dma_tile_full(uint4* tile, const bf16* Xr0, const TileSrc<D, NW>& S) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
  for (int i = 0; i < TG<D, NW>::NI; ++i)
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(Xr0 + S.off[i]),
                                     (lds_void*)(tile + (i * NW + w) * 64), 16, 0, 0);
}
// 64 floats (one per query of a tile, rows clamped) by a 4-byte DMA from wave 0
__device__ __forceinline__ void dma_vec64(float* dst, const float* src, int r0, int rlast) {
  if ((threadIdx.x >> 6) == 0) {
    int r = r0 + (threadIdx.x & 63);
    r = r < rlast ? r : rlast;
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(src + r),
                                     (lds_void*)(dst), 4, 0, 0);
  }
}
// Wait until at most `n` of this wave's vector-memory operations are outstanding
// (gfx9 s_waitcnt encoding: vmcnt in bits 3:0 and 15:14; expcnt, lgkmcnt left at max).
template <int n>
__device__ __forceinline__ void wait_vm() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (15 << 8) | (((n >> 4) & 3) << 14));
}
// Workgroup barrier without the release fence of __syncthreads (which would wait for
// every outstanding DMA); LDS reads are finished before it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));   // lgkmcnt(0)
  asm volatile("s_barrier" ::: "memory");
}
// Transposed fragment of a raw [row][d] tile: for the 16-lane group g of this lane, rows
// {kb + 4g ..+3} then {kb + 16 + 4g ..+3} at column c0 + (lane & 15).
template <int D>
__device__ __forceinline__ bf16x8 frag_trt(const uint4* tile, int kb, int c0, int g, int r) {
  // rows kb + 4g + r/4 (first read) and 16 further (second read), kb a multiple of 8: the
  // swizzle bit of those rows is bit 1 of g.  Lane r reads 8 bytes at column c0 + 4 (r mod 4).
  constexpr int PC = AD<D>::PC;
  const char* base = reinterpret_cast<const char*>(tile);
  const int sb = AD<D>::SWZ ? (g >> 1) & 1 : 0;
  const int lane_off = ((4 * g + (r >> 2)) * PC + (((r & 3) >> 1) ^ sb)) * 16 + (r & 1) * 8;
  const int off = (kb * PC + c0 / 8) * 16 + lane_off;
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + off));
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + off + 16 * PC * 16));
  bf16x8 v;
  const bf16* pa = reinterpret_cast<const bf16*>(&a);
  const bf16* pb = reinterpret_cast<const bf16*>(&b);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[e] = pa[e];
    v[4 + e] = pb[e];
  }
  return v;
}

// ---- forward ----------------------------------------------------------------------
// 2-stage pipeline over 64-key tiles: tile t+1 is in flight while tile t is used, and
// the other two blocks on the CU cover what one tile of lookahead leaves exposed.
// The softmax offset m of a query (log2 domain) moves only when the tile's maximum
// exceeds it by more than kRescaleLog2: weights exp2(s - m) then stay below 2^8, exact in
// fp32 and as representable in bf16 as any weight <= 1, and the output rescale (a
// multiply per accumulator) runs on a few tiles instead of most.  Row sums of the bf16
// weights come from the PV MFMAs themselves, with a ones operand in place of V.
template <int D, int NS>
__global__ __launch_bounds__(64 * (8 / NS), NS == 2 ? 3 : 1) void attn_fwd_kernel(AttnArgs p) {
  constexpr int NW = 8 / NS, RW = 16 * NS;   // waves per block, rows per wave
  constexpr int NDT = AD<D>::NDT, SL = TG<D, NW>::SLOTS;
  __shared__ uint4 k0s[SL], k1s[SL], v0s[SL], v1s[SL];
  const int work = blockIdx.x / p.heads, head = blockIdx.x % p.heads;
  const int4 wk = p.work[work];
  const int q0 = wk.x, s0 = wk.y, s1 = wk.z;
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, g = l >> 4, r = l & 15;
  const bf16* Q = reinterpret_cast<const bf16*>(p.q) + head * D;
  const bf16* K = reinterpret_cast<const bf16*>(p.k) + head * D;
  const bf16* V = reinterpret_cast<const bf16*>(p.v) + head * D;
  const float sl2 = p.scale * kLog2e;
  const int nt = (s1 - s0 + 63) / 64;
  constexpr float kRescaleLog2 = 8.0f;
  bf16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = (bf16)1.0f;

  RowFrag<D> qf[NS];
  int qrow[NS];
#pragma unroll
  for (int qs = 0; qs < NS; ++qs) {
    qrow[qs] = q0 + RW * w + 16 * qs + r;
    load_rowfrag<D>(qf[qs], Q, p.ld, min(qrow[qs], s1 - 1), g);
  }
  float m[NS];
  f32x4 o[NS][NDT], osum[NS];   // osum: every element holds the query's weight sum
#pragma unroll
  for (int qs = 0; qs < NS; ++qs) {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) o[qs][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    osum[qs] = f32x4{0.f, 0.f, 0.f, 0.f};
    m[qs] = -INFINITY;
  }

  TileSrc<D, NW> kvsrc;
  tile_src_init<D, NW>(kvsrc, p.ld);
  auto issue = [&](int t, uint4* kt, uint4* vt) __attribute__((always_inline)) {
    if (t < nt) {
      const int r0 = s0 + 64 * t;
      if (r0 + 63 <= s1 - 1) {
        dma_tile_full<D, NW>(kt, K + (int64_t)r0 * p.ld, kvsrc);
        dma_tile_full<D, NW>(vt, V + (int64_t)r0 * p.ld, kvsrc);
      } else {
        dma_tile<D, NW>(kt, K, p.ld, r0, s1 - 1);
        dma_tile<D, NW>(vt, V, p.ld, r0, s1 - 1);
      }
    }
  };
  auto body = [&](int t, const uint4* kt_s, const uint4* vt_s, uint4* kn, uint4* vn)
      __attribute__((always_inline)) {
    wait_vm<0>();
    lds_barrier();
    // MFMA stretches run at raised wave priority, so that the waves sharing the SIMD issue
    // their softmax VALU work beside them rather than ahead of them (all three kernels do
    // this; same-call A/B: backward 1.5 % faster, step 293.1 -> 289.5 ms)
    __builtin_amdgcn_s_setprio(1);
    const int k0 = s0 + 64 * t;
    f32x4 s[4][NS];
#pragma unroll
    for (int kq = 0; kq < 4; ++kq)
#pragma unroll
      for (int qs = 0; qs < NS; ++qs)
        s[kq][qs] = dot_d<D>(kt_s, 16 * kq, r, qf[qs], g, f32x4{0.f, 0.f, 0.f, 0.f});
    // the next DMAs go out after the score MFMAs, not ahead of their fragment reads
    // (measured 3% faster on the Qwen2-VL segment mix)
    issue(t + 1, kn, vn);
    __builtin_amdgcn_s_setprio(0);
    if (k0 + 64 > s1) {   // ragged last tile: keys past the segment never win or weigh
#pragma unroll
      for (int kq = 0; kq < 4; ++kq)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const bool out = k0 + 16 * kq + 4 * g + v >= s1;
#pragma unroll
          for (int qs = 0; qs < NS; ++qs) s[kq][qs][v] = out ? -INFINITY : s[kq][qs][v];
        }
    }
    bf16x8 pb[NS][2];
#pragma unroll
    for (int qs = 0; qs < NS; ++qs) {
      // running max in the scaled log2 domain; scaling by sl2 > 0 commutes with max
      float mx = -INFINITY;
#pragma unroll
      for (int kq = 0; kq < 4; ++kq)
#pragma unroll
        for (int v = 0; v < 4; ++v) mx = fmaxf(mx, s[kq][qs][v]);
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      // move the offset (and rescale, uniformly skipped when no query needs it) only
      // when the tile's maximum exceeds it by more than kRescaleLog2
      const float mt = mx * sl2;
      if (__any(mt > m[qs] + kRescaleLog2)) {
        const float mn = mt > m[qs] + kRescaleLog2 ? mt : m[qs];
        const float alpha = fast_exp2(m[qs] - mn);
        m[qs] = mn;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) o[qs][dt] *= alpha;
        osum[qs] *= alpha;
      }
      const float mq = m[qs];
#pragma unroll
      for (int kq = 0; kq < 4; ++kq)
#pragma unroll
        for (int v = 0; v < 4; ++v) s[kq][qs][v] = fast_exp2(fmaf(s[kq][qs][v], sl2, -mq));
      pb[qs][0] = pack8(s[0][qs], s[1][qs]);
      pb[qs][1] = pack8(s[2][qs], s[3][qs]);
    }
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const bf16x8 a = frag_trt<D>(vt_s, 32 * kk, 16 * dt, g, r);
#pragma unroll
        for (int qs = 0; qs < NS; ++qs)
          o[qs][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[qs][kk], o[qs][dt], 0, 0, 0);
      }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int qs = 0; qs < NS; ++qs)
        osum[qs] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[qs][kk], osum[qs], 0, 0, 0);
    __builtin_amdgcn_s_setprio(0);
  };
  issue(0, k0s, v0s);
  for (int t = 0; t < nt; t += 2) {
    body(t, k0s, v0s, k1s, v1s);
    if (t + 1 < nt) body(t + 1, k1s, v1s, k0s, v0s);
  }
  bf16* O = reinterpret_cast<bf16*>(p.out) + head * D;
#pragma unroll
  for (int qs = 0; qs < NS; ++qs) {
    const float tot = osum[qs][0];
    const int q = qrow[qs];
    if (q < s1) {
      const float inv = 1.0f / tot;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        bf16 v4[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) v4[v] = (bf16)(o[qs][dt][v] * inv);
        *reinterpret_cast<uint2*>(O + (int64_t)q * p.ldo + 16 * dt + 4 * g) =
            *reinterpret_cast<uint2*>(v4);
      }
      if (g == 0 && p.lse) p.lse[(int64_t)head * p.N + q] = (m[qs] + log2f(tot)) * kLn2;
    }
  }
}

// ---- backward: dK, dV ------------------------------------------------------------
// Per 128-key tile (32 keys per wave), 3-stage pipeline over 64-query tiles of Q, dO,
// LSE and delta.
template <int D, int NS>
__global__ __launch_bounds__(64 * (8 / NS), NS == 2 ? 2 : 1) void attn_bwd_dkdv_kernel(AttnArgs p) {
  constexpr int NW = 8 / NS, RW = 16 * NS;   // waves per block, rows per wave
  constexpr int NDT = AD<D>::NDT, SL = TG<D, NW>::SLOTS, NI = TG<D, NW>::NI;
  __shared__ uint4 q0s[SL], q1s[SL], q2s[SL], d0s[SL], d1s[SL], d2s[SL];
  __shared__ __attribute__((aligned(16))) float l0s[64], l1s[64], l2s[64], e0s[64], e1s[64], e2s[64];
  const int work = blockIdx.x / p.heads, head = blockIdx.x % p.heads;
  const int4 wk = p.work[work];
  const int k0 = wk.x, s0 = wk.y, s1 = wk.z;
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, g = l >> 4, r = l & 15;
  const bf16* Q = reinterpret_cast<const bf16*>(p.q) + head * D;
  const bf16* K = reinterpret_cast<const bf16*>(p.k) + head * D;
  const bf16* V = reinterpret_cast<const bf16*>(p.v) + head * D;
  const bf16* dO = reinterpret_cast<const bf16*>(p.d_o) + head * D;
  const float* LSE = p.lse + (int64_t)head * p.N;
  const float* DEL = p.delta + (int64_t)head * p.N;
  const float sl2 = p.scale * kLog2e;
  const int nt = (s1 - s0 + 63) / 64;
  constexpr int PER_TILE = 2 * NI + 2;   // wave 0 issues the two 4-byte vectors too

  RowFrag<D> kf[NS], vf[NS];
#pragma unroll
  for (int ks = 0; ks < NS; ++ks) {
    const int key = min(k0 + RW * w + 16 * ks + r, s1 - 1);
    load_rowfrag<D>(kf[ks], K, p.ld, key, g);
    load_rowfrag<D>(vf[ks], V, p.ld, key, g);
  }
  f32x4 dk[NS][NDT], dv[NS][NDT];
#pragma unroll
  for (int ks = 0; ks < NS; ++ks)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) dk[ks][dt] = dv[ks][dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // (per-tile source arithmetic here: keeping precomputed offsets live measured slower,
  // the extra registers spill in this kernel)
  auto issue = [&](int t, uint4* qt, uint4* dt_, float* lt, float* et)
      __attribute__((always_inline)) {
    if (t < nt) {
      const int r0 = s0 + 64 * t;
      dma_tile<D, NW, false>(qt, Q, p.ld, r0, s1 - 1);
      dma_tile<D, NW, false>(dt_, dO, p.ldo, r0, s1 - 1);
      dma_vec64(lt, LSE, r0, s1 - 1);
      dma_vec64(et, DEL, r0, s1 - 1);
    }
  };
  auto body = [&](int t, const uint4* q_s, const uint4* do_s, const float* lse_s,
                  const float* del_s, uint4* qn, uint4* dn, float* ln, float* en)
      __attribute__((always_inline)) {
    if (w == 0) {
      if (t + 1 < nt) wait_vm<PER_TILE>();
      else wait_vm<0>();
    } else {
      if (t + 1 < nt) wait_vm<2 * NI>();
      else wait_vm<0>();
    }
    lds_barrier();
    issue(t + 2, qn, dn, ln, en);
    const int qb = s0 + 64 * t;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      f32x4 P[2][NS], dS[2][NS];   // [query half][ks]
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int qb16 = 16 * (2 * kk + h2);
        const int q4 = 16 * (2 * kk + h2) + 4 * g;   // this lane's four queries
        const float4 lq = *reinterpret_cast<const float4*>(lse_s + q4);
        const float4 eq = *reinterpret_cast<const float4*>(del_s + q4);
        const float nl[4] = {-lq.x * kLog2e, -lq.y * kLog2e, -lq.z * kLog2e, -lq.w * kLog2e};
        const f32x4 mde = {eq.x, eq.y, eq.z, eq.w};   // -delta as stored
#pragma unroll
        for (int ks = 0; ks < NS; ++ks) {
          f32x4 s = dot_d<D>(q_s, qb16, r, kf[ks], g, f32x4{0.f, 0.f, 0.f, 0.f});
          // the dP accumulator starts at -delta, so the products leave dP - delta
          f32x4 dpd = dot_d<D>(do_s, qb16, r, vf[ks], g, mde);
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const float pp = fast_exp2(fmaf(s[v], sl2, nl[v]));
            P[h2][ks][v] = pp;
            dS[h2][ks][v] = pp * dpd[v];
          }
        }
        if (qb + 64 > s1) {   // ragged last tile: queries past the segment contribute nothing
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const bool out = qb + q4 + v >= s1;
#pragma unroll
            for (int ks = 0; ks < NS; ++ks) {
              P[h2][ks][v] = out ? 0.f : P[h2][ks][v];
              dS[h2][ks][v] = out ? 0.f : dS[h2][ks][v];
            }
          }
        }
      }
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int ks = 0; ks < NS; ++ks) {
        const bf16x8 ap = pack8(P[0][ks], P[1][ks]);
        const bf16x8 ads = pack8(dS[0][ks], dS[1][ks]);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const bf16x8 bdo = frag_trt<D>(do_s, 32 * kk, 16 * dt, g, r);
          const bf16x8 bq = frag_trt<D>(q_s, 32 * kk, 16 * dt, g, r);
          dv[ks][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap, bdo, dv[ks][dt], 0, 0, 0);
          dk[ks][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ads, bq, dk[ks][dt], 0, 0, 0);
        }
      }
      __builtin_amdgcn_s_setprio(0);
    }
  };
  issue(0, q0s, d0s, l0s, e0s);
  issue(1, q1s, d1s, l1s, e1s);
  for (int t = 0; t < nt; t += 3) {
    body(t, q0s, d0s, l0s, e0s, q2s, d2s, l2s, e2s);
    if (t + 1 < nt) body(t + 1, q1s, d1s, l1s, e1s, q0s, d0s, l0s, e0s);
    if (t + 2 < nt) body(t + 2, q2s, d2s, l2s, e2s, q1s, d1s, l1s, e1s);
  }
  bf16* dK = reinterpret_cast<bf16*>(p.dk) + head * D;
  bf16* dV = reinterpret_cast<bf16*>(p.dv) + head * D;
  if (p.rope_pos != nullptr) {
    // q, k pair-interleaved and rotated: rotate each dK pair (stored columns c & ~1,
    // c | 1, in lanes r & ~1, r | 1) back and write it in the original column order.  The
    // rotary factors of the lane's keys and column pairs are all loaded first.
    float2 cs[NS][4][NDT];
#pragma unroll
    for (int ks = 0; ks < NS; ++ks)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int key = min(k0 + RW * w + 16 * ks + 4 * g + v, s1 - 1);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
          cs[ks][v][dt] = rope_cs(p.rope_pos, p.rope_tab, D, key, (16 * dt + r) >> 1);
      }
#pragma unroll
    for (int ks = 0; ks < NS; ++ks)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int key = k0 + RW * w + 16 * ks + 4 * g + v;   // the same in lanes r, r ^ 1
        if (key >= s1) continue;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const float x = dk[ks][dt][v] * p.scale;
          const float y = __shfl_xor(x, 1);
          const float2 c = cs[ks][v][dt];
          dK[(int64_t)key * p.ldd + rope_component(16 * dt + r, D)] =
              (bf16)((r & 1) ? rope_second(y, x, c, true) : rope_first(x, y, c, true));
          dV[(int64_t)key * p.ldd + 16 * dt + r] = (bf16)(dv[ks][dt][v]);
        }
      }
    return;
  }
#pragma unroll
  for (int ks = 0; ks < NS; ++ks)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int key = k0 + RW * w + 16 * ks + 4 * g + v;
      if (key >= s1) continue;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        dK[(int64_t)key * p.ldd + 16 * dt + r] = (bf16)(dk[ks][dt][v] * p.scale);
        dV[(int64_t)key * p.ldd + 16 * dt + r] = (bf16)(dv[ks][dt][v]);
      }
    }
}

// ---- backward: dQ (and delta) --------------------------------------------------------
template <int D, int NS>
__global__ __launch_bounds__(64 * (8 / NS), NS == 2 ? 3 : 1) void attn_bwd_dq_kernel(AttnArgs p) {
  constexpr int NW = 8 / NS, RW = 16 * NS;   // waves per block, rows per wave
  constexpr int NDT = AD<D>::NDT, SL = TG<D, NW>::SLOTS;
  __shared__ uint4 k0s[SL], k1s[SL], v0s[SL], v1s[SL];
  const int work = blockIdx.x / p.heads, head = blockIdx.x % p.heads;
  const int4 wk = p.work[work];
  const int q0 = wk.x, s0 = wk.y, s1 = wk.z;
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, g = l >> 4, r = l & 15;
  const bf16* Q = reinterpret_cast<const bf16*>(p.q) + head * D;
  const bf16* K = reinterpret_cast<const bf16*>(p.k) + head * D;
  const bf16* V = reinterpret_cast<const bf16*>(p.v) + head * D;
  const bf16* dO = reinterpret_cast<const bf16*>(p.d_o) + head * D;
  const bf16* O = reinterpret_cast<const bf16*>(p.o) + head * D;
  const float sl2 = p.scale * kLog2e;
  const int nt = (s1 - s0 + 63) / 64;

  RowFrag<D> qf[NS], dof[NS];
  int qrow[NS];
  float lse2[NS];
  f32x4 mdel[NS];   // -delta of the lane's query, in every element
#pragma unroll
  for (int qs = 0; qs < NS; ++qs) {
    qrow[qs] = q0 + RW * w + 16 * qs + r;
    const int qc = min(qrow[qs], s1 - 1);
    load_rowfrag<D>(qf[qs], Q, p.ld, qc, g);
    load_rowfrag<D>(dof[qs], dO, p.ldo, qc, g);
    lse2[qs] = p.lse[(int64_t)head * p.N + qc] * kLog2e;
    // delta = rowsum(dO o O): each lane holds d-chunks of its query; the four lane
    // groups together cover all d
    RowFrag<D> of;
    load_rowfrag<D>(of, O, p.ldo, qc, g);
    float dl = 0.f;
#pragma unroll
    for (int f = 0; f < AD<D>::NS32; ++f)   // (padded lanes hold zeros)
#pragma unroll
      for (int e = 0; e < 8; ++e) dl += (float)of.f[f][e] * (float)dof[qs].f[f][e];
    dl += __shfl_xor(dl, 16);
    dl += __shfl_xor(dl, 32);
    mdel[qs] = f32x4{-dl, -dl, -dl, -dl};
    if (g == 0 && qrow[qs] < s1) p.delta_out[(int64_t)head * p.N + qrow[qs]] = -dl;
  }
  f32x4 dq[NS][NDT];
#pragma unroll
  for (int qs = 0; qs < NS; ++qs)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) dq[qs][dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  TileSrc<D, NW> kvsrc;
  tile_src_init<D, NW>(kvsrc, p.ld);
  auto issue = [&](int t, uint4* kt, uint4* vt) __attribute__((always_inline)) {
    if (t < nt) {
      const int r0 = s0 + 64 * t;
      if (r0 + 63 <= s1 - 1) {
        dma_tile_full<D, NW>(kt, K + (int64_t)r0 * p.ld, kvsrc);
        dma_tile_full<D, NW>(vt, V + (int64_t)r0 * p.ld, kvsrc);
      } else {
        dma_tile<D, NW>(kt, K, p.ld, r0, s1 - 1);
        dma_tile<D, NW>(vt, V, p.ld, r0, s1 - 1);
      }
    }
  };
  auto body = [&](int t, const uint4* k_s, const uint4* v_s, uint4* kn, uint4* vn)
      __attribute__((always_inline)) {
    wait_vm<0>();
    lds_barrier();
    issue(t + 1, kn, vn);
    const int kb = s0 + 64 * t;
    f32x4 ds[4][NS];
#pragma unroll
    for (int kq = 0; kq < 4; ++kq)
#pragma unroll
      for (int qs = 0; qs < NS; ++qs) {
        f32x4 sv = dot_d<D>(k_s, 16 * kq, r, qf[qs], g, f32x4{0.f, 0.f, 0.f, 0.f});
        // the dP accumulator starts at -delta, so the products leave dP - delta
        f32x4 dpd = dot_d<D>(v_s, 16 * kq, r, dof[qs], g, mdel[qs]);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float pp = fast_exp2(fmaf(sv[v], sl2, -lse2[qs]));
          ds[kq][qs][v] = pp * dpd[v];
        }
      }
    if (kb + 64 > s1) {   // ragged last tile: keys past the segment contribute nothing
#pragma unroll
      for (int kq = 0; kq < 4; ++kq)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const bool out = kb + 16 * kq + 4 * g + v >= s1;
#pragma unroll
          for (int qs = 0; qs < NS; ++qs) ds[kq][qs][v] = out ? 0.f : ds[kq][qs][v];
        }
    }
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      bf16x8 b[NS];
#pragma unroll
      for (int qs = 0; qs < NS; ++qs) b[qs] = pack8(ds[2 * kk][qs], ds[2 * kk + 1][qs]);
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x8 a = frag_trt<D>(k_s, 32 * kk, 16 * dt, g, r);
#pragma unroll
        for (int qs = 0; qs < NS; ++qs)
          dq[qs][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[qs], dq[qs][dt], 0, 0, 0);
      }
    }
    __builtin_amdgcn_s_setprio(0);
  };
  issue(0, k0s, v0s);
  for (int t = 0; t < nt; t += 2) {
    body(t, k0s, v0s, k1s, v1s);
    if (t + 1 < nt) body(t + 1, k1s, v1s, k0s, v0s);
  }
  bf16* dQ = reinterpret_cast<bf16*>(p.dq) + head * D;
  if (p.rope_pos != nullptr) {
    // q, k pair-interleaved and rotated: stored columns 16 dt + 4 g .. +3 of a lane are the
    // rotary pairs j0 = 8 dt + 2 g and j0 + 1 (one axis, consecutive table entries).  Their
    // factors are all loaded first; each pair is rotated back and written as components
    // j0, j0 + 1 and j0 + D/2, j0 + 1 + D/2.
    constexpr int Q4 = D / 4;
#pragma unroll
    for (int qs = 0; qs < NS; ++qs) {
      const int q = qrow[qs];
      const uint32_t pp = (uint32_t)p.rope_pos[min(q, s1 - 1)];
      float4 cs[NDT];
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const int j0 = 8 * dt + 2 * g;
        const int coord = (int)(j0 < Q4 ? (pp >> 16) : (pp & 0xFFFFu));
        cs[dt] = *reinterpret_cast<const float4*>(p.rope_tab + coord * Q4 +
                                                  (j0 < Q4 ? j0 : j0 - Q4));
      }
      if (q >= s1) continue;
      bf16* row = dQ + (int64_t)q * p.ldd;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        float x[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) x[v] = dq[qs][dt][v] * p.scale;
        const float4 c = cs[dt];
        rope_unrotate(x[0], x[1], make_float2(c.x, c.y));
        rope_unrotate(x[2], x[3], make_float2(c.z, c.w));
        const int j0 = 8 * dt + 2 * g;
        bf16 a2[2] = {(bf16)x[0], (bf16)x[2]}, b2[2] = {(bf16)x[1], (bf16)x[3]};
        *reinterpret_cast<uint32_t*>(row + j0) = *reinterpret_cast<uint32_t*>(a2);
        *reinterpret_cast<uint32_t*>(row + j0 + D / 2) = *reinterpret_cast<uint32_t*>(b2);
      }
    }
    return;
  }
#pragma unroll
  for (int qs = 0; qs < NS; ++qs) {
    const int q = qrow[qs];
    if (q >= s1) continue;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      bf16 v4[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) v4[v] = (bf16)(dq[qs][dt][v] * p.scale);
      *reinterpret_cast<uint2*>(dQ + (int64_t)q * p.ldd + 16 * dt + 4 * g) =
          *reinterpret_cast<uint2*>(v4);
    }
  }
}

// ---- -delta = -rowsum(dO o O) per (head, query), stored negated --------------------------

template <class T>
__global__ void attn_delta_kernel(const T* O, const T* dO, int64_t ldo, int64_t N, int heads,
                                  int d, float* delta) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N * heads) return;
  const int64_t q = i / heads;
  const int hd = (int)(i % heads);
  float s = 0.f;
  for (int e = 0; e < d; ++e)
    s += to_f(O[q * ldo + hd * d + e]) * to_f(dO[q * ldo + hd * d + e]);
  delta[(int64_t)hd * N + q] = -s;
}

// ---- fp32 kernels: one thread per query (forward, dQ) or per key (dK, dV) -------------

template <int D>
__global__ void attn_fwd_f32_kernel(AttnArgs p) {
  const int work = blockIdx.x / p.heads, head = blockIdx.x % p.heads;
  const int4 wk = p.work[work];
  const int q = wk.x + threadIdx.x, s0 = wk.y, s1 = wk.z;
  if (q >= s1) return;
  const float* Q = reinterpret_cast<const float*>(p.q) + head * D;
  const float* K = reinterpret_cast<const float*>(p.k) + head * D;
  const float* V = reinterpret_cast<const float*>(p.v) + head * D;
  float qv[D], o[D];
  for (int e = 0; e < D; ++e) {
    qv[e] = Q[(int64_t)q * p.ld + e];
    o[e] = 0.f;
  }
  float m = -INFINITY, lsum = 0.f;
  for (int k = s0; k < s1; ++k) {
    float s = 0.f;
    for (int e = 0; e < D; ++e) s += qv[e] * K[(int64_t)k * p.ld + e];
    s *= p.scale;
    const float mn = fmaxf(m, s);
    const float a = expf(m - mn), e1 = expf(s - mn);
    lsum = lsum * a + e1;
    for (int e = 0; e < D; ++e) o[e] = o[e] * a + e1 * V[(int64_t)k * p.ld + e];
    m = mn;
  }
  float* Ot = reinterpret_cast<float*>(p.out) + head * D;
  for (int e = 0; e < D; ++e) Ot[(int64_t)q * p.ldo + e] = o[e] / lsum;
  if (p.lse) p.lse[(int64_t)head * p.N + q] = m + logf(lsum);
}

template <int D>
__global__ void attn_bwd_dq_f32_kernel(AttnArgs p) {
  const int work = blockIdx.x / p.heads, head = blockIdx.x % p.heads;
  const int4 wk = p.work[work];
  const int q = wk.x + threadIdx.x, s0 = wk.y, s1 = wk.z;
  if (q >= s1) return;
  const float* Q = reinterpret_cast<const float*>(p.q) + head * D;
  const float* K = reinterpret_cast<const float*>(p.k) + head * D;
  const float* V = reinterpret_cast<const float*>(p.v) + head * D;
  const float* dO = reinterpret_cast<const float*>(p.d_o) + head * D;
  float qv[D], dov[D], dq[D];
  for (int e = 0; e < D; ++e) {
    qv[e] = Q[(int64_t)q * p.ld + e];
    dov[e] = dO[(int64_t)q * p.ldo + e];
    dq[e] = 0.f;
  }
  const float L = p.lse[(int64_t)head * p.N + q], mdel = p.delta_out[(int64_t)head * p.N + q];
  for (int k = s0; k < s1; ++k) {
    float s = 0.f, dp = 0.f;
    for (int e = 0; e < D; ++e) {
      s += qv[e] * K[(int64_t)k * p.ld + e];
      dp += dov[e] * V[(int64_t)k * p.ld + e];
    }
    const float ds = expf(s * p.scale - L) * (dp + mdel);
    for (int e = 0; e < D; ++e) dq[e] += ds * K[(int64_t)k * p.ld + e];
  }
  float* dQ = reinterpret_cast<float*>(p.dq) + head * D + (int64_t)q * p.ldd;
  if (p.rope_pos != nullptr) {   // pair-interleaved q, k: rotate back, original order
    for (int j = 0; j < D / 2; ++j) {
      float a = dq[2 * j] * p.scale, b = dq[2 * j + 1] * p.scale;
      rope_unrotate(a, b, rope_cs(p.rope_pos, p.rope_tab, D, q, j));
      dQ[j] = a;
      dQ[j + D / 2] = b;
    }
  } else {
    for (int e = 0; e < D; ++e) dQ[e] = dq[e] * p.scale;
  }
}

template <int D>
__global__ void attn_bwd_dkdv_f32_kernel(AttnArgs p) {
  const int work = blockIdx.x / p.heads, head = blockIdx.x % p.heads;
  const int4 wk = p.work[work];
  const int k = wk.x + threadIdx.x, s0 = wk.y, s1 = wk.z;
  if (k >= s1) return;
  const float* Q = reinterpret_cast<const float*>(p.q) + head * D;
  const float* K = reinterpret_cast<const float*>(p.k) + head * D;
  const float* V = reinterpret_cast<const float*>(p.v) + head * D;
  const float* dO = reinterpret_cast<const float*>(p.d_o) + head * D;
  float kv[D], vv[D], dk[D], dv[D];
  for (int e = 0; e < D; ++e) {
    kv[e] = K[(int64_t)k * p.ld + e];
    vv[e] = V[(int64_t)k * p.ld + e];
    dk[e] = dv[e] = 0.f;
  }
  for (int q = s0; q < s1; ++q) {
    float s = 0.f, dp = 0.f;
    for (int e = 0; e < D; ++e) {
      s += Q[(int64_t)q * p.ld + e] * kv[e];
      dp += dO[(int64_t)q * p.ldo + e] * vv[e];
    }
    const float pp = expf(s * p.scale - p.lse[(int64_t)head * p.N + q]);
    const float ds = pp * (dp + p.delta[(int64_t)head * p.N + q]);
    for (int e = 0; e < D; ++e) {
      dv[e] += pp * dO[(int64_t)q * p.ldo + e];
      dk[e] += ds * Q[(int64_t)q * p.ld + e];
    }
  }
  float* dK = reinterpret_cast<float*>(p.dk) + head * D + (int64_t)k * p.ldd;
  float* dV = reinterpret_cast<float*>(p.dv) + head * D + (int64_t)k * p.ldd;
  for (int e = 0; e < D; ++e) dV[e] = dv[e];
  if (p.rope_pos != nullptr) {   // pair-interleaved q, k: rotate back, original order
    for (int j = 0; j < D / 2; ++j) {
      float a = dk[2 * j] * p.scale, b = dk[2 * j + 1] * p.scale;
      rope_unrotate(a, b, rope_cs(p.rope_pos, p.rope_tab, D, k, j));
      dK[j] = a;
      dK[j + D / 2] = b;
    }
  } else {
    for (int e = 0; e < D; ++e) dK[e] = dk[e] * p.scale;
  }
}

template <int D>
hipError_t fwd_bf16(const AttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((attn_fwd_kernel<D, FWD_NS>), dim3(a.n_work * a.heads), dim3(64 * (8 / FWD_NS)), 0, s, a);
  return hipGetLastError();
}
template <int D>
hipError_t dq_bf16(const AttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D, DQ_NS>), dim3(a.n_work * a.heads), dim3(64 * (8 / DQ_NS)), 0, s, a);
  return hipGetLastError();
}
template <int D>
hipError_t dkdv_bf16(const AttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, DKDV_NS>), dim3(a.n_work * a.heads), dim3(64 * (8 / DKDV_NS)), 0, s, a);
  return hipGetLastError();
}
template <int D>
hipError_t fwd_f32(const AttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(attn_fwd_f32_kernel<D>, dim3(a.n_work * a.heads), dim3(ATTN_TILE), 0, s, a);
  return hipGetLastError();
}
template <int D>
hipError_t dq_f32(const AttnArgs& a, hipStream_t s) {
  const int64_t n = a.N * a.heads;
  hipLaunchKernelGGL(attn_delta_kernel<float>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                     (const float*)a.o, (const float*)a.d_o, a.ldo, a.N, a.heads, D, a.delta_out);
  hipLaunchKernelGGL(attn_bwd_dq_f32_kernel<D>, dim3(a.n_work * a.heads), dim3(ATTN_TILE), 0, s, a);
  return hipGetLastError();
}
template <int D>
hipError_t dkdv_f32(const AttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(attn_bwd_dkdv_f32_kernel<D>, dim3(a.n_work * a.heads), dim3(ATTN_TILE), 0, s, a);
  return hipGetLastError();
}

}  // namespace

bool attention_supported(int dtype, int head_dim) {
  if (dtype == DT_BF16) return head_dim == 32 || head_dim == 64 || head_dim == 80;
  return head_dim == 32 || head_dim == 64 || head_dim == 80;
}

hipError_t attention_fwd(int dtype, int head_dim, const AttnArgs& a, hipStream_t s) {
  if (a.n_work == 0) return hipSuccess;
  if (dtype == DT_BF16) {
    switch (head_dim) {
      case 32: return fwd_bf16<32>(a, s);
      case 64: return fwd_bf16<64>(a, s);
      case 80: return fwd_bf16<80>(a, s);
    }
  } else {
    switch (head_dim) {
      case 32: return fwd_f32<32>(a, s);
      case 64: return fwd_f32<64>(a, s);
      case 80: return fwd_f32<80>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

#define MPIPE_ATTN_DISPATCH(BF, FP)                  \
  if (a.n_work == 0) return hipSuccess;              \
  if (dtype == DT_BF16) {                            \
    switch (head_dim) {                              \
      case 32: return BF<32>(a, s);                  \
      case 64: return BF<64>(a, s);                  \
      case 80: return BF<80>(a, s);                  \
    }                                                \
  } else {                                           \
    switch (head_dim) {                              \
      case 32: return FP<32>(a, s);                  \
      case 64: return FP<64>(a, s);                  \
      case 80: return FP<80>(a, s);                  \
    }                                                \
  }                                                  \
  return hipErrorInvalidValue;

hipError_t attention_bwd_dq(int dtype, int head_dim, const AttnArgs& a, hipStream_t s) {
  MPIPE_ATTN_DISPATCH(dq_bf16, dq_f32)
}
hipError_t attention_bwd_dkdv(int dtype, int head_dim, const AttnArgs& a, hipStream_t s) {
  MPIPE_ATTN_DISPATCH(dkdv_bf16, dkdv_f32)
}
#undef MPIPE_ATTN_DISPATCH

}  // namespace mpipe
