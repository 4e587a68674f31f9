// Internal launch interface between the host sequencer and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpipe {

enum { DT_F32 = 0, DT_BF16 = 1 };
enum { GEMM_NT = 0, GEMM_NN = 1, GEMM_TN = 2 };
enum { EPI_STORE = 0, EPI_GELU = 1, EPI_RESID = 2, EPI_GELU_BWD = 3, EPI_F32 = 4,
       EPI_STORE_ROPE = 5 };
constexpr int ATTN_TILE = 128;   // queries (forward, dQ) or keys (dK/dV) per attention work item

// C[m][n] = sum_k A(m,k) B(n,k) + epilogue.
//   NT: A[m*lda + k], B[n*ldb + k];  NN: A[m*lda + k], B[k*ldb + n];  TN: A[k*lda + m], B[k*ldb + n]
//   kps: K range per split (multiple of the K step; <= 0 means no split); split s
//        covers [s*kps, (s+1)*kps) and writes C + s*split_stride (EPI_F32 only).
//   EPI_STORE     C(T)   = acc + bias
//   EPI_GELU      u = T(acc + bias): C(T) = GELU(u), C2(T) = GELU'(u) (optional)
//   EPI_RESID     C(f32) = aux(f32, may alias C, may be null) + acc + bias
//   EPI_GELU_BWD  C(T)   = acc * aux(T)   (aux = the GELU'(u) the forward stored)
//   EPI_F32       C(f32) = acc (+ C if beta)
//   EPI_STORE_ROPE C(T)  = EPI_STORE, then the 2D rotary position on columns < rope_cols
struct GemmArgs {
  const void* A = nullptr;
  const void* B = nullptr;
  int64_t lda = 0, ldb = 0;
  int M = 0, N = 0, K = 0, kps = 0;
  int tiles_m = 0, tiles_n = 0;
  void* C = nullptr;
  int64_t ldc = 0, split_stride = 0;
  const void* bias = nullptr;
  const void* aux = nullptr;
  int64_t ld_aux = 0;
  void* C2 = nullptr;
  int64_t ldc2 = 0;
  int beta = 0;
  // EPI_GELU_BWD on the 128x256 NN kernel only (gemm_fused_colsum says when): column sums
  // of the stored output over each band of 64 rows, colsum[m / 64][n], fp32, row stride N
  float* colsum = nullptr;
  // EPI_STORE_ROPE: 2D rotary position on output columns n < rope_cols (the q and k
  // blocks of a qkv product, heads of rope_d columns, stored pair-interleaved as in
  // common.h); the bias of those columns is indexed by the original column.
  const int32_t* rope_pos = nullptr;
  const float2* rope_tab = nullptr;
  int rope_d = 0, rope_cols = 0;
};
hipError_t gemm(int dtype, int layout, int epi, const GemmArgs& a, hipStream_t s);
// Whether gemm() runs this problem on the NN kernel that can write GemmArgs::colsum.
bool gemm_fused_colsum(int dtype, int layout, int epi, const GemmArgs& a);
// out[c] += sum of part[r][c] over r < rows, in a fixed order (two stages).
hipError_t partials_reduce(float* part, float* out, int64_t rows, int n, hipStream_t s);
// large-tile bf16 kernels (M >= 512, N >= 256): 128x256 NN, 256x256 NT (64-deep K
// stages) and TN; same contract as gemm()
hipError_t gemm_big(int layout, int epi, const GemmArgs& a, hipStream_t s);

struct AttnArgs {
  const void* q = nullptr;     // Q, K, V column blocks, row stride ld (head h at column h*d)
  const void* k = nullptr;
  const void* v = nullptr;
  int64_t ld = 0;
  const void* o = nullptr;     // O and dO, row stride ldo
  const void* d_o = nullptr;
  int64_t ldo = 0;
  void* out = nullptr;         // forward output O (row stride ldo)
  void* dq = nullptr;          // backward outputs, row stride ldd
  void* dk = nullptr;
  void* dv = nullptr;
  int64_t ldd = 0;
  float* lse = nullptr;        // [heads][N], natural log
  // [heads][N] -rowsum(dO o O), stored negated so that the bf16 kernels can start their
  // dP accumulators with it: written by the dQ kernel, read by the dK/dV kernel
  const float* delta = nullptr;
  float* delta_out = nullptr;
  const int4* work = nullptr;  // (tile start row, segment start, segment end, 0)
  int n_work = 0;
  int heads = 0;
  int64_t N = 0;
  float scale = 0.f;
  // Backward only: q and k are stored pair-interleaved with the rotary position applied
  // (the forward's fused qkv epilogue); dQ and dK are then written rotated back and in
  // the original column order.  Null: plain columns, no rotation.
  const int32_t* rope_pos = nullptr;
  const float2* rope_tab = nullptr;
};
bool attention_supported(int dtype, int head_dim);
hipError_t attention_fwd(int dtype, int head_dim, const AttnArgs& a, hipStream_t s);
// dQ over query tiles (work = query tiles; also writes delta_out = rowsum(dO o O));
// then dK, dV over key tiles (work = key tiles; reads delta)
hipError_t attention_bwd_dq(int dtype, int head_dim, const AttnArgs& a, hipStream_t s);
hipError_t attention_bwd_dkdv(int dtype, int head_dim, const AttnArgs& a, hipStream_t s);

hipError_t layernorm_fwd(int dtype, const float* X, int64_t ldx, int64_t rows, int n,
                         const void* g, const void* b, float eps, void* Y, int64_t ldy,
                         float* mean, float* rstd, hipStream_t s);
int64_t layernorm_bwd_partial_rows(int64_t rows);
// dX, dres and dXt use the row stride ldx of X.  dX == nullptr computes only the affine
// gradients (dXt and dres are then ignored).  grad_g, grad_b and grad_c (nullable) are
// accumulated (+=) with the column sums of dy*xhat, dy and the written dX (grad_c needs dX);
// part_g, part_b and part_c each hold layernorm_bwd_partial_rows(rows) x n floats.
hipError_t layernorm_bwd(int dtype, const float* dY, int64_t ldd, const float* X, int64_t ldx,
                         const float* mean, const float* rstd, const void* g, int64_t rows, int n,
                         const float* dres, float* dX, void* dXt, float* part_g, float* part_b,
                         float* part_c, float* grad_g, float* grad_b, float* grad_c,
                         hipStream_t s);
// The two halves of layernorm_bwd, for callers that reduce on another stream: the kernel
// (part_c written when both it and dX are non-null; *blocks = the partial rows written)
// and the deterministic reduction of those partial rows into the (nullable) targets.
// dY is fp32, or bf16 (dy_dtype DT_BF16, with a bf16 layer only)
hipError_t layernorm_bwd_partials(int dtype, const void* dY, int dy_dtype, int64_t ldd,
                                  const float* X, int64_t ldx, const float* mean, const float* rstd,
                                  const void* g, int64_t rows, int n, const float* dres, float* dX,
                                  void* dXt, float* part_g, float* part_b, float* part_c,
                                  int64_t* blocks, hipStream_t s);
hipError_t layernorm_bwd_reduce(float* part_g, float* grad_g, float* part_b, float* grad_b,
                                float* part_c, float* grad_c, int64_t blocks, int n,
                                hipStream_t s);
int64_t colsum_partial_rows(int64_t rows);
hipError_t colsum_accumulate(int dtype_in, const void* X, int64_t ld, int64_t rows, int n,
                             float* part, float* out, hipStream_t s);
hipError_t splitk_reduce(const float* part, int splits, int64_t M, int64_t N, float* out,
                         int64_t ldo, hipStream_t s);
// Batched transpose of up to kMaxTJobs matrices in one launch: dst[c][r] = src[r][c]
// for r < rows, c < cols (row strides lds, ldd in elements; element bits are copied).
// With perm_rows > 0, source rows r < perm_rows are taken in pair-interleaved order
// within each block of perm_d rows (common.h): dst[c][s] = src[row of s][c], where s
// indexes the stored order -- the forward's qkv weight, so that its product comes out
// with q and k pair-interleaved.
struct TJob {
  const void* src = nullptr;
  int64_t lds = 0;
  void* dst = nullptr;
  int64_t ldd = 0;
  int rows = 0, cols = 0;
  int perm_rows = 0, perm_d = 0;
};
constexpr int kMaxTJobs = 4;
hipError_t transpose_batch(int dtype, const TJob* jobs, int n, hipStream_t s);
hipError_t pad_cols(int dtype, const void* src, int64_t rows, int K, void* dst, int Kp,
                    hipStream_t s);
// tab: (cos, sin) pairs [positions][d/4] of p * theta^(-4k/d); requires d % 8 == 0
hipError_t rope(int dtype, void* qk, int64_t ld, int64_t rows, int heads, int d, int kcol,
                const int32_t* pos, const float* tab, int inverse, hipStream_t s);
hipError_t rows_copy(bool scatter, const void* src, void* dst, const int64_t* idx, int64_t n_idx,
                     int64_t row_bytes, int64_t n_rows, hipStream_t s);
hipError_t check_indices(const int64_t* idx, int64_t n, int64_t n_rows, int32_t* marks,
                         int32_t* status, hipStream_t s);

}  // namespace mpipe
