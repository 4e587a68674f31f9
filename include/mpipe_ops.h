/*
 * libmpipe kernel-level entry points.
 *
 * The encoder step of mpipe.h is a sequence of these operations; they are
 * exported individually so that each gfx950 kernel can be checked against the
 * CPU oracle's building block of the same name.  Same conventions as mpipe.h:
 * device pointers unless marked host, row-major, work enqueued on hip_stream,
 * status return, nothing enqueued on a non-OK status.  Calls that upload host
 * metadata (segment tables, positions) synchronize hip_stream before returning.
 */
#ifndef MPIPE_OPS_H
#define MPIPE_OPS_H
#include "mpipe.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Layouts: 0 NT  C[m][n] = sum_k A[m][k] B[n][k]     (Linear forward, Y = X W^T)
 *          1 NN  C[m][n] = sum_k A[m][k] B[k][n]     (input gradient, dX = dY W)
 *          2 TN  C[m][n] = sum_k A[k][m] B[k][n]     (weight gradient, dW = dY^T X)
 * Epilogues (acc = the sum, bias per column, cfg dtype unless noted):
 *          0 C = acc + bias
 *          1 u = acc + bias rounded to dtype: C = GELU(u), C2 = GELU'(u) (C2 optional).
 *            GELU is the erf form: fp32 evaluates erf exactly; bf16 uses the
 *            Abramowitz & Stegun 7.1.26 erf (|error| <= 1.5e-7), in every kernel.
 *          2 C(fp32) = aux(fp32, nullable, may alias C) + acc + bias
 *          3 C = acc * aux   (aux = the GELU'(u) that epilogue 1 stored: the MLP backward)
 *          4 C(fp32) = acc, or C + acc when beta != 0; with k_per_split > 0 the
 *            K range is split and split s writes C + s * split_stride.
 * Requirements: K-contiguous operands need K and their row stride to be
 * multiples of 8 (bf16) / 4 (fp32); K-major operands need their column count
 * and row stride to be multiples of 8 / 4; 16-byte aligned pointers. */
mpipe_status mpipe_op_gemm(int32_t dtype, int32_t layout, int32_t epilogue, int32_t M, int32_t N,
                           int32_t K, const void* A, int64_t lda, const void* B, int64_t ldb,
                           void* C, int64_t ldc, const void* bias, const void* aux, int64_t ld_aux,
                           void* C2, int64_t ldc2, int32_t beta, int32_t k_per_split,
                           int64_t split_stride, void* hip_stream);

/* Deterministic split-K reduction of the weight gradient (the Accumulate edge of
 * Sec. 4.1: gradients are added into what the buffer holds):
 *   out[m][n] += sum over s = 0 .. splits-1, in that order, of part[s][m][n]
 * part: fp32 [splits][M][N] dense (the partials epilogue 4 writes with split_stride
 * M*N); out: fp32 [M][ldo], ldo >= N.  Four columns per thread when N and ldo are
 * multiples of 4 and both pointers 16-byte aligned, one column per thread otherwise;
 * both paths add in the same order. */
mpipe_status mpipe_op_splitk_reduce(const float* part, int32_t splits, int64_t M, int64_t N,
                                    float* out, int64_t ldo, void* hip_stream);

/* The number of K splits the encoder backward gives the weight-gradient product
 * dW[M][N] = sum over K tokens (host query, no device work): 1 means one unsplit
 * launch accumulating into d_weights; s > 1 means s fp32 partials then
 * mpipe_op_splitk_reduce.  -1 for negative sizes. */
int32_t mpipe_op_weight_grad_splits(int64_t M, int64_t N, int64_t K);

/* LayerNorm over rows of width n (n % 4 == 0, n <= 2048): X fp32 [rows][n];
 * g, b, Y in dtype; mean, rstd fp32 [rows] (nullable). */
mpipe_status mpipe_op_layernorm_fwd(int32_t dtype, const float* X, int64_t rows, int32_t n,
                                    const void* g, const void* b, float eps, void* Y, float* mean,
                                    float* rstd, void* hip_stream);

/* LayerNorm backward: dX = dres + LN'(dY) (fp32), dXt = the same in dtype
 * (nullable), grad_g / grad_b += column sums of dY*xhat and dY, colsum_dx +=
 * column sums of dX (the bias gradient of the product whose output gradient dX
 * is), all fp32 [n] and nullable.  scratch: at least
 * mpipe_op_scratch_bytes(rows, 1, n, 0) bytes. */
mpipe_status mpipe_op_layernorm_bwd(int32_t dtype, const float* dY, const float* X,
                                    const float* mean, const float* rstd, const void* g,
                                    int64_t rows, int32_t n, const float* dres, float* dX,
                                    void* dXt, float* grad_g, float* grad_b, float* colsum_dx,
                                    void* scratch, size_t scratch_bytes, void* hip_stream);

/* 2D rotary position, in place on the q and k blocks of qkv [rows][3*heads*d]
 * (inverse != 0 rotates back: the backward).  Positions come from grid_thw
 * (host) in the packed row order of mpipe.h. */
mpipe_status mpipe_op_rope(int32_t dtype, void* qkv, int64_t rows, int32_t heads, int32_t head_dim,
                           const int32_t* grid_thw, int32_t n_items, float theta, int32_t inverse,
                           void* scratch, size_t scratch_bytes, void* hip_stream);

/* Block-diagonal attention over segments cu_seqlens (host) of qkv [N][3*heads*d]
 * (columns q | k | v, head j at j*d).  o: [N][heads*d]; lse: fp32 [heads][N]
 * natural-log sum-exp of the scaled scores. */
mpipe_status mpipe_op_attention_fwd(int32_t dtype, const void* qkv, int64_t N, int32_t heads,
                                    int32_t head_dim, const int32_t* cu_seqlens, int32_t n_seg,
                                    void* o, float* lse, void* scratch, size_t scratch_bytes,
                                    void* hip_stream);

/* Attention backward: dqkv [N][3*heads*d] overwritten with dQ | dK | dV. */
mpipe_status mpipe_op_attention_bwd(int32_t dtype, const void* qkv, const void* o, const void* d_o,
                                    const float* lse, int64_t N, int32_t heads, int32_t head_dim,
                                    const int32_t* cu_seqlens, int32_t n_seg, void* dqkv,
                                    void* scratch, size_t scratch_bytes, void* hip_stream);

/* Scratch bytes the ops above need for rows N, heads, width n and n_seg segments. */
size_t mpipe_op_scratch_bytes(int64_t N, int32_t heads, int32_t n, int32_t n_seg);

#ifdef __cplusplus
}
#endif
#endif
