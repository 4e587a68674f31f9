/*
 * Plain CPU oracle for the replicated-encoder step -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may load
 * this library.  It shares no code, header, table or helper with the HIP
 * library: it is written from the definitions alone, in plain loops, so that a
 * reader can check it against the paper and the encoder description by eye.
 *
 * What it computes (the method only relocates this computation -- Sec. 4.2 --
 * and leaves the loss unchanged, Sec. 5 Analysis):
 *   Fwd(enc, m): a pre-LayerNorm ViT over a packed variable-length patch
 *     sequence with block-diagonal (per-item) attention and 2D rotary position
 *     on (y, x), followed by a 2x2 patch merger (LN -> concat -> Linear+GELU ->
 *     Linear).
 *   Bwd(enc, m)^?: exact reverse-mode gradients, present only when the encoder
 *     is trainable (Lemma 1); weight gradients accumulate (+=), the Accumulate
 *     edge of the instantiation in Sec. 4.1.
 *   Coll(Gather, (enc, llm), m), local half: row scatter of the merged
 *     embeddings into the LLM input buffer at placeholder rows, and its adjoint
 *     row gather for the reverse Scatter^? (Table 2).
 *
 * Every floating-point routine exists in double (suffix _f64) and float (_f32).
 * Return codes: 0 ok, 1 frozen no-op (backward requested on a frozen encoder),
 * negative on invalid metadata or arguments.
 */
#ifndef MPIPE_REF_H
#define MPIPE_REF_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t in_chans, patch, temporal_patch, hidden, layers, heads, mlp, merge, llm_hidden;
  double ln_eps, rope_theta;
} ref_cfg;

int64_t ref_param_count(const ref_cfg* c);
/* name written into `name` (cap bytes); rows/cols of the tensor (cols = 1 for vectors). */
int ref_param_info(const ref_cfg* c, int32_t i, char* name, int32_t cap,
                   int64_t* offset, int64_t* rows, int64_t* cols);
int32_t ref_param_tensors(const ref_cfg* c);

/* Patch position (y, x) of every packed row, from the window-major row order. */
int ref_positions(const int32_t* grid_thw, int32_t n_items, int32_t* pos_y, int32_t* pos_x);

/* Whole encoder.  merged: [n_merged][llm_hidden].  trainable: 0 nothing trainable,
 * 1 every part trainable, 2 only the merger trainable.  If d_merged is non-NULL the
 * backward runs (trainable == 0 returns 1 and writes nothing to d_w / d_patches):
 * d_w += dL/dw for the trainable parts, and d_patches (if non-NULL; trainable == 1
 * only) = dL/dpatches.  With only the merger trainable, Lemma 1 read over the
 * encoder's parts (patch embedding and blocks, then merger) makes the merger the
 * trainable source: its backward stops at its own LayerNorm, nothing before it runs
 * a backward, and their d_w entries are not touched. */
int ref_encoder_f64(const ref_cfg* c, const double* w, const double* patches,
                    const int32_t* cu_seqlens, int32_t n_seg,
                    const int32_t* grid_thw, int32_t n_items, int32_t trainable,
                    double* merged, const double* d_merged, double* d_w, double* d_patches);
int ref_encoder_f32(const ref_cfg* c, const float* w, const float* patches,
                    const int32_t* cu_seqlens, int32_t n_seg,
                    const int32_t* grid_thw, int32_t n_items, int32_t trainable,
                    float* merged, const float* d_merged, float* d_w, float* d_patches);

/* Building blocks (used by the pins). Row-major; ld* are row strides in elements. */
void ref_linear_f64(const double* X, const double* W, const double* b,
                    int64_t M, int64_t K, int64_t N, double* Y);
void ref_linear_bwd_f64(const double* dY, const double* X, const double* W,
                        int64_t M, int64_t K, int64_t N, double* dX, double* dW, double* db);
void ref_layernorm_f64(const double* X, const double* g, const double* b, int64_t M, int64_t n,
                       double eps, double* Y, double* mean, double* rstd);
void ref_layernorm_bwd_f64(const double* dY, const double* X, const double* g,
                           const double* mean, const double* rstd, int64_t M, int64_t n,
                           double* dX, double* dg, double* db);
void ref_gelu_f64(const double* u, int64_t n, double* y);
void ref_gelu_grad_f64(const double* u, int64_t n, double* dydu);
void ref_rope2d_f64(double* x, int64_t N, int32_t heads, int32_t d, int64_t ld,
                    const int32_t* pos_y, const int32_t* pos_x, double theta, int32_t inverse);
void ref_attention_f64(const double* q, const double* k, const double* v, int64_t ld,
                       const int32_t* cu_seqlens, int32_t n_seg, int32_t heads, int32_t d,
                       double* o, int64_t ldo, double* lse);
void ref_attention_bwd_f64(const double* q, const double* k, const double* v, int64_t ld,
                           const double* o, const double* d_o, int64_t ldo, const double* lse,
                           const int32_t* cu_seqlens, int32_t n_seg, int32_t heads, int32_t d,
                           double* dq, double* dk, double* dv, int64_t ldd);

/* Row scatter / gather of raw bytes.  Returns -1 (and writes nothing) when an
 * index is out of range or repeated. */
int ref_merge_scatter(const void* merged, int64_t n_merged, int64_t row_bytes,
                      const int64_t* idx, void* emb, int64_t n_rows);
int ref_merge_gather(const void* d_emb, int64_t n_rows, int64_t row_bytes,
                     const int64_t* idx, int64_t n_merged, void* d_merged);

/* Threads the oracle's parallel loops use (OpenMP). */
int32_t ref_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
