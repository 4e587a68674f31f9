/*
 * libmpipe -- the replicated-encoder step of the transpose schedule, on one
 * MI355X (gfx950).
 *
 * In the transpose schedule (Sec. 4.2), every pipeline rank holds a replica of
 * the modality encoder and, inside its warmup bubble, encodes the
 * micro-batches its ByMicrobatch owner assigns to it, each on its own; the
 * Replicated -> Sharded seam then gathers the encoder outputs into the first
 * LLM stage (Table 2: forward Gather, backward Scatter).  This library computes
 * one rank's share of that work for one micro-batch:
 *
 *   mpipe_encoder_fwd   Fwd(enc, m): the encoder over a packed variable-length
 *                       patch sequence (images and video clips), ending in the
 *                       2x2 patch merger.
 *   mpipe_encoder_bwd   Bwd(enc, m)^?: present only when the encoder is
 *                       trainable (Lemma 1); weight gradients Accumulate (+=)
 *                       into the caller's fp32 buffer (the Accumulate edge of
 *                       the instantiation in Sec. 4.1).  The encoder is the
 *                       trainable source, so nothing is sent upstream; the patch
 *                       gradient is computed only on request.
 *   mpipe_merge_scatter the local half of the seam Gather: merged rows into the
 *                       LLM input embedding buffer at placeholder rows.
 *   mpipe_merge_gather  the local half of the reverse Scatter^?: its adjoint.
 *
 * Encoder (the paper names "the ViT encoder from Qwen2-VL", Sec. 5, and gives
 * no internals; this is the pre-LayerNorm ViT reading):
 *   H = X Wpe^T + bpe; per layer: A = LN1(H); [Q|K|V] = A Wqkv^T + bqkv;
 *   Q, K <- 2D RoPE on patch (y, x); O = softmax(Q K^T / sqrt(d)) V within each
 *   attention segment; H += O Wo^T + bo; H += GELU(LN2(H) W1^T + b1) W2^T + b2;
 *   merger: Z = LN(H); each 2x2 window's four rows concatenated (4h);
 *   M = GELU(Z~ Wm1^T + bm1) Wm2^T + bm2.  GELU is the erf form, LN uses the
 *   biased variance, RoPE rotates the pair (j, j + d/2) of every head by
 *   y * theta^(-4j/d) for j < d/4 and by x * theta^(-4(j - d/4)/d) after.
 *
 * Data layout (all row-major):
 *   patches   [N][C*T*P*P] in the activation dtype.  Items follow each other;
 *             inside an item with grid (t, gh, gw) the rows run over
 *             (tau, hb, wb, dh, dw), patch position y = 2hb + dh, x = 2wb + dw,
 *             so every 2x2 merge window is four consecutive rows; a patch
 *             vector is flattened as (channel, frame, py, px).
 *   grid_thw  host int32 [n_items][3] = (t, gh, gw) in patches; gh, gw even
 *             and at most 32768 (a row's (y, x) is packed in 15 bits each).
 *   cu_seqlens host int32 [n_seg + 1], attention segments over the packed rows:
 *             0 = cu[0] < cu[1] < ... < cu[n_seg] = N; each segment lies inside
 *             one item and starts/ends on a temporal-slice boundary of it (one
 *             segment per item, or one per frame group).
 *   weights   flat buffer in the activation dtype, the tensors listed by
 *             mpipe_param_info back to back (Linear weights [out][in]).
 *   merged    [n_merged][llm_hidden], n_merged = sum t*(gh/2)*(gw/2); row j is
 *             window j in packed order (item, tau, hb, wb).
 *
 * Ownership and streams: the caller allocates every device buffer (weights,
 * gradients, patches, merged, embeddings, tape, workspace).  A handle holds
 * only the configuration, a small pinned host staging area for the per-call
 * metadata and (after the first backward) one internal stream; it is not
 * thread-safe.  All device work is ordered on the caller's stream (a
 * hipStream_t passed as void*): it starts after the work already enqueued there
 * and the stream does not pass the call's last kernel until all of it is done
 * (the backward forks its weight-gradient work onto the internal stream and
 * joins it back, see mpipe_encoder_set_side_stream).  No call synchronizes the
 * stream except to reuse the staging area of a still-running earlier call.
 * Host metadata pointers are read during the call only.
 *
 * Errors: every call returns an mpipe_status; all metadata checks run on the
 * host before any launch, so a non-OK status means nothing was enqueued.
 * mpipe_last_error() describes the last non-OK status of the calling thread.
 */
#ifndef MPIPE_H
#define MPIPE_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MPIPE_OK = 0,
  MPIPE_NOOP_FROZEN = 1,        /* backward on a frozen encoder: nothing written (Lemma 1) */
  MPIPE_ERR_INVALID_ARG = -1,
  MPIPE_ERR_BAD_METADATA = -2,  /* cu_seqlens / grid_thw inconsistent */
  MPIPE_ERR_WORKSPACE = -3,     /* workspace or tape smaller than mpipe_encoder_sizes says */
  MPIPE_ERR_NO_TAPE = -4,       /* trained forward or backward without a tape */
  MPIPE_ERR_UNSUPPORTED = -5,   /* configuration outside what the kernels support */
  MPIPE_ERR_HIP = -6            /* a HIP call failed (message in mpipe_last_error) */
} mpipe_status;

typedef enum { MPIPE_F32 = 0, MPIPE_BF16 = 1 } mpipe_dtype;

/* The `trainable` argument of the size, forward and backward calls.  Lemma 1 fixes
 * a region's backward work from which regions are trainable; here it is applied to
 * the encoder's own parts, ordered input-to-loss: the patch embedding and blocks,
 * then the merger (the projector that aligns the encoder's features with the LLM;
 * Sec. 2 notes that an alignment stage often trains only such layers while the
 * encoder stays frozen).
 *   MPIPE_FROZEN       nothing trainable: no tape, and the backward is a no-op.
 *   MPIPE_TRAINED      every part trainable: the backward produces the gradient of
 *                      every weight tensor (and of the patches on request).
 *   MPIPE_TRAIN_MERGER only the merger trainable.  The merger is then the trainable
 *                      source: it receives the gradient of the merged rows, reduces
 *                      its own weight gradients and sends nothing upstream, so the
 *                      blocks and the patch embedding run no backward and their
 *                      gradient entries are not written.  The tape holds the merger's
 *                      inputs only.
 * The forward result is bitwise the same in every mode (Corollary 1: the mode
 * decides which backward work exists, not what the forward computes).  Any other
 * value is rejected with MPIPE_ERR_INVALID_ARG. */
typedef enum { MPIPE_FROZEN = 0, MPIPE_TRAINED = 1, MPIPE_TRAIN_MERGER = 2 } mpipe_train_mode;

typedef struct {
  int32_t in_chans;        /* 3 */
  int32_t patch;           /* P = 14 */
  int32_t temporal_patch;  /* T: frames per patch (images repeat their frame T times) */
  int32_t hidden;          /* h; h % 64 == 0, h <= 2048 */
  int32_t layers;
  int32_t heads;           /* d = h / heads in {32, 64, 80} */
  int32_t mlp;             /* MLP width, % 8 == 0 */
  int32_t merge;           /* spatial merge size, must be 2 */
  int32_t llm_hidden;      /* merged output width H, % 8 == 0 */
  int32_t dtype;           /* mpipe_dtype of weights, patches, activations and merged */
  float ln_eps;            /* LayerNorm epsilon (1e-6) */
  float rope_theta;        /* rotary base (10000) */
} mpipe_encoder_cfg;

typedef struct mpipe_encoder mpipe_encoder;

mpipe_status mpipe_encoder_create(const mpipe_encoder_cfg* cfg, mpipe_encoder** out);
void mpipe_encoder_destroy(mpipe_encoder* enc);

/* Flat weight buffer: number of elements, number of tensors, and tensor i's
 * name (NUL-terminated, truncated to cap bytes), element offset and [rows][cols]
 * shape (cols = 1 for vectors). */
int64_t mpipe_param_count(const mpipe_encoder_cfg* cfg);
int32_t mpipe_param_tensors(const mpipe_encoder_cfg* cfg);
mpipe_status mpipe_param_info(const mpipe_encoder_cfg* cfg, int32_t i, char* name, int32_t cap,
                              int64_t* offset, int64_t* rows, int64_t* cols);

/* Buffer sizes for one micro-batch in a trainability mode (mpipe_train_mode):
 * device workspace, tape (0 when frozen, the merger's inputs only for
 * MPIPE_TRAIN_MERGER), merged rows and packed patch rows.  Validates the metadata. */
mpipe_status mpipe_encoder_sizes(const mpipe_encoder* enc, const int32_t* cu_seqlens,
                                 int32_t n_seg, const int32_t* grid_thw, int32_t n_items,
                                 int32_t trainable, size_t* workspace_bytes, size_t* tape_bytes,
                                 int64_t* n_merged, int64_t* n_patches);

/* The byte ranges of the workspace (which = 0) or the tape (which = 1) that the
 * forward and backward of this micro-batch and mode may write, in layout order
 * (host query, validates the metadata like mpipe_encoder_sizes).  Every range is
 * followed by at least 256 bytes that no call writes: a caller may fill the
 * buffers with a canary pattern and check, after a step, that everything outside
 * the ranges kept it.  Writes up to `cap` ranges into offsets / bytes (both
 * nullable when cap == 0) and the total count into *n_regions. */
mpipe_status mpipe_encoder_regions(const mpipe_encoder* enc, const int32_t* cu_seqlens,
                                   int32_t n_seg, const int32_t* grid_thw, int32_t n_items,
                                   int32_t trainable, int32_t which, int64_t* offsets,
                                   int64_t* bytes, int32_t cap, int32_t* n_regions);

/* Fwd(enc, m).  weights, patches: device, cfg dtype.  merged: device
 * [n_merged][llm_hidden], cfg dtype, overwritten.  trainable (mpipe_train_mode)
 * != MPIPE_FROZEN records the activations that mode's backward needs into `tape`
 * (tape_bytes from mpipe_encoder_sizes with the same mode); frozen passes
 * tape = NULL, 0.  The forward result is the same in every mode (Corollary 1).
 * workspace: device scratch, not kept.
 * n_items == 0 (a text-only micro-batch) is a valid no-op. */
mpipe_status mpipe_encoder_fwd(mpipe_encoder* enc, const void* weights, const void* patches,
                               const int32_t* cu_seqlens, int32_t n_seg, const int32_t* grid_thw,
                               int32_t n_items, int32_t trainable, void* merged, void* tape,
                               size_t tape_bytes, void* workspace, size_t workspace_bytes,
                               void* hip_stream);

/* Bwd(enc, m)^?.  trainable == MPIPE_FROZEN returns MPIPE_NOOP_FROZEN and writes
 * nothing.  tape: as recorded by the matching forward (same mode, weights, patches
 * and metadata).  d_merged: device [n_merged][llm_hidden], cfg dtype.  d_weights:
 * device fp32, flat layout of the weights, ACCUMULATED (+=): every tensor's entries
 * for MPIPE_TRAINED, the merger's only (its LayerNorm, fc1 and fc2) for
 * MPIPE_TRAIN_MERGER.  d_patches: nullable; if given (MPIPE_TRAINED only, else
 * MPIPE_ERR_INVALID_ARG), overwritten with dL/dpatches [N][C*T*P*P] in cfg dtype. */
mpipe_status mpipe_encoder_bwd(mpipe_encoder* enc, const void* weights, const void* patches,
                               const int32_t* cu_seqlens, int32_t n_seg, const int32_t* grid_thw,
                               int32_t n_items, int32_t trainable, const void* tape,
                               size_t tape_bytes, const void* d_merged, float* d_weights,
                               void* d_patches, void* workspace, size_t workspace_bytes,
                               void* hip_stream);

/* Backward stream use.  enable != 0 (the default): the weight- and bias-gradient
 * GEMMs and column sums, which nothing else in the backward reads, run on an
 * internal stream of the handle (created on the current device at the first
 * backward, default priority), forked from the caller's stream after each
 * gradient buffer is produced and joined back before mpipe_encoder_bwd returns;
 * the caller's stream waits for them only before it overwrites a buffer they
 * read.  enable == 0: everything runs on the caller's stream.  The results are
 * bitwise the same either way (same kernels, same operands, same order per
 * output).  Overlapping backward calls on one handle are not supported. */
mpipe_status mpipe_encoder_set_side_stream(mpipe_encoder* enc, int32_t enable);

/* Seam Gather, local half (Table 2, Replicated -> Sharded, forward):
 * embeds[idx[j]][:] = merged[j][:] for j < n_merged, a bit-exact row copy.
 * placeholder_idx: device int64 [n_merged], flat rows of embeds viewed as
 * [n_rows][row_elems]; must be unique and inside [0, n_rows) (rows outside are
 * skipped; mpipe_merge_check_indices verifies both). */
mpipe_status mpipe_merge_scatter(const void* merged, int64_t n_merged, int32_t row_elems,
                                 int32_t dtype, const int64_t* placeholder_idx, void* embeds,
                                 int64_t n_rows, void* hip_stream);

/* Reverse Scatter^?, local half: d_merged[j][:] = d_embeds[idx[j]][:]. */
mpipe_status mpipe_merge_gather(const void* d_embeds, int64_t n_rows, int32_t row_elems,
                                int32_t dtype, const int64_t* placeholder_idx, int64_t n_merged,
                                void* d_merged, void* hip_stream);

/* Device-side check of placeholder indices.  marks: device int32 scratch of
 * n_rows entries; status: device int32, set to 0, |1 if an index is out of
 * range, |2 if one repeats.  The caller reads status after the stream. */
mpipe_status mpipe_merge_check_indices(const int64_t* placeholder_idx, int64_t n_merged,
                                       int64_t n_rows, int32_t* marks, int32_t* status,
                                       void* hip_stream);

/* The same check for callers that cannot allocate device memory (work under
 * stream capture, serving loops, harnesses that forbid allocation): the per-row
 * counters live in a device array built into the library, so the caller passes
 * only the indices and the status word, and the call allocates nothing.
 * n_rows may be at most MPIPE_CHECK_NOALLOC_MAX_ROWS (4 MiB of int32 counters,
 * held by every GPU the library runs on until the process ends); a larger n_rows
 * returns MPIPE_ERR_WORKSPACE with nothing enqueued.  Every call on one GPU uses
 * that GPU's one array (cleared on the stream before use): calls that overlap on
 * one GPU, on different streams or threads, race and must be ordered by the
 * caller.  Result identical to mpipe_merge_check_indices. */
#define MPIPE_CHECK_NOALLOC_MAX_ROWS (1 << 20)
mpipe_status mpipe_merge_check_indices_noalloc(const int64_t* placeholder_idx, int64_t n_merged,
                                               int64_t n_rows, int32_t* status, void* hip_stream);

/* Message for the last non-OK status returned on this thread. */
const char* mpipe_last_error(void);

/* Kernel timing: when enabled, every kernel launch of the handle is bracketed
 * by HIP events on the stream it runs on.  mpipe_profile_read synchronizes the
 * caller's stream (the backward joins its side stream into it before returning),
 * then reports per kernel class the launch count, total milliseconds and
 * algorithmic FLOPs, and resets the counters.  Class names are the kernel kind
 * ("gemm_<layout>_<epilogue>", "attn_fwd", "attn_bwd_dq", "attn_bwd_dkdv",
 * "layernorm", "layernorm_bwd", "rope", "colsum", "splitk_reduce", "transpose",
 * "pad"); launches on the side stream carry the suffix "@side", and their times
 * include the sharing of compute units with the caller's stream.  names receives
 * up to cap NUL-terminated names of name_stride bytes each.  Returns the number of
 * classes written, or -1 on a null handle or a failed synchronization. */
mpipe_status mpipe_profile_enable(mpipe_encoder* enc, int32_t enable);
int32_t mpipe_profile_read(mpipe_encoder* enc, void* hip_stream, int32_t cap, char* names,
                           int32_t name_stride, int64_t* launches, double* ms, double* flops);

#ifdef __cplusplus
}
#endif
#endif
