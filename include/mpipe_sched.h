/*
 * libmpipe -- the ByMicrobatch owner of the replicated encoder and its cost.
 *
 * Under the transpose schedule (Sec. 4.2) every pipeline rank holds the encoder,
 * and the ByMicrobatch owner decides which rank runs Fwd(enc, m) for each
 * micro-batch m, inside that rank's warmup bubble.  The cost model (Sec. 4.3)
 * weighs a compute event by the roofline of its slab,
 *     cost(Fwd) = cost(Bwd) = max(W / F, D / B),
 * W its FLOPs at rate F, D its HBM traffic at bandwidth B, and prices what a rank
 * cannot hide as its spill,
 *     E_r = sum of cost(Fwd(enc, m)) over the micro-batches r owns,
 *     spill_r = max(0, E_r - w_r),
 * with w_r the rank's warmup bubble (its idle time before its first LLM
 * forward).  The step pays max_r spill_r; the owner that minimises it is a
 * min-max balancing of encode cost against warmup slack, and matching the
 * heaviest encodes to the longest slots is its greedy form.
 *
 * These calls are host-only (no device memory, no stream); they use the same
 * status codes and mpipe_last_error() as mpipe.h.
 */
#ifndef MPIPE_SCHED_H
#define MPIPE_SCHED_H
#include <stdint.h>

#include "mpipe.h"

#ifdef __cplusplus
extern "C" {
#endif

/* W and D of one micro-batch's encoder slabs, and their roofline costs.
 *   fwd_flops  W of Fwd(enc, m): the patch-embedding, block and merger GEMMs
 *              (2 M N K each) and the two attention products (4 h sum L^2 per
 *              layer over the attention segments); LayerNorm, GELU, RoPE and the
 *              softmax are not counted.
 *   fwd_bytes  D of Fwd(enc, m): every kernel's operands read once and results
 *              written once (activations in the cfg dtype, fp32 residual stream,
 *              weights once per use), plus the GELU' the forward stores for a
 *              trainable part.
 *   bwd_*      Bwd(enc, m)^? for the trainability mode (mpipe_train_mode): the
 *              input and weight gradients of every product of a trainable part
 *              (2 W of that part; the patch gradient is not requested), D twice
 *              the part's forward activation traffic plus its weights and their
 *              fp32 gradients (read and written once).  0 when frozen.
 *   *_seconds  max(W / flops_per_second, D / bytes_per_second). */
typedef struct {
  double fwd_flops, fwd_bytes, fwd_seconds;
  double bwd_flops, bwd_bytes, bwd_seconds;
} mpipe_slab_cost;

/* Cost of one micro-batch (the metadata of mpipe_encoder_sizes) on a device of
 * the given sustained rates (both > 0; e.g. the rates a measured step reaches).
 * Validates the metadata like mpipe_encoder_sizes. */
mpipe_status mpipe_encoder_cost(const mpipe_encoder* enc, const int32_t* cu_seqlens,
                                int32_t n_seg, const int32_t* grid_thw, int32_t n_items,
                                int32_t trainable, double flops_per_second,
                                double bytes_per_second, mpipe_slab_cost* out);

typedef enum {
  MPIPE_OWNER_GREEDY = 0,   /* heaviest encode first, each to the rank with the most
                               remaining slack w_r - E_r (ties to the lower rank;
                               equal costs keep index order); O(M log M + M P) */
  MPIPE_OWNER_EXACT = 1,    /* the minimum of max_r spill_r, by depth-first branch
                               and bound from the refined assignment */
  MPIPE_OWNER_REFINED = 2   /* greedy, then a descent by single moves and pairwise
                               swaps out of the most-spilling rank while the sorted
                               profile of E_r - w_r decreases; never worse than greedy */
} mpipe_owner_method;

/* Limits of MPIPE_OWNER_EXACT: more micro-batches or ranks, or a search that visits
 * more nodes, returns MPIPE_ERR_UNSUPPORTED (use the refined owner). */
#define MPIPE_OWNER_EXACT_MAX_MB 16
#define MPIPE_OWNER_EXACT_MAX_RANKS 64
#define MPIPE_OWNER_EXACT_NODE_CAP 50000000LL

/* ByMicrobatch owner.  cost: host [n_mb], encode cost of each micro-batch
 * (seconds, finite, >= 0); warmup: host [n_ranks], w_r (finite, >= 0).
 * owner: host [n_mb], written with the rank of each micro-batch.  spill:
 * nullable host [n_ranks], written with spill_r; max_spill: nullable, written
 * with max_r spill_r.  E_r is summed over the micro-batches in index order.
 * n_mb == 0 is valid (no spill). */
mpipe_status mpipe_owner_map(const double* cost, int32_t n_mb, const double* warmup,
                             int32_t n_ranks, int32_t method, int32_t* owner, double* spill,
                             double* max_spill);

#ifdef __cplusplus
}
#endif
#endif /* MPIPE_SCHED_H */
