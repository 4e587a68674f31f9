/*
 * libmpipe -- the schedule algebra: derive, its cost model and memory read-out.
 *
 * A model is a list of L layers.  A cut of k - 1 interior boundaries
 * 0 < c_1 < ... < c_{k-1} < L splits it into k contiguous regions, and a
 * schedule gives each region a skeleton (Sec. 4.1).  The skeleton fixes the
 * region's layout: transpose is Replicated (the whole region on every rank,
 * micro-batches spread over the ranks by a ByMicrobatch owner); 1f1b and gpipe
 * are Sharded (the region's layers split into P contiguous ByLayer slabs, one
 * per rank).  A (cut, schedule) pair is valid when the cut tiles the layers and
 * no two adjacent regions are Replicated (the normal form; such a pair would be
 * one region).
 *
 * derive maps a valid pair, each region's trainable bit, P ranks and M
 * micro-batches to
 *   placement   per region: layout, owner (ByLayer slabs or ByMicrobatch map),
 *               and whether any backward runs in it;
 *   collectives per seam (adjacent pair) the forward collective of its layout
 *               pair (Table 2) and the reverse one when it fires; per trainable
 *               region its weight reduction and group;
 *   order       the events, their typed edges and each rank's event sequence.
 * Backward work is gated by trainability alone (Lemma 1): region j runs a
 * backward iff some region i <= j is trainable; it sends its input gradient
 * back across seam (j-1, j) iff some region i < j is trainable; it reduces
 * weight gradients iff it is trainable.  None of the three reads the schedule
 * (Corollary 1), so two schedules of one cut have the same backward footprint.
 *
 * The order is built for every valid pair whose Sharded regions share one
 * skeleton, whose Replicated region (if any) is the first (the source region
 * that transpose moves into the warmup bubble), and, when several Sharded
 * regions are interleaved under 1f1b, whose M is a multiple of P.  Other valid
 * pairs (a Replicated sink, mixed Sharded skeletons) get placement and
 * collectives but no order (n_events = 0; mpipe_makespan returns
 * MPIPE_ERR_UNSUPPORTED).
 *
 * Each rank's sequence: a Replicated first region's forwards of the
 * micro-batches the rank owns (ascending m), then the Sharded regions' events
 * woven into one wavefront over stage = rank + region * P, then the Replicated
 * region's backwards of those micro-batches.  One Sharded region under 1f1b:
 * min(P - 1 - r, M) warmup forwards, then alternately one forward and one
 * backward, then the remaining backwards.  Several under 1f1b: the interleaved
 * 1F1B order (virtual micro-batches in groups of P per region chunk, warmup
 * 2 (P - 1 - r) + (S - 1) P, all warmup when M == P).  gpipe: every forward
 * (region by region, micro-batch by micro-batch), then every backward in
 * reverse region order.  The Loss of micro-batch m is the last forward stage's
 * event: rank P - 1 under a Sharded last region, the owner of m when the only
 * region is Replicated.  Coll, DpReduce and StepBarrier events are collective
 * and belong to no rank's sequence.
 *
 * Edges: Activation along the forward chain of a micro-batch (stage to stage,
 * through the forward seam collective, into its Loss) and from each Fwd to the
 * Bwd of the same stage and micro-batch (the stored activation); Turnaround
 * from Loss(m) to the first Bwd of m; Gradient along the backward chain and
 * into each reverse seam collective; Accumulate from every Bwd of a trainable
 * region to its DpReduce; Sequence from each DpReduce (or, with no backward
 * anywhere, each Loss) to the StepBarrier.  The graph with the rank sequences
 * is acyclic; mpipe_makespan checks it.
 *
 * All calls are host-only and use the status codes and mpipe_last_error() of
 * mpipe.h.
 */
#ifndef MPIPE_DERIVE_H
#define MPIPE_DERIVE_H
#include <stdint.h>

#include "mpipe.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { MPIPE_SK_1F1B = 0, MPIPE_SK_GPIPE = 1, MPIPE_SK_TRANSPOSE = 2 } mpipe_skeleton;
typedef enum { MPIPE_LAYOUT_SHARDED = 0, MPIPE_LAYOUT_REPLICATED = 1 } mpipe_layout;
typedef enum {
  MPIPE_COMM_NONE = -1,   /* a reverse collective that does not fire */
  MPIPE_COMM_GATHER = 0,
  MPIPE_COMM_SCATTER = 1,
  MPIPE_COMM_SEND = 2,
  MPIPE_COMM_RECVGRAD = 3
} mpipe_comm;
typedef enum { MPIPE_GROUP_REPLICA = 0, MPIPE_GROUP_DATA = 1 } mpipe_group;
typedef enum {
  MPIPE_EV_FWD = 0,
  MPIPE_EV_BWD = 1,
  MPIPE_EV_COLL = 2,
  MPIPE_EV_DPREDUCE = 3,
  MPIPE_EV_LOSS = 4,
  MPIPE_EV_STEP_BARRIER = 5
} mpipe_event_kind;
typedef enum {
  MPIPE_EDGE_ACTIVATION = 0,
  MPIPE_EDGE_GRADIENT = 1,
  MPIPE_EDGE_TURNAROUND = 2,
  MPIPE_EDGE_ACCUMULATE = 3,
  MPIPE_EDGE_SEQUENCE = 4
} mpipe_edge_kind;

/* One event.  Fields that do not apply to the kind are -1:
 *   Fwd/Bwd    region, rank, mb, stage = rank + region * P
 *   Coll       comm, seam (the seam between regions seam and seam + 1), mb
 *   DpReduce   region, group
 *   Loss       rank, mb
 * Regions, ranks, micro-batches and seams are numbered from 0. */
typedef struct {
  int32_t kind, region, rank, mb, stage, comm, seam, group;
} mpipe_event;

/* An edge from event `from` to event `to` (indices into the event list). */
typedef struct {
  int32_t from, to, kind;
} mpipe_edge;

/* Seam between regions `left` and `left + 1`: its forward collective and its
 * reverse one (MPIPE_COMM_NONE when Lemma 1 keeps it from firing). */
typedef struct {
  int32_t left, fwd, bwd;
} mpipe_seam;

typedef struct mpipe_derived mpipe_derived;

/* MPIPE_OK iff (cut, schedule) is valid; otherwise MPIPE_ERR_INVALID_ARG with
 * the reason.  cut: host [n_regions - 1] (may be null when n_regions == 1);
 * schedule: host [n_regions] of mpipe_skeleton. */
mpipe_status mpipe_schedule_valid(const int32_t* cut, int32_t n_regions, int32_t n_layers,
                                  const int32_t* schedule);

/* Derive placement, collectives and (when supported, see above) order.
 * trainable: host [n_regions], nonzero for a trainable region.  mb_owner:
 * nullable host [n_mb], the ByMicrobatch owner (rank of each micro-batch) of
 * the Replicated region; null means m mod P.  Each Sharded region needs at
 * least n_ranks layers.  On success *out is a handle the caller frees with
 * mpipe_derived_destroy; on error *out is null. */
mpipe_status mpipe_derive(const int32_t* cut, int32_t n_regions, int32_t n_layers,
                          const int32_t* schedule, const int32_t* trainable, int32_t n_ranks,
                          int32_t n_mb, const int32_t* mb_owner, mpipe_derived** out);

void mpipe_derived_destroy(mpipe_derived* d);

/* Sizes of the lists (each pointer nullable).  has_order is 1 when the order
 * was built; then n_events and n_edges are its sizes, else both are 0. */
mpipe_status mpipe_derived_shape(const mpipe_derived* d, int32_t* has_order, int32_t* n_events,
                                 int32_t* n_edges, int32_t* n_seams, int32_t* n_reduces);

/* Placement of one region.  layout: mpipe_layout; runs_bwd: 1 iff the region
 * runs a backward (Lemma 1 (ii)); slab_lo/slab_hi: nullable host [n_ranks],
 * the ByLayer slab [lo, hi) of each rank (global layer indices; -1 for a
 * Replicated region, whose owner is the ByMicrobatch map of mpipe_derived_owner). */
mpipe_status mpipe_derived_placement(const mpipe_derived* d, int32_t region, int32_t* layout,
                                     int32_t* runs_bwd, int32_t* slab_lo, int32_t* slab_hi);

/* The ByMicrobatch owner map: host [n_mb]. */
mpipe_status mpipe_derived_owner(const mpipe_derived* d, int32_t* owner);

/* Copy out the lists (each pointer nullable; sizes from mpipe_derived_shape):
 * events [n_events], edges [n_edges], seams [n_seams], reduce_region and
 * reduce_group [n_reduces] (ascending region). */
mpipe_status mpipe_derived_lists(const mpipe_derived* d, mpipe_event* events, mpipe_edge* edges,
                                 mpipe_seam* seams, int32_t* reduce_region, int32_t* reduce_group);

/* nodes(rank): the rank's event sequence.  Returns its length (copying at most
 * cap indices into out when out is not null), or -1 for a bad handle or rank. */
int32_t mpipe_derived_nodes(const mpipe_derived* d, int32_t rank, int32_t* out, int32_t cap);

/* Event costs of the cost model (Sec. 4.3), written to cost [n_events]:
 *   Fwd(j, r, m)   fwd_cost[j * n_mb + m] scaled by the slab's share of region
 *                  j's layers (Sharded), or whole (Replicated, on owner(m));
 *   Bwd(j, r, m)   the same with bwd_cost;
 *   Coll(c, s, m)  alpha + beta * seam_bytes[s * n_mb + m] (the activation, or
 *                  its gradient, crossing seam s);
 *   DpReduce(j)    alpha + beta * reduce_bytes[j] (region j's weight gradients);
 *   Loss(m)        loss_cost;  StepBarrier 0.
 * fwd_cost/bwd_cost: host [n_regions * n_mb], seconds of the whole region's
 * forward/backward of micro-batch m (e.g. max(W/F, D/B) of mpipe_encoder_cost);
 * seam_bytes: host [(n_regions - 1) * n_mb] (nullable when n_regions == 1);
 * reduce_bytes: host [n_regions].  Every value must be finite and >= 0. */
mpipe_status mpipe_event_costs(const mpipe_derived* d, const double* fwd_cost,
                               const double* bwd_cost, const double* seam_bytes,
                               const double* reduce_bytes, double alpha, double beta,
                               double loss_cost, double* cost);

/* Makespan and bubbles (Sec. 4.3): with cost [n_events] (finite, >= 0) as event
 * durations, every event starts when its predecessors (edges, and the previous
 * event of its rank's sequence) have finished; the makespan T is the longest
 * path, bubble[r] = T - (sum of the costs in nodes(r)).  makespan, bubble
 * (host [n_ranks]), start and finish (host [n_events]) are nullable.
 * MPIPE_ERR_UNSUPPORTED without an order; MPIPE_ERR_INVALID_ARG on a cycle. */
mpipe_status mpipe_makespan(const mpipe_derived* d, const double* cost, double* makespan,
                            double* bubble, double* start, double* finish);

/* Memory as a read-out of placement and order: act_bytes [n_events] gives the
 * bytes each Fwd keeps (ignored for other kinds).  On each rank, in nodes(r)
 * order, a Fwd's bytes become live when it runs and stay live until the Bwd of
 * the same stage and micro-batch has run; in a region that runs no backward
 * they are live only while the Fwd runs.  peak: host [n_ranks], the largest
 * sum of live bytes on each rank.  MPIPE_ERR_UNSUPPORTED without an order. */
mpipe_status mpipe_memory_peak(const mpipe_derived* d, const double* act_bytes, double* peak);

#ifdef __cplusplus
}
#endif
#endif /* MPIPE_DERIVE_H */
