// The schedule algebra's derive, its event costs, makespan and memory read-out
// (Sec. 4.1 and 4.3), host code.  What each call computes is stated in mpipe_derive.h.
#include <algorithm>
#include <cmath>
#include <string>
#include <vector>

#include "../../include/mpipe_derive.h"

namespace mpipe {
mpipe_status set_error(mpipe_status s, const std::string& m);
}

struct mpipe_derived {
  int P = 0, M = 0, k = 0, L = 0;
  std::vector<int> layout, skel, trainable, runs_bwd, lo, hi;
  std::vector<int> slab_lo, slab_hi;   // [region * P + rank]; -1 for Replicated regions
  std::vector<int> owner;              // [mb], the ByMicrobatch map
  std::vector<mpipe_seam> seams;
  std::vector<int> red_region, red_group;
  bool has_order = false;
  std::string no_order;                // why the order was not built
  std::vector<mpipe_event> events;
  std::vector<mpipe_edge> edges;
  std::vector<std::vector<int>> nodes;
  std::vector<int> partner;            // [event]: Fwd -> its Bwd, Bwd -> its Fwd, else -1
};

namespace {

using mpipe::set_error;

bool check_valid(const int32_t* cut, int k, int L, const int32_t* sched, std::string& why) {
  if (k < 1 || L < 1) return why = "need at least one region and one layer", false;
  if (!sched || (k > 1 && !cut)) return why = "null cut or schedule", false;
  int prev = 0;
  for (int j = 0; j + 1 < k; ++j) {   // the cut tiles the layers: 0 < c_1 < ... < c_{k-1} < L
    if (cut[j] <= prev || cut[j] >= L)
      return why = "cut boundaries must increase strictly inside (0, L)", false;
    prev = cut[j];
  }
  for (int j = 0; j < k; ++j)
    if (sched[j] != MPIPE_SK_1F1B && sched[j] != MPIPE_SK_GPIPE && sched[j] != MPIPE_SK_TRANSPOSE)
      return why = "unknown skeleton", false;
  for (int j = 0; j + 1 < k; ++j)   // normal form: no two adjacent Replicated regions
    if (sched[j] == MPIPE_SK_TRANSPOSE && sched[j + 1] == MPIPE_SK_TRANSPOSE)
      return why = "adjacent transposed regions are not in normal form (they are one region)", false;
  return true;
}

// Table 2: the forward collective of a seam from its two layouts, and the mirror row
int seam_fwd(int a, int b) {
  if (a == MPIPE_LAYOUT_REPLICATED) return MPIPE_COMM_GATHER;
  if (b == MPIPE_LAYOUT_REPLICATED) return MPIPE_COMM_SCATTER;
  return MPIPE_COMM_SEND;
}
int seam_bwd(int a, int b) {
  if (a == MPIPE_LAYOUT_REPLICATED) return MPIPE_COMM_SCATTER;
  if (b == MPIPE_LAYOUT_REPLICATED) return MPIPE_COMM_GATHER;
  return MPIPE_COMM_RECVGRAD;
}

// Events and edges of the order graph, then each rank's sequence.
class OrderBuilder {
 public:
  explicit OrderBuilder(mpipe_derived& d)
      : d_(d),
        fwd_((size_t)d.k * d.P * d.M, -1),
        bwd_((size_t)d.k * d.P * d.M, -1),
        loss_(d.M, -1),
        dpr_(d.k, -1) {}

  void build() {
    const int k = d_.k, M = d_.M;
    const bool any_bwd = d_.runs_bwd[k - 1];
    for (int m = 0; m < M; ++m) {
      int prev = -1;   // the event the next one of m's forward chain depends on
      for (int j = 0; j < k; ++j) {
        for (int r : stages(j, m)) {
          const int e = add_compute(MPIPE_EV_FWD, j, r, m);
          F(j, r, m) = e;
          edge(prev, e, MPIPE_EDGE_ACTIVATION);
          prev = e;
        }
        if (j + 1 < k) {
          const int c = add(MPIPE_EV_COLL, -1, -1, m, d_.seams[j].fwd, j, -1);
          edge(prev, c, MPIPE_EDGE_ACTIVATION);
          prev = c;
        }
      }
      loss_[m] = add(MPIPE_EV_LOSS, -1, loss_rank(m), m, -1, -1, -1);
      edge(prev, loss_[m], MPIPE_EDGE_ACTIVATION);
      if (!any_bwd) continue;
      prev = loss_[m];
      int kind = MPIPE_EDGE_TURNAROUND;
      for (int j = k - 1; j >= 0 && d_.runs_bwd[j]; --j) {
        const std::vector<int> st = stages(j, m);
        for (int i = (int)st.size() - 1; i >= 0; --i) {
          const int r = st[i];
          const int e = add_compute(MPIPE_EV_BWD, j, r, m);
          B(j, r, m) = e;
          d_.partner[e] = F(j, r, m), d_.partner[F(j, r, m)] = e;
          edge(prev, e, kind);
          edge(F(j, r, m), e, MPIPE_EDGE_ACTIVATION);   // the activation the forward stored
          prev = e;
          kind = MPIPE_EDGE_GRADIENT;
        }
        if (j > 0 && d_.runs_bwd[j - 1]) {   // Lemma 1 (i): region j sends its input gradient
          const int c = add(MPIPE_EV_COLL, -1, -1, m, d_.seams[j - 1].bwd, j - 1, -1);
          edge(prev, c, MPIPE_EDGE_GRADIENT);
          prev = c;
        }
      }
    }
    for (size_t i = 0; i < d_.red_region.size(); ++i)
      dpr_[d_.red_region[i]] =
          add(MPIPE_EV_DPREDUCE, d_.red_region[i], -1, -1, -1, -1, d_.red_group[i]);
    const int barrier = add(MPIPE_EV_STEP_BARRIER, -1, -1, -1, -1, -1, -1);
    for (int j = 0; j < k; ++j) {
      if (dpr_[j] < 0) continue;
      for (int m = 0; m < M; ++m)
        for (int r : stages(j, m)) edge(B(j, r, m), dpr_[j], MPIPE_EDGE_ACCUMULATE);
      edge(dpr_[j], barrier, MPIPE_EDGE_SEQUENCE);
    }
    if (!any_bwd)   // nothing trainable: the step ends with its losses
      for (int m = 0; m < M; ++m) edge(loss_[m], barrier, MPIPE_EDGE_SEQUENCE);
    d_.nodes.assign(d_.P, {});
    for (int r = 0; r < d_.P; ++r) sequence(r, any_bwd);
  }

 private:
  mpipe_derived& d_;
  std::vector<int> fwd_, bwd_, loss_, dpr_;

  int& F(int j, int r, int m) { return fwd_[((size_t)j * d_.P + r) * d_.M + m]; }
  int& B(int j, int r, int m) { return bwd_[((size_t)j * d_.P + r) * d_.M + m]; }

  int add(int kind, int region, int rank, int mb, int comm, int seam, int group) {
    const int stage = (kind == MPIPE_EV_FWD || kind == MPIPE_EV_BWD) ? rank + region * d_.P : -1;
    d_.events.push_back({kind, region, rank, mb, stage, comm, seam, group});
    d_.partner.push_back(-1);
    return (int)d_.events.size() - 1;
  }
  int add_compute(int kind, int j, int r, int m) { return add(kind, j, r, m, -1, -1, -1); }
  void edge(int a, int b, int kind) {
    if (a >= 0 && b >= 0) d_.edges.push_back({a, b, kind});
  }
  // the ranks that region j's forward of micro-batch m passes, in order
  std::vector<int> stages(int j, int m) const {
    if (d_.layout[j] == MPIPE_LAYOUT_REPLICATED) return {d_.owner[m]};
    std::vector<int> v(d_.P);
    for (int r = 0; r < d_.P; ++r) v[r] = r;
    return v;
  }
  int loss_rank(int m) const {
    return d_.layout[d_.k - 1] == MPIPE_LAYOUT_SHARDED ? d_.P - 1 : d_.owner[m];
  }

  void sequence(int r, bool any_bwd) {
    std::vector<int>& seq = d_.nodes[r];
    const int M = d_.M, P = d_.P;
    std::vector<int> sh;   // the Sharded regions, in order
    for (int j = 0; j < d_.k; ++j)
      if (d_.layout[j] == MPIPE_LAYOUT_SHARDED) sh.push_back(j);
    const int S = (int)sh.size();
    const bool rep_source = d_.layout[0] == MPIPE_LAYOUT_REPLICATED;
    auto pushF = [&](int j, int m) {
      seq.push_back(F(j, r, m));
      if (j == d_.k - 1 && loss_rank(m) == r) seq.push_back(loss_[m]);
    };
    auto pushB = [&](int j, int m) {
      if (B(j, r, m) >= 0) seq.push_back(B(j, r, m));
    };
    if (rep_source)   // transpose: the owned forwards fill the warmup bubble
      for (int m = 0; m < M; ++m)
        if (d_.owner[m] == r) pushF(0, m);
    if (S == 0 || !any_bwd) {
      for (int m = 0; m < M; ++m)
        for (int s = 0; s < S; ++s) pushF(sh[s], m);
    } else if (d_.skel[sh[0]] == MPIPE_SK_GPIPE) {
      for (int s = 0; s < S; ++s)
        for (int m = 0; m < M; ++m) pushF(sh[s], m);
      for (int s = S - 1; s >= 0; --s)
        for (int m = 0; m < M; ++m) pushB(sh[s], m);
    } else if (S == 1) {   // 1F1B
      const int nw = std::min(P - 1 - r, M);
      for (int m = 0; m < nw; ++m) pushF(sh[0], m);
      for (int i = 0; i < M - nw; ++i) {
        pushF(sh[0], nw + i);
        pushB(sh[0], i);
      }
      for (int i = M - nw; i < M; ++i) pushB(sh[0], i);
    } else {   // interleaved 1F1B over S chunks per rank (M a multiple of P)
      const int total = M * S, grp = P * S;
      auto chunk_f = [&](int q) { return (q % grp) / P; };
      auto chunk_b = [&](int q) { return S - 1 - (q % grp) / P; };
      auto mb_of = [&](int q) { return (q / grp) * P + q % P; };
      const int nw = M == P ? total : std::min(2 * (P - 1 - r) + (S - 1) * P, total);
      for (int q = 0; q < nw; ++q) pushF(sh[chunk_f(q)], mb_of(q));
      for (int q = 0; q < total - nw; ++q) {
        pushF(sh[chunk_f(nw + q)], mb_of(nw + q));
        pushB(sh[chunk_b(q)], mb_of(q));
      }
      for (int q = total - nw; q < total; ++q) pushB(sh[chunk_b(q)], mb_of(q));
    }
    if (rep_source && any_bwd)   // transpose: the owned backwards run in the cooldown
      for (int m = 0; m < M; ++m)
        if (d_.owner[m] == r) pushB(0, m);
  }
};

// Whether derive builds an order for this placement, and why not.
bool order_supported(const mpipe_derived& d, std::string& why) {
  int kind = -1, S = 0;
  for (int j = 0; j < d.k; ++j) {
    if (d.layout[j] == MPIPE_LAYOUT_REPLICATED) {
      if (j != 0)
        return why = "a transposed region after the first is a pipeline sink; the order places "
                     "Replicated work only in the warmup and cooldown of a source region",
               false;
      continue;
    }
    if (kind >= 0 && d.skel[j] != kind)
      return why = "the Sharded regions must share one skeleton to be woven", false;
    kind = d.skel[j];
    ++S;
  }
  if (S > 1 && kind == MPIPE_SK_1F1B && d.M % d.P != 0)
    return why = "the interleaved 1F1B order needs M to be a multiple of P", false;
  return true;
}

bool all_finite_nonneg(const double* v, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!std::isfinite(v[i]) || v[i] < 0) return false;
  return true;
}

}  // namespace

extern "C" {

mpipe_status mpipe_schedule_valid(const int32_t* cut, int32_t n_regions, int32_t n_layers,
                                  const int32_t* schedule) {
  std::string why;
  if (!check_valid(cut, n_regions, n_layers, schedule, why))
    return set_error(MPIPE_ERR_INVALID_ARG, why);
  return MPIPE_OK;
}

mpipe_status mpipe_derive(const int32_t* cut, int32_t n_regions, int32_t n_layers,
                          const int32_t* schedule, const int32_t* trainable, int32_t n_ranks,
                          int32_t n_mb, const int32_t* mb_owner, mpipe_derived** out) {
  if (!out) return set_error(MPIPE_ERR_INVALID_ARG, "null output handle");
  *out = nullptr;
  std::string why;
  if (!check_valid(cut, n_regions, n_layers, schedule, why))
    return set_error(MPIPE_ERR_INVALID_ARG, why);
  if (!trainable) return set_error(MPIPE_ERR_INVALID_ARG, "null trainable bits");
  if (n_ranks < 1 || n_mb < 1) return set_error(MPIPE_ERR_INVALID_ARG, "need n_ranks >= 1, n_mb >= 1");
  const int k = n_regions, P = n_ranks, M = n_mb;
  for (int m = 0; mb_owner && m < M; ++m)
    if (mb_owner[m] < 0 || mb_owner[m] >= P)
      return set_error(MPIPE_ERR_INVALID_ARG, "owner rank out of range");
  for (int j = 0; j < k; ++j) {
    const int lo = j == 0 ? 0 : cut[j - 1], hi = j + 1 == k ? n_layers : cut[j];
    if (schedule[j] != MPIPE_SK_TRANSPOSE && hi - lo < P)
      return set_error(MPIPE_ERR_INVALID_ARG, "a Sharded region needs at least one layer per rank");
  }
  auto d = new mpipe_derived();
  d->P = P, d->M = M, d->k = k, d->L = n_layers;
  d->skel.assign(schedule, schedule + k);
  d->layout.resize(k), d->trainable.resize(k), d->runs_bwd.resize(k), d->lo.resize(k), d->hi.resize(k);
  d->slab_lo.assign((size_t)k * P, -1), d->slab_hi.assign((size_t)k * P, -1);
  for (int j = 0; j < k; ++j) {
    d->lo[j] = j == 0 ? 0 : cut[j - 1];
    d->hi[j] = j + 1 == k ? n_layers : cut[j];
    d->trainable[j] = trainable[j] != 0;
    d->layout[j] = schedule[j] == MPIPE_SK_TRANSPOSE ? MPIPE_LAYOUT_REPLICATED : MPIPE_LAYOUT_SHARDED;
    // Lemma 1 (ii): a region runs a backward iff it or a region before it is trainable
    d->runs_bwd[j] = d->trainable[j] || (j > 0 && d->runs_bwd[j - 1]);
    if (d->layout[j] == MPIPE_LAYOUT_SHARDED) {   // ByLayer: P contiguous slabs
      const int n = d->hi[j] - d->lo[j];
      for (int r = 0; r < P; ++r) {
        d->slab_lo[(size_t)j * P + r] = d->lo[j] + (int)((int64_t)r * n / P);
        d->slab_hi[(size_t)j * P + r] = d->lo[j] + (int)((int64_t)(r + 1) * n / P);
      }
    }
  }
  d->owner.resize(M);
  for (int m = 0; m < M; ++m) d->owner[m] = mb_owner ? mb_owner[m] : m % P;
  // A seam's reverse collective carries the later region's input gradient, so it fires
  // iff that region sends (Lemma 1 (i)), i.e. iff the earlier region runs a backward.
  for (int j = 0; j + 1 < k; ++j)
    d->seams.push_back({j, seam_fwd(d->layout[j], d->layout[j + 1]),
                        d->runs_bwd[j] ? seam_bwd(d->layout[j], d->layout[j + 1]) : MPIPE_COMM_NONE});
  for (int j = 0; j < k; ++j)   // Lemma 1 (iii)
    if (d->trainable[j]) {
      d->red_region.push_back(j);
      d->red_group.push_back(d->layout[j] == MPIPE_LAYOUT_REPLICATED ? MPIPE_GROUP_REPLICA
                                                                     : MPIPE_GROUP_DATA);
    }
  d->has_order = order_supported(*d, d->no_order);
  if (d->has_order) OrderBuilder(*d).build();
  *out = d;
  return MPIPE_OK;
}

void mpipe_derived_destroy(mpipe_derived* d) { delete d; }

mpipe_status mpipe_derived_shape(const mpipe_derived* d, int32_t* has_order, int32_t* n_events,
                                 int32_t* n_edges, int32_t* n_seams, int32_t* n_reduces) {
  if (!d) return set_error(MPIPE_ERR_INVALID_ARG, "null derivation");
  if (has_order) *has_order = d->has_order;
  if (n_events) *n_events = (int32_t)d->events.size();
  if (n_edges) *n_edges = (int32_t)d->edges.size();
  if (n_seams) *n_seams = (int32_t)d->seams.size();
  if (n_reduces) *n_reduces = (int32_t)d->red_region.size();
  return MPIPE_OK;
}

mpipe_status mpipe_derived_placement(const mpipe_derived* d, int32_t region, int32_t* layout,
                                     int32_t* runs_bwd, int32_t* slab_lo, int32_t* slab_hi) {
  if (!d) return set_error(MPIPE_ERR_INVALID_ARG, "null derivation");
  if (region < 0 || region >= d->k) return set_error(MPIPE_ERR_INVALID_ARG, "region out of range");
  if (layout) *layout = d->layout[region];
  if (runs_bwd) *runs_bwd = d->runs_bwd[region];
  for (int r = 0; r < d->P; ++r) {
    if (slab_lo) slab_lo[r] = d->slab_lo[(size_t)region * d->P + r];
    if (slab_hi) slab_hi[r] = d->slab_hi[(size_t)region * d->P + r];
  }
  return MPIPE_OK;
}

mpipe_status mpipe_derived_owner(const mpipe_derived* d, int32_t* owner) {
  if (!d || !owner) return set_error(MPIPE_ERR_INVALID_ARG, "null derivation or output");
  std::copy(d->owner.begin(), d->owner.end(), owner);
  return MPIPE_OK;
}

mpipe_status mpipe_derived_lists(const mpipe_derived* d, mpipe_event* events, mpipe_edge* edges,
                                 mpipe_seam* seams, int32_t* reduce_region, int32_t* reduce_group) {
  if (!d) return set_error(MPIPE_ERR_INVALID_ARG, "null derivation");
  if (events) std::copy(d->events.begin(), d->events.end(), events);
  if (edges) std::copy(d->edges.begin(), d->edges.end(), edges);
  if (seams) std::copy(d->seams.begin(), d->seams.end(), seams);
  if (reduce_region) std::copy(d->red_region.begin(), d->red_region.end(), reduce_region);
  if (reduce_group) std::copy(d->red_group.begin(), d->red_group.end(), reduce_group);
  return MPIPE_OK;
}

int32_t mpipe_derived_nodes(const mpipe_derived* d, int32_t rank, int32_t* out, int32_t cap) {
  if (!d || rank < 0 || rank >= d->P || (out && cap < 0)) {
    set_error(MPIPE_ERR_INVALID_ARG, "null derivation, rank out of range or negative capacity");
    return -1;
  }
  if (!d->has_order) return 0;
  const std::vector<int>& v = d->nodes[rank];
  if (out)
    for (int i = 0; i < (int)v.size() && i < cap; ++i) out[i] = v[i];
  return (int32_t)v.size();
}

mpipe_status mpipe_event_costs(const mpipe_derived* d, const double* fwd_cost,
                               const double* bwd_cost, const double* seam_bytes,
                               const double* reduce_bytes, double alpha, double beta,
                               double loss_cost, double* cost) {
  if (!d) return set_error(MPIPE_ERR_INVALID_ARG, "null derivation");
  if (!d->has_order) return set_error(MPIPE_ERR_UNSUPPORTED, d->no_order);
  const size_t km = (size_t)d->k * d->M, sm = (size_t)(d->k - 1) * d->M;
  if (!fwd_cost || !bwd_cost || !reduce_bytes || !cost || (sm && !seam_bytes))
    return set_error(MPIPE_ERR_INVALID_ARG, "null cost input or output");
  if (!all_finite_nonneg(fwd_cost, km) || !all_finite_nonneg(bwd_cost, km) ||
      !all_finite_nonneg(reduce_bytes, d->k) || (sm && !all_finite_nonneg(seam_bytes, sm)) ||
      !all_finite_nonneg(&alpha, 1) || !all_finite_nonneg(&beta, 1) ||
      !all_finite_nonneg(&loss_cost, 1))
    return set_error(MPIPE_ERR_INVALID_ARG, "costs, bytes, alpha and beta must be finite and >= 0");
  for (size_t i = 0; i < d->events.size(); ++i) {
    const mpipe_event& e = d->events[i];
    double c = 0;
    switch (e.kind) {
      case MPIPE_EV_FWD:
      case MPIPE_EV_BWD: {
        c = (e.kind == MPIPE_EV_FWD ? fwd_cost : bwd_cost)[(size_t)e.region * d->M + e.mb];
        if (d->layout[e.region] == MPIPE_LAYOUT_SHARDED) {
          const size_t s = (size_t)e.region * d->P + e.rank;
          c *= double(d->slab_hi[s] - d->slab_lo[s]) / double(d->hi[e.region] - d->lo[e.region]);
        }
        break;
      }
      case MPIPE_EV_COLL: c = alpha + beta * seam_bytes[(size_t)e.seam * d->M + e.mb]; break;
      case MPIPE_EV_DPREDUCE: c = alpha + beta * reduce_bytes[e.region]; break;
      case MPIPE_EV_LOSS: c = loss_cost; break;
      default: c = 0;
    }
    cost[i] = c;
  }
  return MPIPE_OK;
}

mpipe_status mpipe_makespan(const mpipe_derived* d, const double* cost, double* makespan,
                            double* bubble, double* start, double* finish) {
  if (!d) return set_error(MPIPE_ERR_INVALID_ARG, "null derivation");
  if (!d->has_order) return set_error(MPIPE_ERR_UNSUPPORTED, d->no_order);
  const int n = (int)d->events.size();
  if (!cost) return set_error(MPIPE_ERR_INVALID_ARG, "null costs");
  if (!all_finite_nonneg(cost, n)) return set_error(MPIPE_ERR_INVALID_ARG, "event costs must be finite and >= 0");
  // predecessors: the typed edges and the previous event of each rank's sequence
  std::vector<std::vector<int>> succ(n);
  std::vector<int> indeg(n, 0);
  auto link = [&](int a, int b) { succ[a].push_back(b), ++indeg[b]; };
  for (const mpipe_edge& e : d->edges) link(e.from, e.to);
  for (const std::vector<int>& seq : d->nodes)
    for (size_t i = 1; i < seq.size(); ++i) link(seq[i - 1], seq[i]);
  std::vector<double> st(n, 0.0), fin(n, 0.0);
  std::vector<int> ready;
  for (int i = 0; i < n; ++i)
    if (!indeg[i]) ready.push_back(i);
  int done = 0;
  while (!ready.empty()) {   // longest path in topological order
    const int e = ready.back();
    ready.pop_back();
    fin[e] = st[e] + cost[e];
    ++done;
    for (int s : succ[e]) {
      st[s] = std::max(st[s], fin[e]);
      if (--indeg[s] == 0) ready.push_back(s);
    }
  }
  if (done != n) return set_error(MPIPE_ERR_INVALID_ARG, "the order graph has a cycle");
  const double T = n ? *std::max_element(fin.begin(), fin.end()) : 0.0;
  if (makespan) *makespan = T;
  if (bubble)
    for (int r = 0; r < d->P; ++r) {
      double busy = 0;
      for (int e : d->nodes[r]) busy += cost[e];
      bubble[r] = T - busy;
    }
  if (start) std::copy(st.begin(), st.end(), start);
  if (finish) std::copy(fin.begin(), fin.end(), finish);
  return MPIPE_OK;
}

mpipe_status mpipe_memory_peak(const mpipe_derived* d, const double* act_bytes, double* peak) {
  if (!d) return set_error(MPIPE_ERR_INVALID_ARG, "null derivation");
  if (!d->has_order) return set_error(MPIPE_ERR_UNSUPPORTED, d->no_order);
  if (!act_bytes || !peak) return set_error(MPIPE_ERR_INVALID_ARG, "null bytes or output");
  if (!all_finite_nonneg(act_bytes, d->events.size()))
    return set_error(MPIPE_ERR_INVALID_ARG, "activation bytes must be finite and >= 0");
  for (int r = 0; r < d->P; ++r) {
    double live = 0, top = 0;
    for (int e : d->nodes[r]) {
      const mpipe_event& ev = d->events[e];
      if (ev.kind == MPIPE_EV_FWD) {
        live += act_bytes[e];
        top = std::max(top, live);
        if (d->partner[e] < 0) live -= act_bytes[e];   // no backward reads it
      } else if (ev.kind == MPIPE_EV_BWD) {
        live -= act_bytes[d->partner[e]];
      }
    }
    peak[r] = top;
  }
  return MPIPE_OK;
}

}  // extern "C"
