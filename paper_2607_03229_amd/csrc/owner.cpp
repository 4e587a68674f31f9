// The step just before the encoder runs: which rank encodes which micro-batch.
//
// The transpose schedule replicates the encoder and lets the ByMicrobatch owner assign
// each micro-batch's Fwd(enc, m) to one rank, which runs it inside its warmup bubble
// (Sec. 4.2).  The cost model (Sec. 4.3) weighs a compute event by the roofline of its
// slab, max(W/F, D/B), and prices the encoder work a rank cannot hide as its spill,
// max(0, E_r - w_r), with E_r the summed encode cost of the micro-batches the rank owns
// and w_r its warmup bubble; the step pays the worst rank's spill.  The owner that
// minimises that maximum is a min-max balancing of encode cost against warmup slack;
// giving the heaviest encodes to the longest free slots is its greedy form.  Host code
// only.
#include <algorithm>
#include <cmath>
#include <numeric>
#include <string>
#include <vector>

#include "../../include/mpipe_sched.h"
#include "plan.h"

namespace mpipe {
mpipe_status set_error(mpipe_status s, const std::string& m);

// W (FLOPs) and D (algorithmic HBM bytes: each kernel's operands read once and its
// results written once) of the encoder's forward and backward slabs for one micro-batch.
SlabCost encoder_slab_cost(const Cfg& c, const Plan& P) {
  const double N = (double)P.N, Tm = (double)P.Tm, h = c.hidden, m = c.mlp, H = c.llm,
               L = c.layers, nh = c.heads, E = c.esz, kpe = c.kpe, s2 = (double)P.sum_len2;
  SlabCost r{};
  // FLOPs: the GEMMs and the two attention products (LayerNorm, GELU, RoPE and the
  // softmax are not counted)
  const double pe = 2 * N * kpe * h;
  const double blk = 8 * N * h * h + 4 * N * h * m + 4 * h * s2;
  const double mrg = 2 * Tm * (4 * h) * (4 * h) + 2 * Tm * (4 * h) * H;
  r.fwd_flops = pe + L * blk + mrg;
  // bytes
  const double w_pe = (h * kpe + h) * E, w_blk = (4 * h * h + 2 * h * m + 6 * h + 2 * m + 4 * h) * E,
               w_mrg = (16 * h * h + 4 * h + 4 * h * H + H + 2 * h) * E;
  const bool blocks_tape = P.mode == MODE_TRAINED, merger_tape = P.mode != MODE_FROZEN;
  const double a_pe = N * kpe * E + 4 * N * h;
  const double a_blk = (4 * N * h + E * N * h + 8 * N)               // LN1
                       + (E * N * h + 3 * E * N * h)                 // qkv
                       + 2 * (2 * E * N * h)                         // RoPE on q, k
                       + (3 * E * N * h + E * N * h + 4 * nh * N)    // attention
                       + (E * N * h + 8 * N * h)                     // proj + residual
                       + (4 * N * h + E * N * h + 8 * N)             // LN2
                       + (E * N * h + E * N * m * (blocks_tape ? 2 : 1))   // fc1 (+GELU')
                       + (E * N * m + 8 * N * h);                    // fc2 + residual
  const double a_mrg = (4 * N * h + E * N * h + 8 * N)               // LN
                       + (E * N * h + E * N * h * (merger_tape ? 2 : 1))   // fc1 (+GELU')
                       + (E * N * h + E * Tm * H);                   // fc2
  r.fwd_bytes = a_pe + w_pe + L * (a_blk + w_blk) + a_mrg + w_mrg;
  // backward: the input and weight gradients of every product of a trainable part (the
  // patch gradient is not requested); bytes: twice that part's forward activation
  // traffic, plus its weights read once and their fp32 gradients read and written once
  const double g8 = 8.0 / E;   // fp32 gradient read + write per weight, in units of E bytes
  if (P.mode == MODE_TRAINED) {
    r.bwd_flops = 2 * r.fwd_flops - pe;
    r.bwd_bytes = 2 * (a_pe + L * a_blk + a_mrg) + (1 + g8) * (w_pe + L * w_blk + w_mrg);
  } else if (P.mode == MODE_MERGER) {
    r.bwd_flops = 2 * mrg;
    r.bwd_bytes = 2 * a_mrg + (1 + g8) * w_mrg;
  }
  return r;
}

}  // namespace mpipe

namespace {

using mpipe::set_error;

// E_r in the order of the definition (micro-batches by index), so that every caller
// that sums the same assignment gets the same bits.
void rank_loads(const double* cost, int n_mb, const int32_t* owner, int n_ranks,
                std::vector<double>& E) {
  E.assign(n_ranks, 0.0);
  for (int i = 0; i < n_mb; ++i) E[owner[i]] += cost[i];
}

double worst_spill(const std::vector<double>& E, const double* w, double* spill) {
  double worst = 0.0;
  for (size_t r = 0; r < E.size(); ++r) {
    const double s = std::max(0.0, E[r] - w[r]);
    if (spill) spill[r] = s;
    worst = std::max(worst, s);
  }
  return worst;
}

// Heaviest encode first, each to the rank with the most remaining slack w_r - E_r
// (ties to the lower rank); ties in cost keep index order.
void greedy(const double* cost, int n_mb, const double* w, int n_ranks, int32_t* owner) {
  std::vector<int> ord(n_mb);
  std::iota(ord.begin(), ord.end(), 0);
  std::stable_sort(ord.begin(), ord.end(), [&](int a, int b) { return cost[a] > cost[b]; });
  std::vector<double> E(n_ranks, 0.0);
  for (int i : ord) {
    int best = 0;
    for (int r = 1; r < n_ranks; ++r)
      if (w[r] - E[r] > w[best] - E[best]) best = r;
    owner[i] = best;
    E[best] += cost[i];
  }
}

// Improvement of an assignment by single moves and pairwise swaps: while the rank with
// the largest E_r - w_r has any (ties to the lower rank), try moving one of its
// micro-batches to another rank, or swapping one of them with a cheaper one there, and
// apply the candidate that makes the profile of E_r - w_r, sorted in decreasing order,
// lexicographically smallest, if it is smaller than the current profile.  Every step
// strictly decreases that profile, so the descent ends.
void refine(const double* cost, int n_mb, const double* w, int n_ranks, int32_t* owner) {
  std::vector<double> E;
  rank_loads(cost, n_mb, owner, n_ranks, E);
  auto profile = [&](const std::vector<double>& e) {
    std::vector<double> v(n_ranks);
    for (int r = 0; r < n_ranks; ++r) v[r] = e[r] - w[r];
    std::sort(v.begin(), v.end(), [](double x, double y) { return x > y; });
    return v;
  };
  for (;;) {
    int top = 0;
    for (int r = 1; r < n_ranks; ++r)
      if (E[r] - w[r] > E[top] - w[top]) top = r;
    if (E[top] - w[top] <= 0) return;   // nothing spills
    std::vector<double> best = profile(E);
    int bm = -1, bn = -1, bq = -1;
    std::vector<double> e2 = E;
    for (int m = 0; m < n_mb; ++m) {
      if (owner[m] != top) continue;
      for (int q = 0; q < n_ranks; ++q) {
        if (q == top) continue;
        e2[top] = E[top] - cost[m];
        e2[q] = E[q] + cost[m];
        std::vector<double> pr = profile(e2);
        if (pr < best) best = pr, bm = m, bn = -1, bq = q;
        e2[q] = E[q];
        for (int n = 0; n < n_mb; ++n) {
          if (owner[n] != q || cost[n] >= cost[m]) continue;
          e2[top] = E[top] - cost[m] + cost[n];
          e2[q] = E[q] + cost[m] - cost[n];
          pr = profile(e2);
          if (pr < best) best = pr, bm = m, bn = n, bq = q;
          e2[q] = E[q];
        }
        e2[top] = E[top];
      }
    }
    if (bm < 0) return;
    owner[bm] = bq;
    if (bn >= 0) owner[bn] = top;
    rank_loads(cost, n_mb, owner, n_ranks, E);
  }
}

// Exact minimum of max_r max(0, E_r - w_r) by depth-first branch and bound over the
// micro-batches in decreasing cost.  A node's bound is the larger of its partial maximum
// (maxima only grow as micro-batches are added) and the water level of the remaining
// cost R: the least s with sum_r max(0, w_r + s - E_r) >= R, which is what any
// completion needs even if encodes could be split between ranks.  A branch whose bound
// reaches the incumbent is cut; ranks in the same state (equal bubble and load) are
// interchangeable, so only the first of them is tried, and children go in order of
// decreasing slack.  The incumbent starts at the refined assignment, and the search stops
// early when it meets the root's bound.
struct Exact {
  const double* cost;
  const double* w;
  int n_mb, n_ranks;
  std::vector<int> ord;
  std::vector<double> E, rest;   // rest[k]: cost of the micro-batches ord[k..]
  std::vector<int32_t> cur, best;
  double best_val = 0, lower = 0;
  long long nodes = 0, node_cap = 0;
  bool capped = false, done = false;

  double water_level(double R) const {
    double a[MPIPE_OWNER_EXACT_MAX_RANKS];
    for (int r = 0; r < n_ranks; ++r) a[r] = w[r] - E[r];
    std::sort(a, a + n_ranks, [](double x, double y) { return x > y; });
    double sum = 0;
    for (int k = 1; k <= n_ranks; ++k) {   // the k ranks with the most slack take R
      sum += a[k - 1];
      const double s = (R - sum) / k;
      if (k == n_ranks || s <= -a[k]) return s;
    }
    return 0;
  }

  void dfs(int k, double partial) {
    if (done || capped) return;
    if (++nodes > node_cap) {
      capped = true;
      return;
    }
    if (k == n_mb) {
      if (partial < best_val) {
        best_val = partial;
        best = cur;
        if (best_val <= lower) done = true;
      }
      return;
    }
    if (std::max(partial, water_level(rest[k])) >= best_val) return;
    const int i = ord[k];
    int cand[MPIPE_OWNER_EXACT_MAX_RANKS];
    int nc = 0;
    for (int r = 0; r < n_ranks; ++r) {
      bool twin = false;
      for (int q = 0; q < r && !twin; ++q) twin = (w[q] == w[r] && E[q] == E[r]);
      if (!twin) cand[nc++] = r;
    }
    std::stable_sort(cand, cand + nc, [&](int x, int y) { return w[x] - E[x] > w[y] - E[y]; });
    for (int c = 0; c < nc; ++c) {
      const int r = cand[c];
      const double s = std::max(partial, std::max(0.0, E[r] + cost[i] - w[r]));
      if (s >= best_val) continue;
      E[r] += cost[i];
      cur[i] = r;
      dfs(k + 1, s);
      E[r] -= cost[i];
      if (done || capped) return;
    }
  }
};

}  // namespace

extern "C" {

mpipe_status mpipe_owner_map(const double* cost, int32_t n_mb, const double* warmup,
                             int32_t n_ranks, int32_t method, int32_t* owner, double* spill,
                             double* max_spill) {
  if (n_mb < 0 || n_ranks < 1) return set_error(MPIPE_ERR_INVALID_ARG, "need n_mb >= 0, n_ranks >= 1");
  if (!warmup || (n_mb > 0 && (!cost || !owner)))
    return set_error(MPIPE_ERR_INVALID_ARG, "null cost, warmup or owner");
  if (method != MPIPE_OWNER_GREEDY && method != MPIPE_OWNER_EXACT && method != MPIPE_OWNER_REFINED)
    return set_error(MPIPE_ERR_INVALID_ARG, "unknown owner method");
  for (int i = 0; i < n_mb; ++i)
    if (!std::isfinite(cost[i]) || cost[i] < 0)
      return set_error(MPIPE_ERR_INVALID_ARG, "encode costs must be finite and >= 0");
  for (int r = 0; r < n_ranks; ++r)
    if (!std::isfinite(warmup[r]) || warmup[r] < 0)
      return set_error(MPIPE_ERR_INVALID_ARG, "warmup bubbles must be finite and >= 0");
  if (method == MPIPE_OWNER_EXACT && n_ranks > MPIPE_OWNER_EXACT_MAX_RANKS)
    return set_error(MPIPE_ERR_UNSUPPORTED, "exact owner search is limited to " +
                                                std::to_string(MPIPE_OWNER_EXACT_MAX_RANKS) +
                                                " ranks");
  if (method == MPIPE_OWNER_EXACT && n_mb > MPIPE_OWNER_EXACT_MAX_MB)
    return set_error(MPIPE_ERR_UNSUPPORTED, "exact owner search is limited to " +
                                                std::to_string(MPIPE_OWNER_EXACT_MAX_MB) +
                                                " micro-batches");
  std::vector<double> E;
  if (n_mb > 0) {
    greedy(cost, n_mb, warmup, n_ranks, owner);
    if (method != MPIPE_OWNER_GREEDY) refine(cost, n_mb, warmup, n_ranks, owner);
    if (method == MPIPE_OWNER_EXACT) {
      Exact x{cost, warmup, n_mb, n_ranks, {}, {}, {}, {}, {}};
      x.ord.resize(n_mb);
      std::iota(x.ord.begin(), x.ord.end(), 0);
      std::stable_sort(x.ord.begin(), x.ord.end(), [&](int a, int b) { return cost[a] > cost[b]; });
      x.E.assign(n_ranks, 0.0);
      x.rest.assign(n_mb + 1, 0.0);
      for (int k = n_mb - 1; k >= 0; --k) x.rest[k] = x.rest[k + 1] + cost[x.ord[k]];
      x.cur.assign(n_mb, 0);
      x.best.assign(owner, owner + n_mb);
      rank_loads(cost, n_mb, owner, n_ranks, E);
      x.best_val = worst_spill(E, warmup, nullptr);
      double total = 0, cmax = 0, wmax = 0;
      for (int i = 0; i < n_mb; ++i) total += cost[i], cmax = std::max(cmax, cost[i]);
      for (int r = 0; r < n_ranks; ++r) wmax = std::max(wmax, warmup[r]);
      x.lower = std::max({0.0, x.water_level(total), cmax - wmax});
      x.node_cap = MPIPE_OWNER_EXACT_NODE_CAP;
      if (x.best_val > x.lower) x.dfs(0, 0.0);
      if (x.capped)
        return set_error(MPIPE_ERR_UNSUPPORTED, "exact owner search exceeded its node budget");
      std::copy(x.best.begin(), x.best.end(), owner);
    }
  }
  rank_loads(cost, n_mb, owner ? owner : nullptr, n_ranks, E);
  const double worst = worst_spill(E, warmup, spill);
  if (max_spill) *max_spill = worst;
  return MPIPE_OK;
}

}  // extern "C"
