// Host code under AddressSanitizer and UndefinedBehaviorSanitizer: the micro-batch
// planner (metadata validation, workspace and tape layout, split plan), the encoder cost
// model, the ByMicrobatch owner map and the schedule algebra, driven on valid and invalid
// inputs from a fixed-seed generator.  Built and run by tests/test_sanitize.py with g++;
// any sanitizer report, or a broken layout invariant, ends it with a non-zero status.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "../../include/mpipe_derive.h"
#include "../../include/mpipe_sched.h"
#include "../../paper_2607_03229_amd/csrc/plan.h"

namespace mpipe {
// the library's error channel (encoder.cpp) is not linked here: report nothing, keep the code
mpipe_status set_error(mpipe_status s, const std::string&) { return s; }
}  // namespace mpipe

using namespace mpipe;

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint32_t next_u32() {   // xorshift64*
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return (uint32_t)((g_state * 0x2545F4914F6CDD1Dull) >> 32);
}
int uniform(int lo, int hi) { return lo + (int)(next_u32() % (uint32_t)(hi - lo + 1)); }
double unit() { return next_u32() / 4294967296.0; }

int failures = 0;
void expect(bool ok, const char* what, int k) {
  if (!ok) {
    std::fprintf(stderr, "FAILED: %s (case %d)\n", what, k);
    ++failures;
  }
}

Cfg make_cfg(int hidden, int heads, int mlp, int llm, int layers, int tpatch, int dtype) {
  Cfg c;
  c.hidden = hidden;
  c.heads = heads;
  c.mlp = mlp;
  c.llm = llm;
  c.layers = layers;
  c.tpatch = tpatch;
  c.dtype = dtype;
  derive_cfg(c);
  return c;
}

void check_layout(const std::vector<Region>& R, size_t total, int k) {
  size_t prev_end = 0;
  for (size_t i = 0; i < R.size(); ++i) {
    expect(R[i].off % 256 == 0, "region aligned", k);
    expect(i == 0 || R[i].off >= prev_end + 256, "guard gap before region", k);
    prev_end = R[i].off + R[i].bytes;
  }
  expect(R.empty() || prev_end + 256 <= total, "guard after the last region", k);
}

void plan_cases() {
  const Cfg cfgs[] = {make_cfg(128, 4, 512, 256, 2, 1, 0), make_cfg(1280, 16, 5120, 3584, 3, 2, 1),
                      make_cfg(640, 8, 1280, 512, 1, 2, 1), make_cfg(1024, 16, 4096, 4096, 0, 1, 1)};
  for (int k = 0; k < 600; ++k) {
    const Cfg& c = cfgs[k % 4];
    const int n_items = uniform(0, 6);
    std::vector<int32_t> thw;
    std::vector<int32_t> cu{0};
    for (int i = 0; i < n_items; ++i) {
      const int t = uniform(1, 3) == 3 ? 8 : 1, gh = 2 * uniform(1, 24), gw = 2 * uniform(1, 24);
      thw.insert(thw.end(), {t, gh, gw});
      if (t > 1 && uniform(0, 1)) {   // one segment per temporal slice
        for (int s = 0; s < t; ++s) cu.push_back(cu.back() + gh * gw);
      } else {
        cu.push_back(cu.back() + t * gh * gw);
      }
    }
    // corruptions: odd side, oversized side, crossing segment, non-increasing, short end
    const int bad = n_items > 1 ? uniform(0, 9) : 0;
    if (bad == 1) thw[1] += 1;
    if (bad == 2) thw[2] = 32770;
    if (bad == 3 && cu.size() > 2) cu.erase(cu.begin() + 1);
    if (bad == 4 && cu.size() > 2) cu[1] = cu[2];
    if (bad == 5) cu.back() -= 1;
    if (bad == 6) thw[0] = 0;
    if (bad == 7) thw[1] = -4;
    const int n_seg = (int)cu.size() - 1;
    for (int mode = 0; mode <= 3; ++mode) {
      Plan P;
      std::string err;
      const int rc = build_plan(c, cu.data(), n_seg, thw.empty() ? nullptr : thw.data(), n_items,
                                mode, P, err);
      if (mode == 3) {
        expect(rc != 0, "unknown mode rejected", k);
        continue;
      }
      if (bad >= 1 && bad <= 7) {
        expect(rc != 0 || bad == 3, "corrupt metadata rejected", k);
      }
      if (rc != 0) {
        expect(!err.empty(), "rejection has a reason", k);
        continue;
      }
      check_layout(P.ws_regions, P.ws_bytes, k);
      check_layout(P.tape_regions, P.tape_bytes, k);
      expect((int64_t)P.pos.size() == P.N, "one position per row", k);
      for (int64_t r = 0; r < P.N; ++r) expect(P.pos[r] >= 0, "position sign", k);
      const SlabCost sc = encoder_slab_cost(c, P);
      expect(std::isfinite(sc.fwd_flops) && sc.fwd_flops >= 0, "cost finite", k);
    }
  }
  // split plans over a sweep of shapes
  for (int64_t M : {1, 255, 1280, 3840, 5120})
    for (int64_t N : {8, 1176, 1280, 5120})
      for (int64_t K : {0, 1, 1000, 2048, 42940, 500000}) {
        const GemmSplit g = choose_split(M, N, K);
        expect(g.splits >= 1 && g.splits <= 4, "split count", (int)K);
        expect(g.splits == 1 || (int64_t)g.kps * (g.splits - 1) < K, "every split has work", (int)K);
      }
}

void owner_cases() {
  for (int k = 0; k < 300; ++k) {
    const int n_mb = uniform(0, 8), n_ranks = uniform(1, 4);
    std::vector<double> cost(n_mb), warm(n_ranks), spill(n_ranks);
    std::vector<int32_t> owner(n_mb);
    for (auto& v : cost) v = unit() * 3.0;
    for (auto& v : warm) v = unit() * 2.0;
    if (k % 17 == 5 && n_mb) cost[0] = NAN;
    if (k % 19 == 7) warm[0] = -1.0;
    for (int method = 0; method < 4; ++method) {
      double worst = 0;
      const mpipe_status st = mpipe_owner_map(cost.data(), n_mb, warm.data(), n_ranks, method,
                                              owner.data(), spill.data(), &worst);
      if (st == MPIPE_OK)
        for (int m = 0; m < n_mb; ++m) expect(owner[m] >= 0 && owner[m] < n_ranks, "owner rank", k);
    }
  }
  double w = 1.0;
  int32_t o = 0;
  expect(mpipe_owner_map(nullptr, 1, &w, 1, 0, &o, nullptr, nullptr) != MPIPE_OK, "null cost", 0);
}

void derive_cases() {
  const std::vector<std::vector<int32_t>> scheds = {
      {MPIPE_SK_1F1B}, {MPIPE_SK_GPIPE}, {MPIPE_SK_TRANSPOSE},
      {MPIPE_SK_TRANSPOSE, MPIPE_SK_1F1B}, {MPIPE_SK_TRANSPOSE, MPIPE_SK_GPIPE},
      {MPIPE_SK_1F1B, MPIPE_SK_1F1B, MPIPE_SK_1F1B}, {MPIPE_SK_TRANSPOSE, MPIPE_SK_1F1B, MPIPE_SK_1F1B},
      {MPIPE_SK_TRANSPOSE, MPIPE_SK_1F1B, MPIPE_SK_TRANSPOSE}, {MPIPE_SK_1F1B, MPIPE_SK_GPIPE}};
  int k = 0;
  for (const auto& sc : scheds)
    for (int P = 1; P <= 3; ++P)
      for (int M = 1; M <= 5; M += 2)
        for (int mask = 0; mask < (1 << sc.size()); ++mask, ++k) {
          const int R = (int)sc.size();
          std::vector<int32_t> cut, train(R);
          int layers = 0;
          for (int j = 0; j < R; ++j) {
            const int sz = sc[j] == MPIPE_SK_TRANSPOSE ? 3 : (j % 2 ? P + 2 : 2 * P + 1);
            layers += sz;
            if (j + 1 < R) cut.push_back(layers);
            train[j] = (mask >> j) & 1;
          }
          std::vector<int32_t> owner(M);
          for (int m = 0; m < M; ++m) owner[m] = (m * 7 + 3) % P;
          mpipe_derived* d = nullptr;
          const mpipe_status st = mpipe_derive(cut.empty() ? nullptr : cut.data(), R, layers,
                                               sc.data(), train.data(), P, M,
                                               (k & 1) ? owner.data() : nullptr, &d);
          if (st != MPIPE_OK) {
            expect(d == nullptr, "no handle on error", k);
            continue;
          }
          int32_t has_order = 0, ne = 0, nd = 0, ns = 0, nr = 0;
          expect(mpipe_derived_shape(d, &has_order, &ne, &nd, &ns, &nr) == MPIPE_OK, "shape", k);
          std::vector<mpipe_event> ev(ne);
          std::vector<mpipe_edge> ed(nd);
          std::vector<mpipe_seam> sm(ns);
          std::vector<int32_t> rr(nr), rg(nr), own(M), lo(P), hi(P);
          mpipe_derived_lists(d, ev.data(), ed.data(), sm.data(), rr.data(), rg.data());
          mpipe_derived_owner(d, own.data());
          for (int j = 0; j < R; ++j) {
            int32_t lay = 0, rb = 0;
            mpipe_derived_placement(d, j, &lay, &rb, lo.data(), hi.data());
          }
          for (int r = 0; r < P; ++r) {
            const int32_t n = mpipe_derived_nodes(d, r, nullptr, 0);
            std::vector<int32_t> nodes(n > 0 ? n : 0);
            if (n > 0) mpipe_derived_nodes(d, r, nodes.data(), n);
          }
          expect(mpipe_derived_nodes(d, P, nullptr, 0) == -1, "rank out of range", k);
          if (has_order) {
            std::vector<double> fc(R * M), bc(R * M), seam((R > 1 ? R - 1 : 1) * M), red(R),
                cost(ne), bub(P), start(ne), fin(ne), act(ne), peak(P);
            for (auto* v : {&fc, &bc, &seam, &red, &act})
              for (auto& x : *v) x = unit();
            double T = 0;
            expect(mpipe_event_costs(d, fc.data(), bc.data(), R > 1 ? seam.data() : nullptr,
                                     red.data(), 1e-5, 1e-9, 0.1, cost.data()) == MPIPE_OK,
                   "event costs", k);
            expect(mpipe_makespan(d, cost.data(), &T, bub.data(), start.data(), fin.data()) ==
                       MPIPE_OK, "makespan", k);
            expect(mpipe_memory_peak(d, act.data(), peak.data()) == MPIPE_OK, "memory peak", k);
          }
          mpipe_derived_destroy(d);
        }
}

}  // namespace

int main() {
  plan_cases();
  owner_cases();
  derive_cases();
  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("host checks passed\n");
  return 0;
}
