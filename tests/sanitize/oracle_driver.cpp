// The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer: whole-encoder
// forward and backward in both precisions and every trainability mode, the building
// blocks, and the row scatter / gather, on small inputs from a fixed-seed generator
// (images, a temporal-patch-2 clip, per-slice segments, an empty micro-batch, bad
// metadata).  Built and run by tests/test_sanitize.py with g++; any sanitizer report, or
// a status other than the expected one, ends it with a non-zero status.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <vector>

#include "../../oracle/mpipe_ref.h"

namespace {

uint64_t g_state = 0x2545F4914F6CDD1Dull;
double normal01() {   // xorshift64* uniforms through Box-Muller
  auto u = [] {
    g_state ^= g_state >> 12;
    g_state ^= g_state << 25;
    g_state ^= g_state >> 27;
    return ((g_state * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0);
  };
  const double a = u() + 1e-12, b = u();
  return std::sqrt(-2.0 * std::log(a)) * std::cos(6.283185307179586 * b);
}
template <class T> std::vector<T> randn(size_t n, double s = 1.0) {
  std::vector<T> v(n);
  for (auto& x : v) x = (T)(s * normal01());
  return v;
}

int failures = 0;
void expect(bool ok, const char* what) {
  if (!ok) {
    std::fprintf(stderr, "FAILED: %s\n", what);
    ++failures;
  }
}

template <class T, class F>
void encoder_case(const ref_cfg& c, std::vector<int32_t> grid, std::vector<int32_t> cu, F fn) {
  const int n_items = (int)grid.size() / 3;
  int64_t N = 0, Tm = 0;
  for (int i = 0; i < n_items; ++i) {
    N += (int64_t)grid[3 * i] * grid[3 * i + 1] * grid[3 * i + 2];
    Tm += (int64_t)grid[3 * i] * (grid[3 * i + 1] / 2) * (grid[3 * i + 2] / 2);
  }
  const int64_t kpe = (int64_t)c.in_chans * c.temporal_patch * c.patch * c.patch;
  const int64_t np = ref_param_count(&c);
  auto w = randn<T>(np, 0.05);
  auto X = randn<T>((size_t)(N * kpe));
  // (at least one element: an empty vector's data() may be null, which means "no backward")
  auto dM = randn<T>((size_t)(Tm * c.llm_hidden) + 1);
  std::vector<T> M((size_t)(Tm * c.llm_hidden)), dW(np), dX((size_t)(N * kpe));
  const int n_seg = (int)cu.size() - 1;
  for (int mode = 0; mode <= 2; ++mode) {
    int rc = fn(&c, w.data(), X.data(), cu.data(), n_seg, grid.data(), n_items, mode, M.data(),
                nullptr, nullptr, nullptr);
    expect(rc == 0, "forward status");
    rc = fn(&c, w.data(), X.data(), cu.data(), n_seg, grid.data(), n_items, mode, M.data(),
            dM.data(), dW.data(), mode == 1 ? dX.data() : nullptr);
    expect(rc == (mode == 0 ? 1 : 0), "backward status");
  }
  // corrupt metadata: the first segment one row short
  if (n_seg >= 1 && cu[1] > 1) {
    std::vector<int32_t> bad = cu;
    bad[1] -= 1;
    const int rc = fn(&c, w.data(), X.data(), bad.data(), n_seg, grid.data(), n_items, 1, M.data(),
                      nullptr, nullptr, nullptr);
    expect(rc < 0, "bad segments rejected");
  }
}

}  // namespace

int main() {
  ref_cfg c{3, 14, 1, 16, 2, 2, 32, 2, 24, 1e-6, 10000.0};
  encoder_case<double>(c, {1, 4, 4, 1, 4, 6}, {0, 16, 40}, ref_encoder_f64);
  encoder_case<float>(c, {1, 4, 4, 1, 4, 6}, {0, 16, 40}, ref_encoder_f32);
  encoder_case<double>(c, {}, {0}, ref_encoder_f64);               // text-only micro-batch
  ref_cfg v{3, 14, 2, 16, 1, 2, 32, 2, 24, 1e-6, 10000.0};         // temporal patch 2
  encoder_case<double>(v, {3, 2, 4, 1, 2, 2}, {0, 8, 16, 24, 28}, ref_encoder_f64);
  encoder_case<float>(v, {3, 2, 4}, {0, 24}, ref_encoder_f32);

  // building blocks
  const int64_t M = 7, K = 12, Nn = 5;
  auto X = randn<double>(M * K), W = randn<double>(Nn * K), b = randn<double>(Nn);
  std::vector<double> Y(M * Nn), dX(M * K), dW(Nn * K), db(Nn);
  ref_linear_f64(X.data(), W.data(), b.data(), M, K, Nn, Y.data());
  ref_linear_bwd_f64(Y.data(), X.data(), W.data(), M, K, Nn, dX.data(), dW.data(), db.data());
  std::vector<double> Z(M * K), mu(M), rs(M), g(K, 1.0), be(K, 0.0), dg(K), dbe(K);
  ref_layernorm_f64(X.data(), g.data(), be.data(), M, K, 1e-6, Z.data(), mu.data(), rs.data());
  ref_layernorm_bwd_f64(Z.data(), X.data(), g.data(), mu.data(), rs.data(), M, K, dX.data(),
                        dg.data(), dbe.data());
  ref_gelu_f64(X.data(), M * K, Z.data());
  ref_gelu_grad_f64(X.data(), M * K, Z.data());
  const int32_t grid[] = {1, 2, 4, 2, 2, 2};
  std::vector<int32_t> py(16), px(16);
  expect(ref_positions(grid, 2, py.data(), px.data()) == 0, "positions");
  const int heads = 2, d = 8, ld = heads * d, Nq = 16;
  auto q = randn<double>(Nq * ld), k = randn<double>(Nq * ld), vv = randn<double>(Nq * ld);
  ref_rope2d_f64(q.data(), Nq, heads, d, ld, py.data(), px.data(), 10000.0, 0);
  ref_rope2d_f64(q.data(), Nq, heads, d, ld, py.data(), px.data(), 10000.0, 1);
  const int32_t cu[] = {0, 5, 16};
  std::vector<double> o(Nq * ld), lse(Nq * heads), dq(Nq * ld), dk(Nq * ld), dv(Nq * ld);
  ref_attention_f64(q.data(), k.data(), vv.data(), ld, cu, 2, heads, d, o.data(), ld, lse.data());
  ref_attention_bwd_f64(q.data(), k.data(), vv.data(), ld, o.data(), o.data(), ld, lse.data(), cu,
                        2, heads, d, dq.data(), dk.data(), dv.data(), ld);

  // scatter / gather: valid, out of range, repeated
  std::vector<uint16_t> mrows(3 * 4), emb(10 * 4), back(3 * 4);
  for (size_t i = 0; i < mrows.size(); ++i) mrows[i] = (uint16_t)(i * 977u);
  const int64_t good[] = {7, 0, 4}, out_of_range[] = {7, 10, 4}, repeated[] = {7, 7, 4};
  expect(ref_merge_scatter(mrows.data(), 3, 8, good, emb.data(), 10) == 0, "scatter");
  expect(ref_merge_gather(emb.data(), 10, 8, good, 3, back.data()) == 0, "gather");
  expect(back == mrows, "gather inverts scatter");
  expect(ref_merge_scatter(mrows.data(), 3, 8, out_of_range, emb.data(), 10) == -1, "range");
  expect(ref_merge_scatter(mrows.data(), 3, 8, repeated, emb.data(), 10) == -1, "repeat");
  expect(ref_merge_gather(emb.data(), 10, 8, out_of_range, 3, back.data()) == -1, "range g");

  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("oracle checks passed\n");
  return 0;
}
