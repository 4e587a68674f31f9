// Plain CPU oracle for the replicated-encoder step -- TEST INFRASTRUCTURE ONLY.
//
// Written from the definitions, in plain loops (OpenMP only splits independent
// rows / columns / (segment, head) pairs across threads; every sum runs in its
// natural index order, so results do not depend on the thread count).
// It shares nothing with the HIP library.  See mpipe_ref.h for the contract.
//
// Encoder definition (the paper names only "the ViT encoder from Qwen2-VL",
// Sec. 5 Experiment A; the block structure below is the stated reading):
//   H0 = X Wpe^T + bpe
//   per layer:  A = LN1(H); [Q|K|V] = A Wqkv^T + bqkv; Q,K <- RoPE2D(y, x)
//               O = softmax(Q K^T / sqrt(d)) V   within each attention segment
//               H <- H + O Wo^T + bo
//               B = LN2(H); H <- H + GELU(B W1^T + b1) W2^T + b2
//   merger:     Z = LN(H); z~ = [Z(0,0)|Z(0,1)|Z(1,0)|Z(1,1)] per 2x2 window
//               M = GELU(z~ Wm1^T + bm1) Wm2^T + bm2
// Backward: standard reverse-mode derivatives of the above; present only for
// a trainable encoder (Lemma 1, gate iii), weight gradients Accumulate (+=).
#include "mpipe_ref.h"

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>
#include <omp.h>

namespace {

template <class T> using Vec = std::vector<T>;

// ------------------------------------------------------------------------
// Parameter table: (name, rows, cols) in flat-buffer order; Linear W is [out][in].
// ------------------------------------------------------------------------
struct PEntry { std::string name; int64_t rows, cols; };

std::vector<PEntry> param_entries(const ref_cfg& c) {
  const int64_t h = c.hidden, m = c.mlp, H = c.llm_hidden;
  const int64_t kpe = (int64_t)c.in_chans * c.temporal_patch * c.patch * c.patch;
  const int64_t mh = (int64_t)c.merge * c.merge * h;
  std::vector<PEntry> t;
  t.push_back({"pe.w", h, kpe});
  t.push_back({"pe.b", h, 1});
  for (int l = 0; l < c.layers; ++l) {
    std::string p = "blk" + std::to_string(l) + ".";
    t.push_back({p + "ln1.g", h, 1});
    t.push_back({p + "ln1.b", h, 1});
    t.push_back({p + "qkv.w", 3 * h, h});
    t.push_back({p + "qkv.b", 3 * h, 1});
    t.push_back({p + "proj.w", h, h});
    t.push_back({p + "proj.b", h, 1});
    t.push_back({p + "ln2.g", h, 1});
    t.push_back({p + "ln2.b", h, 1});
    t.push_back({p + "fc1.w", m, h});
    t.push_back({p + "fc1.b", m, 1});
    t.push_back({p + "fc2.w", h, m});
    t.push_back({p + "fc2.b", h, 1});
  }
  t.push_back({"merger.ln.g", h, 1});
  t.push_back({"merger.ln.b", h, 1});
  t.push_back({"merger.fc1.w", mh, mh});
  t.push_back({"merger.fc1.b", mh, 1});
  t.push_back({"merger.fc2.w", H, mh});
  t.push_back({"merger.fc2.b", H, 1});
  return t;
}

// ------------------------------------------------------------------------
// Building blocks
// ------------------------------------------------------------------------

// Y[m][n] = sum_k X[m][k] W[n][k] + b[n]
template <class T>
void linear(const T* X, const T* W, const T* b, int64_t M, int64_t K, int64_t N, T* Y) {
  Vec<T> Wt((size_t)K * N);  // W transposed, so the inner loop runs over n
  for (int64_t n = 0; n < N; ++n)
    for (int64_t k = 0; k < K; ++k) Wt[(size_t)k * N + n] = W[(size_t)n * K + k];
#pragma omp parallel for schedule(static)
  for (int64_t m = 0; m < M; ++m) {
    T* y = Y + (size_t)m * N;
    for (int64_t n = 0; n < N; ++n) y[n] = 0;
    for (int64_t k = 0; k < K; ++k) {
      const T a = X[(size_t)m * K + k];
      const T* w = &Wt[(size_t)k * N];
      for (int64_t n = 0; n < N; ++n) y[n] += a * w[n];
    }
    if (b)
      for (int64_t n = 0; n < N; ++n) y[n] += b[n];
  }
}

// dX = dY W ; dW += dY^T X ; db += column sums of dY   (any output may be null)
template <class T>
void linear_bwd(const T* dY, const T* X, const T* W, int64_t M, int64_t K, int64_t N,
                T* dX, T* dW, T* db) {
  if (dX) {
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
      T* dx = dX + (size_t)m * K;
      for (int64_t k = 0; k < K; ++k) dx[k] = 0;
      for (int64_t n = 0; n < N; ++n) {
        const T a = dY[(size_t)m * N + n];
        const T* w = W + (size_t)n * K;
        for (int64_t k = 0; k < K; ++k) dx[k] += a * w[k];
      }
    }
  }
  if (dW) {
#pragma omp parallel
    {
      Vec<T> acc((size_t)K);
#pragma omp for schedule(static)
      for (int64_t n = 0; n < N; ++n) {
        for (int64_t k = 0; k < K; ++k) acc[k] = 0;
        for (int64_t m = 0; m < M; ++m) {
          const T a = dY[(size_t)m * N + n];
          const T* x = X + (size_t)m * K;
          for (int64_t k = 0; k < K; ++k) acc[k] += a * x[k];
        }
        T* dw = dW + (size_t)n * K;
        for (int64_t k = 0; k < K; ++k) dw[k] += acc[k];
      }
    }
  }
  if (db) {
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
      T s = 0;
      for (int64_t m = 0; m < M; ++m) s += dY[(size_t)m * N + n];
      db[n] += s;
    }
  }
}

// LayerNorm over each row of length n: biased variance, eps inside the sqrt.
template <class T>
void layernorm(const T* X, const T* g, const T* b, int64_t M, int64_t n, double eps,
               T* Y, T* mean, T* rstd) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < M; ++r) {
    const T* x = X + (size_t)r * n;
    T mu = 0;
    for (int64_t i = 0; i < n; ++i) mu += x[i];
    mu /= (T)n;
    T var = 0;
    for (int64_t i = 0; i < n; ++i) var += (x[i] - mu) * (x[i] - mu);
    var /= (T)n;
    const T rs = (T)1 / std::sqrt(var + (T)eps);
    T* y = Y + (size_t)r * n;
    for (int64_t i = 0; i < n; ++i) y[i] = (x[i] - mu) * rs * g[i] + b[i];
    if (mean) mean[r] = mu;
    if (rstd) rstd[r] = rs;
  }
}

// dX = rstd * (gdy - mean(gdy) - xhat * mean(gdy * xhat)), gdy = dY * g ;
// dg += sum_rows dY * xhat ; db += sum_rows dY
template <class T>
void layernorm_bwd(const T* dY, const T* X, const T* g, const T* mean, const T* rstd,
                   int64_t M, int64_t n, T* dX, T* dg, T* db) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < M; ++r) {
    const T* x = X + (size_t)r * n;
    const T* dy = dY + (size_t)r * n;
    T s1 = 0, s2 = 0;
    for (int64_t i = 0; i < n; ++i) {
      const T xh = (x[i] - mean[r]) * rstd[r];
      const T gd = dy[i] * g[i];
      s1 += gd;
      s2 += gd * xh;
    }
    s1 /= (T)n;
    s2 /= (T)n;
    T* dx = dX + (size_t)r * n;
    for (int64_t i = 0; i < n; ++i) {
      const T xh = (x[i] - mean[r]) * rstd[r];
      dx[i] = rstd[r] * (dy[i] * g[i] - s1 - xh * s2);
    }
  }
  if (dg || db) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
      T sg = 0, sb = 0;
      for (int64_t r = 0; r < M; ++r) {
        const T dy = dY[(size_t)r * n + i];
        sg += dy * (X[(size_t)r * n + i] - mean[r]) * rstd[r];
        sb += dy;
      }
      if (dg) dg[i] += sg;
      if (db) db[i] += sb;
    }
  }
}

// GELU, exact erf form: u * Phi(u)
template <class T> inline T gelu(T u) {
  return (T)0.5 * u * ((T)1 + std::erf(u / std::sqrt((T)2)));
}
// d/du GELU = Phi(u) + u * phi(u)
template <class T> inline T gelu_grad(T u) {
  const T Phi = (T)0.5 * ((T)1 + std::erf(u / std::sqrt((T)2)));
  const T phi = std::exp(-(T)0.5 * u * u) / std::sqrt((T)2 * (T)M_PI);
  return Phi + u * phi;
}

// 2D rotary position per head of width d (d % 4 == 0):
// omega_k = theta^(-4k/d), k < d/4; angle a_j = y*omega_j for j < d/4 and
// x*omega_(j-d/4) for d/4 <= j < d/2; rotate the pair (j, j + d/2) by a_j.
// inverse != 0 rotates by -a_j (the adjoint, used by the backward).
template <class T>
void rope2d(T* x, int64_t N, int heads, int d, int64_t ld, const int32_t* py, const int32_t* px,
            double theta, bool inverse) {
  const int half = d / 2, quarter = d / 4;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < N; ++r) {
    for (int hd = 0; hd < heads; ++hd) {
      T* v = x + (size_t)r * ld + (size_t)hd * d;
      for (int j = 0; j < half; ++j) {
        const int k = (j < quarter) ? j : j - quarter;
        const double omega = std::pow(theta, -4.0 * k / (double)d);
        const double a = ((j < quarter) ? py[r] : px[r]) * omega;
        const T cs = (T)std::cos(a), sn = inverse ? -(T)std::sin(a) : (T)std::sin(a);
        const T x1 = v[j], x2 = v[j + half];
        v[j] = x1 * cs - x2 * sn;
        v[j + half] = x2 * cs + x1 * sn;
      }
    }
  }
}

// Softmax attention inside each segment [cu[s], cu[s+1]), per head:
// S = Q K^T / sqrt(d); P = softmax over the segment's keys; O = P V;
// lse = rowmax + log(sum exp(S - rowmax)).
template <class T>
void attention(const T* q, const T* k, const T* v, int64_t ld, const int32_t* cu, int n_seg,
               int heads, int d, T* o, int64_t ldo, T* lse) {
  const T scale = (T)1 / std::sqrt((T)d);
#pragma omp parallel for schedule(dynamic)
  for (int64_t sh = 0; sh < (int64_t)n_seg * heads; ++sh) {
    const int s = (int)(sh / heads), hd = (int)(sh % heads);
    const int64_t a = cu[s], len = cu[s + 1] - cu[s];
    Vec<T> sc((size_t)len);
    for (int64_t i = 0; i < len; ++i) {
      const T* qi = q + (size_t)(a + i) * ld + (size_t)hd * d;
      T mx = -INFINITY;
      for (int64_t j = 0; j < len; ++j) {
        const T* kj = k + (size_t)(a + j) * ld + (size_t)hd * d;
        T dot = 0;
        for (int e = 0; e < d; ++e) dot += qi[e] * kj[e];
        sc[j] = dot * scale;
        if (sc[j] > mx) mx = sc[j];
      }
      T sum = 0;
      for (int64_t j = 0; j < len; ++j) {
        sc[j] = std::exp(sc[j] - mx);
        sum += sc[j];
      }
      T* oi = o + (size_t)(a + i) * ldo + (size_t)hd * d;
      for (int e = 0; e < d; ++e) oi[e] = 0;
      for (int64_t j = 0; j < len; ++j) {
        const T p = sc[j] / sum;
        const T* vj = v + (size_t)(a + j) * ld + (size_t)hd * d;
        for (int e = 0; e < d; ++e) oi[e] += p * vj[e];
      }
      if (lse) lse[(size_t)(a + i) * heads + hd] = mx + std::log(sum);  // [N][heads]
    }
  }
}

// Backward of the segment attention, with P recomputed from Q, K and lse:
// dV = P^T dO ; dP = dO V^T ; dS = P o (dP - rowsum(dO o O)) ; dQ = dS K / sqrt(d) ;
// dK = dS^T Q / sqrt(d).  Outputs are overwritten.
template <class T>
void attention_bwd(const T* q, const T* k, const T* v, int64_t ld, const T* o, const T* d_o,
                   int64_t ldo, const T* lse, const int32_t* cu, int n_seg, int heads, int d,
                   T* dq, T* dk, T* dv, int64_t ldd) {
  const T scale = (T)1 / std::sqrt((T)d);
#pragma omp parallel for schedule(dynamic)
  for (int64_t sh = 0; sh < (int64_t)n_seg * heads; ++sh) {
    const int s = (int)(sh / heads), hd = (int)(sh % heads);
    const int64_t a = cu[s], len = cu[s + 1] - cu[s];
    for (int64_t i = 0; i < len; ++i)
      for (int e = 0; e < d; ++e) {
        dq[(size_t)(a + i) * ldd + (size_t)hd * d + e] = 0;
        dk[(size_t)(a + i) * ldd + (size_t)hd * d + e] = 0;
        dv[(size_t)(a + i) * ldd + (size_t)hd * d + e] = 0;
      }
    Vec<T> p((size_t)len), dp((size_t)len);
    for (int64_t i = 0; i < len; ++i) {
      const T* qi = q + (size_t)(a + i) * ld + (size_t)hd * d;
      const T* oi = o + (size_t)(a + i) * ldo + (size_t)hd * d;
      const T* doi = d_o + (size_t)(a + i) * ldo + (size_t)hd * d;
      const T L = lse[(size_t)(a + i) * heads + hd];
      T delta = 0;
      for (int e = 0; e < d; ++e) delta += doi[e] * oi[e];
      for (int64_t j = 0; j < len; ++j) {
        const T* kj = k + (size_t)(a + j) * ld + (size_t)hd * d;
        const T* vj = v + (size_t)(a + j) * ld + (size_t)hd * d;
        T dot = 0, dd = 0;
        for (int e = 0; e < d; ++e) {
          dot += qi[e] * kj[e];
          dd += doi[e] * vj[e];
        }
        p[j] = std::exp(dot * scale - L);
        dp[j] = dd;
      }
      T* dqi = dq + (size_t)(a + i) * ldd + (size_t)hd * d;
      for (int64_t j = 0; j < len; ++j) {
        const T ds = p[j] * (dp[j] - delta);
        const T* kj = k + (size_t)(a + j) * ld + (size_t)hd * d;
        T* dkj = dk + (size_t)(a + j) * ldd + (size_t)hd * d;
        T* dvj = dv + (size_t)(a + j) * ldd + (size_t)hd * d;
        for (int e = 0; e < d; ++e) {
          dqi[e] += ds * kj[e] * scale;
          dkj[e] += ds * qi[e] * scale;
          dvj[e] += p[j] * doi[e];
        }
      }
    }
  }
}

// ------------------------------------------------------------------------
// Metadata
// ------------------------------------------------------------------------

// Inverse of the window-major row order: row r of an item with grid (t, gh, gw)
// is window w = r / 4 with (dh, dw) = ((r % 4) / 2, r % 2); the window index
// runs over (tau, hb, wb) with wb fastest.  y = 2 hb + dh, x = 2 wb + dw.
int positions(const int32_t* thw, int n_items, int32_t* py, int32_t* px) {
  int64_t row = 0;
  for (int it = 0; it < n_items; ++it) {
    const int t = thw[3 * it], gh = thw[3 * it + 1], gw = thw[3 * it + 2];
    if (t <= 0 || gh <= 0 || gw <= 0 || gh % 2 || gw % 2) return -2;
    const int64_t n = (int64_t)t * gh * gw;
    for (int64_t r = 0; r < n; ++r) {
      const int64_t w = r / 4;
      const int dh = (int)((r % 4) / 2), dw = (int)(r % 2);
      const int wb = (int)(w % (gw / 2));
      const int hb = (int)((w / (gw / 2)) % (gh / 2));
      py[row + r] = 2 * hb + dh;
      px[row + r] = 2 * wb + dw;
    }
    row += n;
  }
  return 0;
}

// Row of patch (tau, y, x) inside an item of grid (t, gh, gw): the forward map
// of the window-major order.
inline int64_t row_of(int tau, int y, int x, int gh, int gw) {
  const int64_t window = ((int64_t)tau * (gh / 2) + y / 2) * (gw / 2) + x / 2;
  return window * 4 + (y % 2) * 2 + (x % 2);
}

// Check cu_seqlens / grid_thw: items tile the packed rows; every segment lies
// inside one item and starts/ends on a temporal-slice boundary of that item.
int validate(const int32_t* cu, int n_seg, const int32_t* thw, int n_items, int64_t* n_rows) {
  if (n_items < 0 || n_seg < 0) return -1;
  int64_t N = 0;
  Vec<int64_t> start(n_items + 1);
  for (int it = 0; it < n_items; ++it) {
    const int t = thw[3 * it], gh = thw[3 * it + 1], gw = thw[3 * it + 2];
    if (t <= 0 || gh <= 0 || gw <= 0 || gh % 2 || gw % 2) return -2;
    start[it] = N;
    N += (int64_t)t * gh * gw;
  }
  start[n_items] = N;
  *n_rows = N;
  if (n_items == 0) return (n_seg == 0 || (n_seg >= 0 && cu && cu[n_seg] == 0)) ? 0 : -2;
  if (cu[0] != 0 || cu[n_seg] != N) return -2;
  int it = 0;
  for (int s = 0; s < n_seg; ++s) {
    if (cu[s + 1] <= cu[s]) return -2;
    while (it < n_items && cu[s] >= start[it + 1]) ++it;
    if (it >= n_items || cu[s + 1] > start[it + 1]) return -2;
    const int64_t slice = (int64_t)thw[3 * it + 1] * thw[3 * it + 2];
    if ((cu[s] - start[it]) % slice || (cu[s + 1] - start[it]) % slice) return -2;
  }
  return 0;
}

// ------------------------------------------------------------------------
// Encoder
// ------------------------------------------------------------------------
template <class T>
struct Layer {
  Vec<T> hin, a, mean1, rstd1, qkv, o, lse, hmid, b, mean2, rstd2, u, g;
};

template <class T>
int encoder(const ref_cfg& c, const T* w, const T* X, const int32_t* cu, int n_seg,
            const int32_t* thw, int n_items, int trainable, T* merged, const T* dM, T* dw,
            T* dX) {
  int64_t N = 0;
  int rc = validate(cu, n_seg, thw, n_items, &N);
  if (rc) return rc;
  if (c.hidden % c.heads || (c.hidden / c.heads) % 4 || c.merge != 2) return -1;
  if (trainable < 0 || trainable > 2) return -1;
  if (trainable == 2 && dX) return -1;   // the trainable source sends nothing upstream
  if (dM && !trainable) return 1;  // Lemma 1: a frozen encoder has no backward
  const bool merger_only = trainable == 2;
  if (N == 0) return 0;

  const int64_t h = c.hidden, m = c.mlp, Hl = c.llm_hidden, nh = c.heads, d = h / nh;
  const int64_t kpe = (int64_t)c.in_chans * c.temporal_patch * c.patch * c.patch;
  const int64_t mh = 4 * h;
  const int64_t Tm = N / 4;
  const double eps = c.ln_eps;

  // parameter views
  std::vector<PEntry> pe = param_entries(c);
  Vec<int64_t> off(pe.size() + 1, 0);
  for (size_t i = 0; i < pe.size(); ++i) off[i + 1] = off[i] + pe[i].rows * pe[i].cols;
  auto P = [&](int i) { return w + off[i]; };
  auto G = [&](int i) { return dw + off[i]; };
  const int L0 = 2, LN = 12;  // first block tensor, tensors per block
  const int MG = L0 + LN * c.layers;

  Vec<int32_t> py(N), px(N);
  positions(thw, n_items, py.data(), px.data());

  // ---- forward -----------------------------------------------------------
  Vec<T> H((size_t)N * h);
  linear(X, P(0), P(1), N, kpe, h, H.data());
  std::vector<Layer<T>> st(c.layers);
  Vec<T> tmp((size_t)N * h), tmpm((size_t)N * m);
  for (int l = 0; l < c.layers; ++l) {
    Layer<T>& S = st[l];
    const int b0 = L0 + LN * l;
    S.hin = H;
    S.a.resize(N * h); S.mean1.resize(N); S.rstd1.resize(N);
    layernorm(H.data(), P(b0 + 0), P(b0 + 1), N, h, eps, S.a.data(), S.mean1.data(), S.rstd1.data());
    S.qkv.resize(N * 3 * h);
    linear(S.a.data(), P(b0 + 2), P(b0 + 3), N, h, 3 * h, S.qkv.data());
    rope2d(S.qkv.data(), N, (int)nh, (int)d, 3 * h, py.data(), px.data(), c.rope_theta, false);
    rope2d(S.qkv.data() + h, N, (int)nh, (int)d, 3 * h, py.data(), px.data(), c.rope_theta, false);
    S.o.resize(N * h); S.lse.resize(N * nh);
    attention(S.qkv.data(), S.qkv.data() + h, S.qkv.data() + 2 * h, 3 * h, cu, n_seg, (int)nh,
              (int)d, S.o.data(), h, S.lse.data());
    linear(S.o.data(), P(b0 + 4), P(b0 + 5), N, h, h, tmp.data());
    for (size_t i = 0; i < H.size(); ++i) H[i] += tmp[i];
    S.hmid = H;
    S.b.resize(N * h); S.mean2.resize(N); S.rstd2.resize(N);
    layernorm(H.data(), P(b0 + 6), P(b0 + 7), N, h, eps, S.b.data(), S.mean2.data(), S.rstd2.data());
    S.u.resize(N * m); S.g.resize(N * m);
    linear(S.b.data(), P(b0 + 8), P(b0 + 9), N, h, m, S.u.data());
    for (size_t i = 0; i < S.u.size(); ++i) S.g[i] = gelu(S.u[i]);
    linear(S.g.data(), P(b0 + 10), P(b0 + 11), N, m, h, tmp.data());
    for (size_t i = 0; i < H.size(); ++i) H[i] += tmp[i];
    if (!dM || merger_only) { Layer<T> empty; std::swap(st[l], empty); }  // no block backward
  }
  // merger
  Vec<T> Z((size_t)N * h), meanz(N), rstdz(N);
  layernorm(H.data(), P(MG + 0), P(MG + 1), N, h, eps, Z.data(), meanz.data(), rstdz.data());
  // window concat: merged token (item, tau, hb, wb) takes the rows of patches
  // (tau, 2hb+dh, 2wb+dw) for (dh, dw) = (0,0), (0,1), (1,0), (1,1), in that order.
  Vec<int64_t> win_rows((size_t)Tm * 4);
  {
    int64_t base = 0, j = 0;
    for (int it = 0; it < n_items; ++it) {
      const int t = thw[3 * it], gh = thw[3 * it + 1], gw = thw[3 * it + 2];
      for (int tau = 0; tau < t; ++tau)
        for (int hb = 0; hb < gh / 2; ++hb)
          for (int wb = 0; wb < gw / 2; ++wb, ++j)
            for (int q = 0; q < 4; ++q)
              win_rows[(size_t)j * 4 + q] = base + row_of(tau, 2 * hb + q / 2, 2 * wb + q % 2, gh, gw);
      base += (int64_t)t * gh * gw;
    }
  }
  Vec<T> Zc((size_t)Tm * mh);
  for (int64_t j = 0; j < Tm; ++j)
    for (int q = 0; q < 4; ++q)
      std::memcpy(&Zc[(size_t)j * mh + q * h], &Z[(size_t)win_rows[j * 4 + q] * h], sizeof(T) * h);
  Vec<T> Um((size_t)Tm * mh), Gm((size_t)Tm * mh);
  linear(Zc.data(), P(MG + 2), P(MG + 3), Tm, mh, mh, Um.data());
  for (size_t i = 0; i < Um.size(); ++i) Gm[i] = gelu(Um[i]);
  linear(Gm.data(), P(MG + 4), P(MG + 5), Tm, mh, Hl, merged);
  if (!dM) return 0;

  // ---- backward (trainable only) ------------------------------------------
  Vec<T> dGm((size_t)Tm * mh), dZc((size_t)Tm * mh);
  linear_bwd(dM, Gm.data(), P(MG + 4), Tm, mh, Hl, dGm.data(), G(MG + 4), G(MG + 5));
  for (size_t i = 0; i < dGm.size(); ++i) dGm[i] *= gelu_grad(Um[i]);
  linear_bwd(dGm.data(), Zc.data(), P(MG + 2), Tm, mh, mh, dZc.data(), G(MG + 2), G(MG + 3));
  Vec<T> dZ((size_t)N * h);
  for (int64_t j = 0; j < Tm; ++j)
    for (int q = 0; q < 4; ++q)
      std::memcpy(&dZ[(size_t)win_rows[j * 4 + q] * h], &dZc[(size_t)j * mh + q * h], sizeof(T) * h);
  Vec<T> dH((size_t)N * h);
  layernorm_bwd(dZ.data(), H.data(), P(MG + 0), meanz.data(), rstdz.data(), N, h, dH.data(),
                G(MG + 0), G(MG + 1));
  // only the merger trainable: it is the trainable source (Lemma 1 over the encoder's
  // parts), so the frozen blocks and patch embedding below it run no backward
  if (merger_only) return 0;

  Vec<T> dG((size_t)N * m), dB((size_t)N * h), dHm((size_t)N * h), dO((size_t)N * h);
  Vec<T> dqkv((size_t)N * 3 * h), dA((size_t)N * h);
  for (int l = c.layers - 1; l >= 0; --l) {
    Layer<T>& S = st[l];
    const int b0 = L0 + LN * l;
    // MLP branch: H_out = H_mid + GELU(B W1^T + b1) W2^T + b2
    linear_bwd(dH.data(), S.g.data(), P(b0 + 10), N, m, h, dG.data(), G(b0 + 10), G(b0 + 11));
    for (size_t i = 0; i < dG.size(); ++i) dG[i] *= gelu_grad(S.u[i]);
    linear_bwd(dG.data(), S.b.data(), P(b0 + 8), N, h, m, dB.data(), G(b0 + 8), G(b0 + 9));
    layernorm_bwd(dB.data(), S.hmid.data(), P(b0 + 6), S.mean2.data(), S.rstd2.data(), N, h,
                  dHm.data(), G(b0 + 6), G(b0 + 7));
    for (size_t i = 0; i < dHm.size(); ++i) dHm[i] += dH[i];  // residual
    // attention branch: H_mid = H_in + O Wo^T + bo
    linear_bwd(dHm.data(), S.o.data(), P(b0 + 4), N, h, h, dO.data(), G(b0 + 4), G(b0 + 5));
    attention_bwd(S.qkv.data(), S.qkv.data() + h, S.qkv.data() + 2 * h, 3 * h, S.o.data(),
                  dO.data(), h, S.lse.data(), cu, n_seg, (int)nh, (int)d, dqkv.data(),
                  dqkv.data() + h, dqkv.data() + 2 * h, 3 * h);
    rope2d(dqkv.data(), N, (int)nh, (int)d, 3 * h, py.data(), px.data(), c.rope_theta, true);
    rope2d(dqkv.data() + h, N, (int)nh, (int)d, 3 * h, py.data(), px.data(), c.rope_theta, true);
    linear_bwd(dqkv.data(), S.a.data(), P(b0 + 2), N, h, 3 * h, dA.data(), G(b0 + 2), G(b0 + 3));
    layernorm_bwd(dA.data(), S.hin.data(), P(b0 + 0), S.mean1.data(), S.rstd1.data(), N, h,
                  dH.data(), G(b0 + 0), G(b0 + 1));
    for (size_t i = 0; i < dH.size(); ++i) dH[i] += dHm[i];  // residual
    Layer<T> empty;
    std::swap(st[l], empty);
  }
  // patch embed: the trainable source sends nothing upstream (Lemma 1 (i));
  // the patch gradient is computed only on request.
  linear_bwd(dH.data(), X, P(0), N, kpe, h, dX, G(0), G(1));
  return 0;
}

}  // namespace

// ------------------------------------------------------------------------
// C ABI
// ------------------------------------------------------------------------
extern "C" {

int64_t ref_param_count(const ref_cfg* c) {
  int64_t n = 0;
  for (auto& e : param_entries(*c)) n += e.rows * e.cols;
  return n;
}

int32_t ref_param_tensors(const ref_cfg* c) { return (int32_t)param_entries(*c).size(); }

int ref_param_info(const ref_cfg* c, int32_t i, char* name, int32_t cap, int64_t* offset,
                   int64_t* rows, int64_t* cols) {
  auto t = param_entries(*c);
  if (i < 0 || i >= (int32_t)t.size()) return -1;
  int64_t off = 0;
  for (int32_t j = 0; j < i; ++j) off += t[j].rows * t[j].cols;
  if (name && cap > 0) std::snprintf(name, (size_t)cap, "%s", t[i].name.c_str());
  *offset = off;
  *rows = t[i].rows;
  *cols = t[i].cols;
  return 0;
}

int ref_positions(const int32_t* thw, int32_t n_items, int32_t* py, int32_t* px) {
  return positions(thw, n_items, py, px);
}

int ref_encoder_f64(const ref_cfg* c, const double* w, const double* patches, const int32_t* cu,
                    int32_t n_seg, const int32_t* thw, int32_t n_items, int32_t trainable,
                    double* merged, const double* d_merged, double* d_w, double* d_patches) {
  return encoder<double>(*c, w, patches, cu, n_seg, thw, n_items, trainable, merged, d_merged,
                         d_w, d_patches);
}
int ref_encoder_f32(const ref_cfg* c, const float* w, const float* patches, const int32_t* cu,
                    int32_t n_seg, const int32_t* thw, int32_t n_items, int32_t trainable,
                    float* merged, const float* d_merged, float* d_w, float* d_patches) {
  return encoder<float>(*c, w, patches, cu, n_seg, thw, n_items, trainable, merged, d_merged,
                        d_w, d_patches);
}

void ref_linear_f64(const double* X, const double* W, const double* b, int64_t M, int64_t K,
                    int64_t N, double* Y) {
  linear(X, W, b, M, K, N, Y);
}
void ref_linear_bwd_f64(const double* dY, const double* X, const double* W, int64_t M, int64_t K,
                        int64_t N, double* dX, double* dW, double* db) {
  linear_bwd(dY, X, W, M, K, N, dX, dW, db);
}
void ref_layernorm_f64(const double* X, const double* g, const double* b, int64_t M, int64_t n,
                       double eps, double* Y, double* mean, double* rstd) {
  layernorm(X, g, b, M, n, eps, Y, mean, rstd);
}
void ref_layernorm_bwd_f64(const double* dY, const double* X, const double* g, const double* mean,
                           const double* rstd, int64_t M, int64_t n, double* dX, double* dg,
                           double* db) {
  layernorm_bwd(dY, X, g, mean, rstd, M, n, dX, dg, db);
}
void ref_gelu_f64(const double* u, int64_t n, double* y) {
  for (int64_t i = 0; i < n; ++i) y[i] = gelu(u[i]);
}
void ref_gelu_grad_f64(const double* u, int64_t n, double* y) {
  for (int64_t i = 0; i < n; ++i) y[i] = gelu_grad(u[i]);
}
void ref_rope2d_f64(double* x, int64_t N, int32_t heads, int32_t d, int64_t ld,
                    const int32_t* py, const int32_t* px, double theta, int32_t inverse) {
  rope2d(x, N, heads, d, ld, py, px, theta, inverse != 0);
}
void ref_attention_f64(const double* q, const double* k, const double* v, int64_t ld,
                       const int32_t* cu, int32_t n_seg, int32_t heads, int32_t d, double* o,
                       int64_t ldo, double* lse) {
  attention(q, k, v, ld, cu, n_seg, heads, d, o, ldo, lse);
}
void ref_attention_bwd_f64(const double* q, const double* k, const double* v, int64_t ld,
                           const double* o, const double* d_o, int64_t ldo, const double* lse,
                           const int32_t* cu, int32_t n_seg, int32_t heads, int32_t d, double* dq,
                           double* dk, double* dv, int64_t ldd) {
  attention_bwd(q, k, v, ld, o, d_o, ldo, lse, cu, n_seg, heads, d, dq, dk, dv, ldd);
}

static int check_idx(const int64_t* idx, int64_t n, int64_t n_rows) {
  Vec<unsigned char> seen((size_t)(n_rows > 0 ? n_rows : 0), 0);
  for (int64_t j = 0; j < n; ++j) {
    if (idx[j] < 0 || idx[j] >= n_rows || seen[idx[j]]) return -1;
    seen[idx[j]] = 1;
  }
  return 0;
}

// emb[idx[j]] <- merged[j]   (Replicated -> Sharded seam, forward Gather, local half)
int ref_merge_scatter(const void* merged, int64_t n_merged, int64_t row_bytes, const int64_t* idx,
                      void* emb, int64_t n_rows) {
  if (check_idx(idx, n_merged, n_rows)) return -1;
  for (int64_t j = 0; j < n_merged; ++j)
    std::memcpy((char*)emb + idx[j] * row_bytes, (const char*)merged + j * row_bytes,
                (size_t)row_bytes);
  return 0;
}

// d_merged[j] <- d_emb[idx[j]]   (the mirrored reverse Scatter^?, local half)
int ref_merge_gather(const void* d_emb, int64_t n_rows, int64_t row_bytes, const int64_t* idx,
                     int64_t n_merged, void* d_merged) {
  if (check_idx(idx, n_merged, n_rows)) return -1;
  for (int64_t j = 0; j < n_merged; ++j)
    std::memcpy((char*)d_merged + j * row_bytes, (const char*)d_emb + idx[j] * row_bytes,
                (size_t)row_bytes);
  return 0;
}

int32_t ref_num_threads(void) { return (int32_t)omp_get_max_threads(); }

}  // extern "C"
