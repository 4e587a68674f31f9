// Host planner for one micro-batch (see plan.h).
#include "plan.h"

#include <algorithm>
#include <cmath>
#include <numeric>

namespace mpipe {

namespace {
constexpr int kTile = 128;      // attention rows per work item (matches ATTN_TILE)
constexpr size_t kAlign = 256;

// Regions are 256-byte aligned and each is followed by at least kGuard bytes that no
// kernel writes, so a caller can fill a buffer with a canary pattern and find any write
// that strays out of its region (mpipe_encoder_regions lists the regions).
constexpr size_t kGuard = 256;

struct Arena {
  size_t top = 0;
  std::vector<Region>* log = nullptr;
  size_t take(size_t bytes) {
    const size_t off = (top + kAlign - 1) / kAlign * kAlign;
    top = off + bytes + kGuard;
    if (log && bytes) log->push_back({off, bytes});
    return off;
  }
};
}  // namespace

void derive_cfg(Cfg& c) {
  c.d = c.heads > 0 ? c.hidden / c.heads : 0;
  c.kpe = c.in_chans * c.tpatch * c.patch * c.patch;
  c.kp = (c.kpe + 63) / 64 * 64;
  c.esz = c.dtype == 1 ? 2 : 4;
}

std::string check_cfg(const Cfg& c) {
  if (c.in_chans <= 0 || c.patch <= 0 || c.tpatch <= 0 || c.layers < 0 || c.heads <= 0)
    return "sizes must be positive";
  if (c.dtype != 0 && c.dtype != 1) return "dtype must be MPIPE_F32 or MPIPE_BF16";
  if (c.merge != 2) return "only the 2x2 spatial merge is supported";
  if (c.hidden <= 0 || c.hidden % 64 || c.hidden > 2048) return "hidden must be a multiple of 64, <= 2048";
  if (c.hidden % c.heads) return "hidden must be divisible by heads";
  const int d = c.hidden / c.heads;
  if (d != 32 && d != 64 && d != 80) return "head_dim must be 32, 64 or 80";
  if (c.mlp <= 0 || c.mlp % 8) return "mlp must be a positive multiple of 8";
  if (c.llm <= 0 || c.llm % 8) return "llm_hidden must be a positive multiple of 8";
  if (!(c.eps > 0.f) || !(c.theta > 0.f)) return "ln_eps and rope_theta must be positive";
  return "";
}

std::vector<ParamEntry> param_table(const Cfg& c) {
  const int64_t h = c.hidden, m = c.mlp, H = c.llm, mh = 4 * h;
  std::vector<ParamEntry> t;
  int64_t off = 0;
  auto add = [&](const std::string& n, int64_t r, int64_t cc) {
    t.push_back({n, off, r, cc});
    off += r * cc;
  };
  add("pe.w", h, c.kpe);
  add("pe.b", h, 1);
  for (int l = 0; l < c.layers; ++l) {
    const std::string p = "blk" + std::to_string(l) + ".";
    add(p + "ln1.g", h, 1);
    add(p + "ln1.b", h, 1);
    add(p + "qkv.w", 3 * h, h);
    add(p + "qkv.b", 3 * h, 1);
    add(p + "proj.w", h, h);
    add(p + "proj.b", h, 1);
    add(p + "ln2.g", h, 1);
    add(p + "ln2.b", h, 1);
    add(p + "fc1.w", m, h);
    add(p + "fc1.b", m, 1);
    add(p + "fc2.w", h, m);
    add(p + "fc2.b", h, 1);
  }
  add("merger.ln.g", h, 1);
  add("merger.ln.b", h, 1);
  add("merger.fc1.w", mh, mh);
  add("merger.fc1.b", mh, 1);
  add("merger.fc2.w", H, mh);
  add("merger.fc2.b", H, 1);
  return t;
}

std::vector<float> rope_table(const Cfg& c, int positions) {
  const int q4 = c.d / 4;
  std::vector<float> t((size_t)positions * q4 * 2);
  for (int pp = 0; pp < positions; ++pp)
    for (int k = 0; k < q4; ++k) {
      const double a = pp * std::pow((double)c.theta, -4.0 * k / (double)c.d);
      t[((size_t)pp * q4 + k) * 2] = (float)std::cos(a);
      t[((size_t)pp * q4 + k) * 2 + 1] = (float)std::sin(a);
    }
  return t;
}

// At most four K splits: each split adds an fp32 partial of the whole output, written
// and read back by the reduction (ten splits of the qkv weight gradient moved 400 MB),
// and the weight-gradient GEMMs share the chip with the caller's stream anyway.
// Measured against a cap of 16 at the Qwen2-VL shape: 292.7 -> 290.4 ms/step with the
// side stream, 304.3 -> 293.5 ms/step without it.
constexpr int64_t kMaxSplitK = 4;

GemmSplit choose_split(int64_t M, int64_t N, int64_t K) {
  // Weight-gradient GEMMs have few output tiles and a long K (tokens): split K so
  // the grid fills whole rounds of 256 CUs as far as the cap allows (each split keeps
  // >= 1024 rows of K).
  // Tile size follows the kernel the GEMM dispatches to (256 when M >= 512, N >= 256).
  const bool big = M >= 512 && N >= 256;
  const int64_t t = big ? 256 : 128;
  const int64_t tiles = ((M + t - 1) / t) * ((N + t - 1) / t);
  const int64_t per_round = big ? 256 : 512;
  int64_t best = 1;
  double best_eff = 0.0;
  for (int64_t s = 1; s <= kMaxSplitK; ++s) {
    if (s > 1 && K / s < 1024) break;
    const int64_t blocks = tiles * s;
    const int64_t rounds = (blocks + per_round - 1) / per_round;
    const double eff = (double)blocks / (double)(rounds * per_round);
    if (eff > best_eff + 1e-9) {
      best_eff = eff;
      best = s;
    }
    if (eff >= 0.9) break;
  }
  GemmSplit g;
  if (best <= 1) {
    g.splits = 1;
    g.kps = 0;
    return g;
  }
  int64_t kps = (K + best - 1) / best;
  kps = (kps + 63) / 64 * 64;
  g.kps = (int)kps;
  g.splits = (int)((K + kps - 1) / kps);
  if (g.splits <= 1) {
    g.splits = 1;
    g.kps = 0;
  }
  return g;
}

int build_plan(const Cfg& c, const int32_t* cu, int n_seg, const int32_t* thw, int n_items,
               int mode, Plan& p, std::string& err) {
  p = Plan();
  if (mode != MODE_FROZEN && mode != MODE_TRAINED && mode != MODE_MERGER) {
    err = "trainable must be 0 (frozen), 1 (trained) or 2 (merger only)";
    return -1;
  }
  p.mode = mode;
  p.trainable = mode == MODE_TRAINED;
  if (n_items < 0 || n_seg < 0) {
    err = "negative item or segment count";
    return -1;
  }
  if (n_items > 0 && (!thw || !cu)) {
    err = "grid_thw and cu_seqlens are required";
    return -1;
  }
  // items
  std::vector<int64_t> start(n_items + 1, 0);
  int64_t N = 0, Tm = 0;
  for (int i = 0; i < n_items; ++i) {
    const int t = thw[3 * i], gh = thw[3 * i + 1], gw = thw[3 * i + 2];
    if (t <= 0 || gh <= 0 || gw <= 0) {
      err = "grid_thw entries must be positive (item " + std::to_string(i) + ")";
      return -2;
    }
    if (gh % 2 || gw % 2) {
      err = "grid height and width must be even for the 2x2 merge (item " + std::to_string(i) + ")";
      return -2;
    }
    // a row's position is packed as y << 16 | x into 32 bits: both sides stay below 2^15
    if (gh > kMaxGridSide || gw > kMaxGridSide) {
      err = "grid height and width must be at most " + std::to_string(kMaxGridSide) +
            " patches (item " + std::to_string(i) + ")";
      return -2;
    }
    start[i] = N;
    N += (int64_t)t * gh * gw;
    Tm += (int64_t)t * (gh / 2) * (gw / 2);
  }
  start[n_items] = N;
  if (N > (int64_t)INT32_MAX / 4) {
    err = "too many patches";
    return -2;
  }
  p.N = N;
  p.Tm = Tm;
  p.n_items = n_items;
  p.n_seg = n_seg;
  if (n_items == 0) {
    if (n_seg != 0 && !(cu && cu[n_seg] == 0)) {
      err = "segments given for an empty micro-batch";
      return -2;
    }
    p.n_seg = 0;
    return 0;
  }
  if (n_seg <= 0 || cu[0] != 0 || cu[n_seg] != N) {
    err = "cu_seqlens must start at 0 and end at the packed row count " + std::to_string(N);
    return -2;
  }
  int it = 0;
  for (int s = 0; s < n_seg; ++s) {
    if (cu[s + 1] <= cu[s]) {
      err = "cu_seqlens must be strictly increasing (segment " + std::to_string(s) + ")";
      return -2;
    }
    while (it < n_items && cu[s] >= start[it + 1]) ++it;
    if (it >= n_items || cu[s + 1] > start[it + 1]) {
      err = "segment " + std::to_string(s) + " crosses an item boundary";
      return -2;
    }
    const int64_t slice = (int64_t)thw[3 * it + 1] * thw[3 * it + 2];
    if ((cu[s] - start[it]) % slice || (cu[s + 1] - start[it]) % slice) {
      err = "segment " + std::to_string(s) + " does not start/end on a temporal slice";
      return -2;
    }
  }

  // positions (inverse of the window-major row order)
  p.pos.resize(N);
  for (int i = 0; i < n_items; ++i) {
    const int gh = thw[3 * i + 1], gw = thw[3 * i + 2];
    const int64_t n = start[i + 1] - start[i];
    const int wpr = gw / 2, wpc = gh / 2;
    for (int64_t r = 0; r < n; ++r) {
      const int64_t w = r >> 2;
      const int dh = (int)((r >> 1) & 1), dw = (int)(r & 1);
      const int wb = (int)(w % wpr);
      const int hb = (int)((w / wpr) % wpc);
      p.pos[start[i] + r] = ((2 * hb + dh) << 16) | (2 * wb + dw);
    }
  }
  // attention work lists: tiles of 128 rows, longest segments first
  std::vector<int> order(n_seg);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
    return (cu[a + 1] - cu[a]) > (cu[b + 1] - cu[b]);
  });
  for (int s : order) {
    const int s0 = cu[s], s1 = cu[s + 1];
    p.sum_len2 += (int64_t)(s1 - s0) * (s1 - s0);
    for (int r = s0; r < s1; r += kTile) {
      p.q_work.insert(p.q_work.end(), {r, s0, s1, 0});
      p.k_work.insert(p.k_work.end(), {r, s0, s1, 0});
    }
  }
  int max_side = 1;
  for (int i = 0; i < n_items; ++i) max_side = std::max({max_side, thw[3 * i + 1], thw[3 * i + 2]});
  p.rope_tab = rope_table(c, max_side);
  const int q4 = c.d / 4;

  // ---- workspace ----
  const int64_t h = c.hidden, m = c.mlp, H = c.llm, E = c.esz, nh = c.heads;
  Arena ws;
  p.ws_pos = ws.take(sizeof(int32_t) * N);
  p.ws_qwork = ws.take(sizeof(int32_t) * p.q_work.size());
  p.ws_kwork = ws.take(sizeof(int32_t) * p.k_work.size());
  p.ws_rope = ws.take(sizeof(float) * p.rope_tab.size());
  (void)q4;
  // uploaded by one copy (the guards between them included): one region
  p.meta_bytes = p.ws_rope + sizeof(float) * p.rope_tab.size();
  p.ws_regions.push_back({0, p.meta_bytes});
  ws.log = &p.ws_regions;
  if (c.kp != c.kpe) {
    p.ws_xp = ws.take((size_t)N * c.kp * E);
    p.ws_wpe = ws.take((size_t)h * c.kp * E);
  }
  // The forward multiplies by transposed weights ([in][out], so the GEMM's weight
  // operand is K-major); they are transposed one layer (or the merger, or the patch
  // embedding) at a time into this region.
  p.ws_wt = ws.take((size_t)E * std::max({3 * h * h + h * h + 2 * h * m, 16 * h * h + 4 * h * H,
                                          (int64_t)c.kp * h}));
  auto act_set = [&](Arena& a, bool keep_u, bool share_h) {
    ActSet s{};
    s.hin = a.take((size_t)N * h * 4);
    s.hmid = share_h ? s.hin : a.take((size_t)N * h * 4);
    s.hout = share_h ? s.hin : 0;  // filled by the caller when not shared
    s.a = a.take((size_t)N * h * E);
    s.mean1 = a.take((size_t)N * 4);
    s.rstd1 = a.take((size_t)N * 4);
    s.qkv = a.take((size_t)N * 3 * h * E);
    s.o = a.take((size_t)N * h * E);
    s.lse = a.take((size_t)N * nh * 4);
    s.b = a.take((size_t)N * h * E);
    s.mean2 = a.take((size_t)N * 4);
    s.rstd2 = a.take((size_t)N * 4);
    s.u = keep_u ? a.take((size_t)N * m * E) : 0;
    s.g = a.take((size_t)N * m * E);
    return s;
  };
  auto merger_set = [&](Arena& a, size_t hfin, bool keep_u) {
    MergerSet s{};
    s.hfin = hfin;
    s.z = a.take((size_t)N * h * E);
    s.meanz = a.take((size_t)N * 4);
    s.rstdz = a.take((size_t)N * 4);
    s.um = keep_u ? a.take((size_t)Tm * 4 * h * E) : 0;
    s.gm = a.take((size_t)Tm * 4 * h * E);
    return s;
  };
  if (mode != MODE_TRAINED) {   // blocks without a tape: activations shared by all layers
    p.ws_act = act_set(ws, false, true);
    p.ws_mrg = merger_set(ws, p.ws_act.hin, false);
  }
  if (mode != MODE_FROZEN) {
    // backward scratch
    p.ws_dh = ws.take((size_t)N * h * 4);
    p.ws_dht = ws.take((size_t)N * h * E);
    p.ws_dhm = ws.take((size_t)N * h * 4);
    p.ws_dhmt = ws.take((size_t)N * h * E);
    p.ws_dxln = ws.take((size_t)N * h * E);   // LayerNorm input gradient, activation dtype
    p.ws_du = ws.take((size_t)N * std::max<int64_t>(m, h) * E);
    p.ws_do = ws.take((size_t)N * h * E);
    p.ws_delta = ws.take((size_t)N * nh * 4);
    p.ws_dqkv = ws.take((size_t)N * 3 * h * E);
    p.ws_dqkv2 = mode == MODE_TRAINED ? ws.take((size_t)N * 3 * h * E) : 0;
    const int64_t widest = std::max({3 * h, m, 4 * h, H, (int64_t)c.kpe});
    // LayerNorm-backward partials (two buffers of three sets: gain, shift and the column
    // sums of the residual-stream gradient, h columns each) and bias column-sum partials
    // (own region: the backward runs the remaining column sums on its side stream)
    p.ws_part = ws.take((size_t)kPartialRowsMax * 6 * h * 4);
    p.ws_cpart = ws.take((size_t)kPartialRowsMax * widest * 4);
    // GELU-backward column sums per 64-row band, written by the input-gradient GEMM of fc1
    p.ws_gpart = ws.take((size_t)((std::max(N, Tm) + 63) / 64) * std::max(m, 4 * h) * 4);
    // largest split-K partial over the weight-gradient GEMMs
    size_t dw = 0;
    auto need = [&](int64_t M_, int64_t N_, int64_t K_) {
      GemmSplit g = choose_split(M_, N_, K_);
      if (g.splits > 1) dw = std::max(dw, (size_t)g.splits * M_ * N_ * 4);
    };
    need(h, c.kpe, N);
    need(3 * h, h, N);
    need(h, h, N);
    need(m, h, N);
    need(h, m, N);
    need(4 * h, 4 * h, Tm);
    need(H, 4 * h, Tm);
    p.ws_dwpart = dw ? ws.take(dw) : 0;
  }
  p.ws_bytes = ws.top;

  // ---- tape ----
  if (mode == MODE_MERGER) {   // the merger's inputs only: the blocks run no backward
    Arena tp;
    tp.log = &p.tape_regions;
    p.tape_mrg = merger_set(tp, tp.take((size_t)N * h * 4), true);
    p.tape_bytes = tp.top;
  } else if (mode == MODE_TRAINED) {
    Arena tp;
    tp.log = &p.tape_regions;
    p.tape_act.resize(c.layers);
    size_t h_in = tp.take((size_t)N * h * 4);
    for (int l = 0; l < c.layers; ++l) {
      ActSet s{};
      s.hin = h_in;
      s.hmid = tp.take((size_t)N * h * 4);
      s.hout = tp.take((size_t)N * h * 4);
      s.a = tp.take((size_t)N * h * E);
      s.mean1 = tp.take((size_t)N * 4);
      s.rstd1 = tp.take((size_t)N * 4);
      s.qkv = tp.take((size_t)N * 3 * h * E);
      s.o = tp.take((size_t)N * h * E);
      s.lse = tp.take((size_t)N * nh * 4);
      s.b = tp.take((size_t)N * h * E);
      s.mean2 = tp.take((size_t)N * 4);
      s.rstd2 = tp.take((size_t)N * 4);
      s.u = tp.take((size_t)N * m * E);
      s.g = tp.take((size_t)N * m * E);
      p.tape_act[l] = s;
      h_in = s.hout;
    }
    p.tape_mrg = merger_set(tp, h_in, true);
    p.tape_bytes = tp.top;
  }
  return 0;
}

}  // namespace mpipe
