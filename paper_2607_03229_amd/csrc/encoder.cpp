// C ABI of libmpipe: handle, metadata validation, and the launch sequence of the
// encoder forward / backward on the caller's stream.  See include/mpipe.h.
#include "../../include/mpipe.h"
#include "../../include/mpipe_ops.h"
#include "../../include/mpipe_sched.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <tuple>
#include <map>
#include <string>
#include <vector>

#include "internal.h"
#include "plan.h"

using namespace mpipe;

namespace {
thread_local std::string g_err;

mpipe_status fail(mpipe_status s, const std::string& m) {
  g_err = m;
  return s;
}
}  // namespace

namespace mpipe {
mpipe_status set_error(mpipe_status s, const std::string& m) { return fail(s, m); }
}  // namespace mpipe

namespace {

struct Rec {
  std::string cls;
  hipEvent_t a, b;
  double flops;
  bool side;   // launched on the handle's side stream (overlaps the caller's stream)
};
}  // namespace

struct mpipe_encoder {
  Cfg cfg;
  std::vector<ParamEntry> params;
  void* staging = nullptr;  // pinned host memory for the per-call metadata upload
  size_t staging_cap = 0;
  hipEvent_t staging_ev = nullptr;
  bool staging_pending = false;
  bool prof = false;
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  // Weight-gradient side stream of the backward (default priority) and its sync events:
  // 0 fork (caller -> side), 1..7 buffer-free signals (side -> caller), 8 join.
  bool side_on = true;
  hipStream_t side = nullptr;
  int side_dev = -1;
  hipEvent_t sync[9] = {};

  hipEvent_t event() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};

namespace {

// Bracket one launch with events when profiling is on.
template <class F>
hipError_t run(mpipe_encoder* e, hipStream_t s, const char* cls, double flops, F&& f) {
  if (!e || !e->prof) return f();
  hipEvent_t a = e->event(), b = e->event();
  const bool ra = a && hipEventRecord(a, s) == hipSuccess;
  hipError_t r = f();
  const bool rb = b && hipEventRecord(b, s) == hipSuccess;
  if (ra && rb) {
    e->recs.push_back({cls, a, b, flops, e->side != nullptr && s == e->side});
  } else {   // an event that could not be recorded times nothing: give both back
    if (a) e->pool.push_back(a);
    if (b) e->pool.push_back(b);
  }
  return r;
}

const char* gemm_name(int layout, int epi) {
  static const char* L[] = {"NT", "NN", "TN"};
  static const char* E[] = {"store", "gelu", "resid", "gelubwd", "f32", "storerope"};
  static std::map<int, std::string> names;
  const int key = layout * 8 + epi;
  auto it = names.find(key);
  if (it == names.end())
    it = names.emplace(key, std::string("gemm_") + L[layout] + "_" + E[epi]).first;
  return it->second.c_str();
}

#define MP_CHECK(expr)                                                              \
  do {                                                                              \
    hipError_t _e = (expr);                                                         \
    if (_e != hipSuccess)                                                           \
      return fail(MPIPE_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(_e)); \
  } while (0)

Cfg to_cfg(const mpipe_encoder_cfg* c) {
  Cfg o;
  o.in_chans = c->in_chans;
  o.patch = c->patch;
  o.tpatch = c->temporal_patch;
  o.hidden = c->hidden;
  o.layers = c->layers;
  o.heads = c->heads;
  o.mlp = c->mlp;
  o.merge = c->merge;
  o.llm = c->llm_hidden;
  o.dtype = c->dtype;
  o.eps = c->ln_eps;
  o.theta = c->rope_theta;
  derive_cfg(o);
  return o;
}

struct Ctx {
  mpipe_encoder* e;
  const Cfg& c;
  const Plan& P;
  hipStream_t s;   // the caller's stream (critical path)
  const char* w;   // weights (device)
  char* ws;        // workspace (device)
  int dt;
  int64_t E;
  hipStream_t s2 = nullptr;   // weight-gradient work (== s when there is no side stream)
  const char* W(int i) const { return w + e->params[i].off * E; }
  float* grad(float* dw, int i) const { return dw + e->params[i].off; }
};

mpipe_status gemm_on(Ctx& x, hipStream_t st, int layout, int epi, GemmArgs a) {
  const double fl = 2.0 * a.M * a.N * (double)a.K;
  MP_CHECK(run(x.e, st, gemm_name(layout, epi), fl, [&] { return gemm(x.dt, layout, epi, a, st); }));
  return MPIPE_OK;
}
mpipe_status gemm_call(Ctx& x, int layout, int epi, GemmArgs a) {
  return gemm_on(x, x.s, layout, epi, a);
}

GemmArgs ga(const void* A, int64_t lda, const void* B, int64_t ldb, int64_t M, int64_t N,
            int64_t K, void* C, int64_t ldc) {
  GemmArgs a;
  a.A = A;
  a.lda = lda;
  a.B = B;
  a.ldb = ldb;
  a.M = (int)M;
  a.N = (int)N;
  a.K = (int)K;
  a.C = C;
  a.ldc = ldc;
  return a;
}

// dW[M][N] (+)= sum_k A[k][m] B[k][n]  (weight gradient, K = tokens)
mpipe_status dw_gemm(Ctx& x, const void* A, int64_t lda, const void* B, int64_t ldb, int64_t M,
                     int64_t N, int64_t K, float* out, int64_t ldo) {
  GemmSplit sp = choose_split(M, N, K);
  GemmArgs a = ga(A, lda, B, ldb, M, N, K, nullptr, 0);
  if (sp.splits <= 1) {
    a.C = out;
    a.ldc = ldo;
    a.beta = 1;
    return gemm_on(x, x.s2, GEMM_TN, EPI_F32, a);
  }
  float* part = reinterpret_cast<float*>(x.ws + x.P.ws_dwpart);
  a.C = part;
  a.ldc = N;
  a.kps = sp.kps;
  a.split_stride = M * N;
  mpipe_status st = gemm_on(x, x.s2, GEMM_TN, EPI_F32, a);
  if (st) return st;
  MP_CHECK(run(x.e, x.s2, "splitk_reduce", 0,
               [&] { return splitk_reduce(part, sp.splits, M, N, out, ldo, x.s2); }));
  return MPIPE_OK;
}

// out += the column sums that the fc1 input-gradient GEMM wrote per 64-row band
mpipe_status band_reduce(Ctx& x, int64_t rows, int n, float* out) {
  float* part = reinterpret_cast<float*>(x.ws + x.P.ws_gpart);
  MP_CHECK(run(x.e, x.s2, "colsum", 0,
               [&] { return partials_reduce(part, out, (rows + 63) / 64, n, x.s2); }));
  return MPIPE_OK;
}

mpipe_status colsum(Ctx& x, int dtype_in, const void* X, int64_t ld, int64_t rows, int n,
                    float* out) {
  float* part = reinterpret_cast<float*>(x.ws + x.P.ws_cpart);
  MP_CHECK(run(x.e, x.s2, "colsum", 0,
               [&] { return colsum_accumulate(dtype_in, X, ld, rows, n, part, out, x.s2); }));
  return MPIPE_OK;
}

// Stream hand-offs of the backward: fork makes everything enqueued on the caller's stream
// so far visible to the side stream; release(i) marks on the side stream that the buffers
// its gradient work reads are free again, and acquire(i) makes the caller's stream wait for
// that before it overwrites them.
struct SideSync {
  Ctx& x;
  bool on;
  bool recorded[9] = {};
  hipError_t fork() {
    if (!on) return hipSuccess;
    hipError_t r = hipEventRecord(x.e->sync[0], x.s);
    return r != hipSuccess ? r : hipStreamWaitEvent(x.s2, x.e->sync[0], 0);
  }
  hipError_t release(int i) {
    if (!on) return hipSuccess;
    recorded[i] = true;
    return hipEventRecord(x.e->sync[i], x.s2);
  }
  hipError_t acquire(int i) {
    if (!on || !recorded[i]) return hipSuccess;
    return hipStreamWaitEvent(x.s, x.e->sync[i], 0);
  }
  hipError_t join() {
    if (!on) return hipSuccess;
    hipError_t r = hipEventRecord(x.e->sync[8], x.s2);
    return r != hipSuccess ? r : hipStreamWaitEvent(x.s, x.e->sync[8], 0);
  }
};
enum { FREE_DU = 1, FREE_DH = 2, FREE_DHM = 3, FREE_DQKV = 4, FREE_LNP0 = 5, FREE_LNP1 = 6,
       FREE_DQKV1 = 7 };

// Creates the side stream and its events on the current device (once per device).
hipError_t ensure_side(mpipe_encoder* e) {
  int dev = 0;
  hipError_t r = hipGetDevice(&dev);
  if (r != hipSuccess) return r;
  if (e->side && e->side_dev == dev) return hipSuccess;
  if (e->side) {   // the handle moved to another device: rebuild its side stream there
    (void)hipStreamSynchronize(e->side);
    (void)hipStreamDestroy(e->side);
    for (auto& ev : e->sync) {
      if (ev) (void)hipEventDestroy(ev);
      ev = nullptr;
    }
    e->side = nullptr;
  }
  r = hipStreamCreateWithFlags(&e->side, hipStreamNonBlocking);
  if (r != hipSuccess) {
    e->side = nullptr;
    return r;
  }
  for (auto& ev : e->sync) {
    r = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (r != hipSuccess) return r;
  }
  e->side_dev = dev;
  return hipSuccess;
}

mpipe_status upload_meta(mpipe_encoder* e, const Plan& P, char* ws, hipStream_t s) {
  const size_t bytes = P.meta_bytes;
  if (bytes == 0) return MPIPE_OK;
  if (e->staging_pending) {
    MP_CHECK(hipEventSynchronize(e->staging_ev));
    e->staging_pending = false;
  }
  if (bytes > e->staging_cap) {
    if (e->staging) MP_CHECK(hipHostFree(e->staging));
    e->staging = nullptr;
    e->staging_cap = 0;
    MP_CHECK(hipHostMalloc(&e->staging, bytes, hipHostMallocDefault));
    e->staging_cap = bytes;
  }
  char* st = reinterpret_cast<char*>(e->staging);
  std::memcpy(st + P.ws_pos, P.pos.data(), P.pos.size() * sizeof(int32_t));
  std::memcpy(st + P.ws_qwork, P.q_work.data(), P.q_work.size() * sizeof(int32_t));
  std::memcpy(st + P.ws_kwork, P.k_work.data(), P.k_work.size() * sizeof(int32_t));
  std::memcpy(st + P.ws_rope, P.rope_tab.data(), P.rope_tab.size() * sizeof(float));
  MP_CHECK(hipMemcpyAsync(ws, st, bytes, hipMemcpyHostToDevice, s));
  if (!e->staging_ev) MP_CHECK(hipEventCreateWithFlags(&e->staging_ev, hipEventDisableTiming));
  MP_CHECK(hipEventRecord(e->staging_ev, s));
  e->staging_pending = true;
  return MPIPE_OK;
}

AttnArgs attn_args(Ctx& x, const char* qkv, bool k_tiles) {
  const Cfg& c = x.c;
  AttnArgs a;
  a.q = qkv;
  a.k = qkv + (int64_t)c.hidden * x.E;
  a.v = qkv + 2 * (int64_t)c.hidden * x.E;
  a.ld = 3 * c.hidden;
  a.heads = c.heads;
  a.N = x.P.N;
  a.scale = 1.0f / std::sqrt((float)c.d);
  a.work = reinterpret_cast<const int4*>(x.ws + (k_tiles ? x.P.ws_kwork : x.P.ws_qwork));
  a.n_work = (int)((k_tiles ? x.P.k_work.size() : x.P.q_work.size()) / 4);
  return a;
}

// pointers of the padded patch matrix and patch-embedding weight
void pe_operands(Ctx& x, const void* patches, const void*& Xp, const void*& Wpe, int64_t& ld) {
  const Cfg& c = x.c;
  if (c.kp != c.kpe) {
    Xp = x.ws + x.P.ws_xp;
    Wpe = x.ws + x.P.ws_wpe;
    ld = c.kp;
  } else {
    Xp = patches;
    Wpe = x.W(P_PE_W);
    ld = c.kpe;
  }
}

mpipe_status pad_pe(Ctx& x, const void* patches) {
  const Cfg& c = x.c;
  if (c.kp == c.kpe) return MPIPE_OK;
  MP_CHECK(run(x.e, x.s, "pad", 0, [&] { return pad_cols(x.dt, patches, x.P.N, c.kpe, x.ws + x.P.ws_xp, c.kp, x.s); }));
  MP_CHECK(run(x.e, x.s, "pad", 0, [&] { return pad_cols(x.dt, x.W(P_PE_W), c.hidden, c.kpe, x.ws + x.P.ws_wpe, c.kp, x.s); }));
  return MPIPE_OK;
}

// Transposed copies of the [out][in] weights the next GEMMs multiply by, back to back in
// the workspace: wt[i] = W_i^T ([in][out], row stride out), so that every forward GEMM
// reads its weight operand K-major (whole 128-byte lines per DMA row).
// qk_rows > 0: the first weight is the qkv weight, whose first qk_rows output rows (the q
// and k blocks) are taken pair-interleaved within each head, so that its product comes
// out in the layout the fused rotary epilogue and the attention kernels work on.
mpipe_status weights_t(Ctx& x, int n, const void* const* W, const int64_t* out_f,
                       const int64_t* in_f, const int64_t* ld, const void** wt,
                       int qk_rows = 0) {
  TJob jobs[kMaxTJobs];
  char* dst = x.ws + x.P.ws_wt;
  for (int i = 0; i < n; ++i) {
    jobs[i].src = W[i];
    jobs[i].lds = ld[i];
    jobs[i].dst = dst;
    jobs[i].ldd = out_f[i];
    jobs[i].rows = (int)out_f[i];
    jobs[i].cols = (int)in_f[i];
    if (i == 0 && qk_rows > 0) {
      jobs[i].perm_rows = qk_rows;
      jobs[i].perm_d = x.c.d;
    }
    wt[i] = dst;
    dst += out_f[i] * in_f[i] * x.E;
  }
  MP_CHECK(run(x.e, x.s, "transpose", 0, [&] { return transpose_batch(x.dt, jobs, n, x.s); }));
  return MPIPE_OK;
}

#define MP_RET(expr)                  \
  do {                                \
    mpipe_status _s = (expr);         \
    if (_s != MPIPE_OK) return _s;    \
  } while (0)

mpipe_status forward(Ctx& x, const void* patches, void* merged, char* tape) {
  const Cfg& c = x.c;
  const Plan& P = x.P;
  const int64_t N = P.N, h = c.hidden, m = c.mlp, H = c.llm, E = x.E;
  const bool tr = P.mode == MODE_TRAINED;     // every layer records its activations
  const bool mt = P.mode != MODE_FROZEN;      // the merger records its inputs
  char* base = tr ? tape : x.ws;
  char* mbase = mt ? tape : x.ws;
  auto act = [&](int l) -> const ActSet& { return tr ? P.tape_act[l] : P.ws_act; };
  const MergerSet& MS = mt ? P.tape_mrg : P.ws_mrg;
  const int32_t* pos = reinterpret_cast<const int32_t*>(x.ws + P.ws_pos);
  const float* freq = reinterpret_cast<const float*>(x.ws + P.ws_rope);

  MP_RET(pad_pe(x, patches));
  const void *Xp, *Wpe;
  int64_t ldx;
  pe_operands(x, patches, Xp, Wpe, ldx);
  char* h0 = c.layers > 0 ? base + act(0).hin : mbase + MS.hfin;
  {
    const void* wt[1];
    const int64_t of[1] = {h}, inf[1] = {c.kp}, ld[1] = {ldx};
    MP_RET(weights_t(x, 1, &Wpe, of, inf, ld, wt));
    GemmArgs a = ga(Xp, ldx, wt[0], h, N, h, c.kp, h0, h);
    a.bias = x.W(P_PE_B);
    MP_RET(gemm_call(x, GEMM_NN, EPI_RESID, a));
  }
  for (int l = 0; l < c.layers; ++l) {
    const ActSet& S = act(l);
    float* hin = reinterpret_cast<float*>(base + S.hin);
    float* hmid = reinterpret_cast<float*>(base + S.hmid);
    // (with only the merger trainable, the last layer writes the merger's tape input)
    float* hout = reinterpret_cast<float*>(
        P.mode == MODE_MERGER && l == c.layers - 1 ? mbase + MS.hfin
                                                   : base + (tr ? S.hout : S.hin));
    char* A = base + S.a;
    char* qkv = base + S.qkv;
    char* O = base + S.o;
    char* B = base + S.b;
    char* G = base + S.g;
    // W^T of qkv, proj, fc1, fc2
    const void* wt[4];
    {
      const void* W[4] = {x.W(blk_param(c, l, B_QKVW)), x.W(blk_param(c, l, B_PROJW)),
                          x.W(blk_param(c, l, B_FC1W)), x.W(blk_param(c, l, B_FC2W))};
      const int64_t of[4] = {3 * h, h, m, h}, inf[4] = {h, h, h, m};
      MP_RET(weights_t(x, 4, W, of, inf, inf, wt, (int)(2 * h)));
    }
    MP_CHECK(run(x.e, x.s, "layernorm", 0, [&] {
      return layernorm_fwd(x.dt, hin, h, N, (int)h, x.W(blk_param(c, l, B_LN1G)),
                           x.W(blk_param(c, l, B_LN1B)), c.eps, A, h,
                           reinterpret_cast<float*>(base + S.mean1),
                           reinterpret_cast<float*>(base + S.rstd1), x.s);
    }));
    {
      // q, k come out pair-interleaved per head with the 2D rotary position applied in
      // the epilogue; v in plain order
      GemmArgs a = ga(A, h, wt[0], 3 * h, N, 3 * h, h, qkv, 3 * h);
      a.bias = x.W(blk_param(c, l, B_QKVB));
      a.rope_pos = pos;
      a.rope_tab = reinterpret_cast<const float2*>(freq);
      a.rope_d = c.d;
      a.rope_cols = (int)(2 * h);
      MP_RET(gemm_call(x, GEMM_NN, EPI_STORE_ROPE, a));
    }
    {
      AttnArgs a = attn_args(x, qkv, false);
      a.out = O;
      a.ldo = h;
      a.lse = reinterpret_cast<float*>(base + S.lse);
      const double fl = 4.0 * c.heads * c.d * (double)P.sum_len2;
      MP_CHECK(run(x.e, x.s, "attn_fwd", fl, [&] { return attention_fwd(x.dt, c.d, a, x.s); }));
    }
    {
      GemmArgs a = ga(O, h, wt[1], h, N, h, h, hmid, h);
      a.bias = x.W(blk_param(c, l, B_PROJB));
      a.aux = hin;
      a.ld_aux = h;
      MP_RET(gemm_call(x, GEMM_NN, EPI_RESID, a));
    }
    MP_CHECK(run(x.e, x.s, "layernorm", 0, [&] {
      return layernorm_fwd(x.dt, hmid, h, N, (int)h, x.W(blk_param(c, l, B_LN2G)),
                           x.W(blk_param(c, l, B_LN2B)), c.eps, B, h,
                           reinterpret_cast<float*>(base + S.mean2),
                           reinterpret_cast<float*>(base + S.rstd2), x.s);
    }));
    {
      GemmArgs a = ga(B, h, wt[2], m, N, m, h, G, m);
      a.bias = x.W(blk_param(c, l, B_FC1B));
      a.C2 = tr ? base + S.u : nullptr;
      a.ldc2 = m;
      MP_RET(gemm_call(x, GEMM_NN, EPI_GELU, a));
    }
    {
      GemmArgs a = ga(G, m, wt[3], h, N, h, m, hout, h);
      a.bias = x.W(blk_param(c, l, B_FC2B));
      a.aux = hmid;
      a.ld_aux = h;
      MP_RET(gemm_call(x, GEMM_NN, EPI_RESID, a));
    }
  }
  // 2x2 merger: LN, the four window rows side by side ([Tm][4h] view), fc1+GELU, fc2
  char* Z = mbase + MS.z;
  char* Gm = mbase + MS.gm;
  const void* wtm[2];
  {
    const void* W[2] = {x.W(merger_param(c, M_FC1W)), x.W(merger_param(c, M_FC2W))};
    const int64_t of[2] = {4 * h, H}, inf[2] = {4 * h, 4 * h};
    MP_RET(weights_t(x, 2, W, of, inf, inf, wtm));
  }
  MP_CHECK(run(x.e, x.s, "layernorm", 0, [&] {
    return layernorm_fwd(x.dt, reinterpret_cast<float*>(mbase + MS.hfin), h, N, (int)h,
                         x.W(merger_param(c, M_LNG)), x.W(merger_param(c, M_LNB)), c.eps, Z, h,
                         reinterpret_cast<float*>(mbase + MS.meanz),
                         reinterpret_cast<float*>(mbase + MS.rstdz), x.s);
  }));
  {
    GemmArgs a = ga(Z, 4 * h, wtm[0], 4 * h, P.Tm, 4 * h, 4 * h, Gm, 4 * h);
    a.bias = x.W(merger_param(c, M_FC1B));
    a.C2 = mt ? mbase + MS.um : nullptr;
    a.ldc2 = 4 * h;
    MP_RET(gemm_call(x, GEMM_NN, EPI_GELU, a));
  }
  {
    GemmArgs a = ga(Gm, 4 * h, wtm[1], H, P.Tm, H, 4 * h, merged, H);
    a.bias = x.W(merger_param(c, M_FC2B));
    MP_RET(gemm_call(x, GEMM_NN, EPI_STORE, a));
  }
  (void)E;
  return MPIPE_OK;
}

mpipe_status backward(Ctx& x, const void* patches, const char* tape, const void* dM, float* dw,
                      void* d_patches) {
  const Cfg& c = x.c;
  const Plan& P = x.P;
  const int64_t N = P.N, Tm = P.Tm, h = c.hidden, m = c.mlp, H = c.llm;
  const char* base = tape;
  const MergerSet& MS = P.tape_mrg;
  const int32_t* pos = reinterpret_cast<const int32_t*>(x.ws + P.ws_pos);
  const float* freq = reinterpret_cast<const float*>(x.ws + P.ws_rope);
  float* dh = reinterpret_cast<float*>(x.ws + P.ws_dh);
  char* dht = x.ws + P.ws_dht;
  float* dhm = reinterpret_cast<float*>(x.ws + P.ws_dhm);
  char* dhmt = x.ws + P.ws_dhmt;
  // input gradient of each LayerNorm: bf16 for a bf16 encoder (the GEMM stores it with the
  // plain epilogue), fp32 for the fp32 one
  void* dxln = x.ws + P.ws_dxln;
  const int epi_dxln = x.dt == DT_BF16 ? EPI_STORE : EPI_F32;
  char* du = x.ws + P.ws_du;
  char* dO = x.ws + P.ws_do;
  float* delta = reinterpret_cast<float*>(x.ws + P.ws_delta);
  char* const dqkvb[2] = {x.ws + P.ws_dqkv, x.ws + P.ws_dqkv2};
  // LayerNorm-backward partials: two buffers of three sets (gain, shift, and the column sums
  // of the residual-stream gradient it writes, which is the next bias gradient), each
  // kPartialRowsMax x h floats
  float* part = reinterpret_cast<float*>(x.ws + P.ws_part);
  const int64_t ln_set = kPartialRowsMax * h;

  // Only the merger trainable: it is the trainable source (Lemma 1 applied to the
  // encoder's parts), so its backward ends with its own LayerNorm's affine gradients.
  const bool merger_only = P.mode == MODE_MERGER;
  const void *Xp = nullptr, *Wpe = nullptr;
  int64_t ldx = 0;
  if (!merger_only) {
    MP_RET(pad_pe(x, patches));
    pe_operands(x, patches, Xp, Wpe, ldx);
  }

  // Weight and bias gradients feed nothing else in the backward: they run on the side
  // stream (x.s2), which forks off after the gradient buffers they read are produced (in a
  // block, after the LayerNorm backward that follows them); the caller's stream waits for
  // a buffer's side readers only before it overwrites that buffer.
  SideSync ss{x, x.s2 != x.s};
  // LayerNorm backward of dxln on the caller's stream; its partial sums are reduced into
  // the gain, shift and bias gradients on the side stream (nothing in the backward reads
  // them).  The partial buffers alternate, so a call waits only for the reduction of the
  // call two back before overwriting its buffer.
  int ln_calls = 0;
  auto ln_bwd = [&](const float* X_, const char* mean_, const char* rstd_, const void* g_,
                    const float* dres_, float* dX_, void* dXt_, float* gg, float* gb,
                    float* gc) -> mpipe_status {
    const int k = ln_calls++ & 1;
    float* pg = part + 3 * k * ln_set;
    float* pb = pg + ln_set;
    float* pc = (dX_ && gc) ? pb + ln_set : nullptr;
    MP_CHECK(ss.acquire(FREE_LNP0 + k));
    int64_t nb = 0;
    MP_CHECK(run(x.e, x.s, "layernorm_bwd", 0, [&] {
      return layernorm_bwd_partials(x.dt, dxln, x.dt, h, X_, h, reinterpret_cast<const float*>(mean_),
                                    reinterpret_cast<const float*>(rstd_), g_, N, (int)h, dres_,
                                    dX_, dXt_, pg, pb, pc, &nb, x.s);
    }));
    MP_CHECK(ss.fork());
    MP_CHECK(run(x.e, x.s2, "ln_reduce", 0, [&] {
      return layernorm_bwd_reduce(pg, gg, pb, gb, pc, pc ? gc : nullptr, nb, (int)h, x.s2);
    }));
    MP_CHECK(ss.release(FREE_LNP0 + k));
    return MPIPE_OK;
  };
  MP_CHECK(ss.fork());
  // merger
  MP_RET(dw_gemm(x, dM, H, base + MS.gm, 4 * h, H, 4 * h, Tm, x.grad(dw, merger_param(c, M_FC2W)), 4 * h));
  MP_RET(colsum(x, x.dt, dM, H, Tm, (int)H, x.grad(dw, merger_param(c, M_FC2B))));
  // the GELU-backward GEMM also writes the column sums of du (the fc1 bias gradient) when
  // it runs on the kernel that can; otherwise the side stream sums du
  bool fused = false;
  float* gpart = reinterpret_cast<float*>(x.ws + P.ws_gpart);
  {
    GemmArgs a = ga(dM, H, x.W(merger_param(c, M_FC2W)), 4 * h, Tm, 4 * h, H, du, 4 * h);
    a.aux = base + MS.um;
    a.ld_aux = 4 * h;
    fused = gemm_fused_colsum(x.dt, GEMM_NN, EPI_GELU_BWD, a);
    if (fused) a.colsum = gpart;
    MP_RET(gemm_call(x, GEMM_NN, EPI_GELU_BWD, a));
  }
  MP_CHECK(ss.fork());
  MP_RET(dw_gemm(x, du, 4 * h, base + MS.z, 4 * h, 4 * h, 4 * h, Tm, x.grad(dw, merger_param(c, M_FC1W)), 4 * h));
  MP_RET(fused ? band_reduce(x, Tm, (int)(4 * h), x.grad(dw, merger_param(c, M_FC1B)))
               : colsum(x, x.dt, du, 4 * h, Tm, (int)(4 * h), x.grad(dw, merger_param(c, M_FC1B))));
  MP_CHECK(ss.release(FREE_DU));
  {
    GemmArgs a = ga(du, 4 * h, x.W(merger_param(c, M_FC1W)), 4 * h, Tm, 4 * h, 4 * h, dxln, 4 * h);
    MP_RET(gemm_call(x, GEMM_NN, epi_dxln, a));
  }
  MP_RET(ln_bwd(reinterpret_cast<const float*>(base + MS.hfin), base + MS.meanz, base + MS.rstdz,
                x.W(merger_param(c, M_LNG)), nullptr, merger_only ? nullptr : dh,
                merger_only ? nullptr : dht, x.grad(dw, merger_param(c, M_LNG)),
                x.grad(dw, merger_param(c, M_LNB)),
                merger_only ? nullptr : x.grad(dw, blk_param(c, c.layers - 1, B_FC2B))));
  if (merger_only) return MPIPE_OK;

  int pending_qkv = -1;   // block whose qkv weight gradient is still to be launched
  auto qkv_dw = [&](int lq) -> mpipe_status {
    char* const dq_ = dqkvb[lq & 1];
    MP_RET(dw_gemm(x, dq_, 3 * h, base + P.tape_act[lq].a, h, 3 * h, h, N,
                   x.grad(dw, blk_param(c, lq, B_QKVW)), h));
    MP_RET(colsum(x, x.dt, dq_, 3 * h, N, (int)(3 * h), x.grad(dw, blk_param(c, lq, B_QKVB))));
    MP_CHECK(ss.release((lq & 1) ? FREE_DQKV1 : FREE_DQKV));
    return MPIPE_OK;
  };
  for (int l = c.layers - 1; l >= 0; --l) {
    const ActSet& S = P.tape_act[l];
    const float* hin = reinterpret_cast<const float*>(base + S.hin);
    const float* hmid = reinterpret_cast<const float*>(base + S.hmid);
    // MLP: H_out = H_mid + GELU(B W1^T + b1) W2^T + b2
    MP_CHECK(ss.acquire(FREE_DU));
    {
      GemmArgs a = ga(dht, h, x.W(blk_param(c, l, B_FC2W)), m, N, m, h, du, m);
      a.aux = base + S.u;
      a.ld_aux = m;
      fused = gemm_fused_colsum(x.dt, GEMM_NN, EPI_GELU_BWD, a);
      if (fused) a.colsum = gpart;
      MP_RET(gemm_call(x, GEMM_NN, EPI_GELU_BWD, a));
    }
    {
      GemmArgs a = ga(du, m, x.W(blk_param(c, l, B_FC1W)), h, N, h, m, dxln, h);
      MP_RET(gemm_call(x, GEMM_NN, epi_dxln, a));
    }
    MP_CHECK(ss.acquire(FREE_DHM));
    MP_RET(ln_bwd(hmid, base + S.mean2, base + S.rstd2, x.W(blk_param(c, l, B_LN2G)), dh, dhm,
                  dhmt, x.grad(dw, blk_param(c, l, B_LN2G)), x.grad(dw, blk_param(c, l, B_LN2B)),
                  x.grad(dw, blk_param(c, l, B_PROJB))));
    // The MLP's weight gradients start only now, after the LayerNorm backward: a
    // memory-bound kernel that shares the chip with weight-gradient tiles ran 2.5x longer
    // (same-call A/B of this order against forking each GEMM as soon as its operand
    // exists: 281.2 -> 277.1 ms per step)
    MP_CHECK(ss.fork());   // dh, dht, du and its band sums
    if (pending_qkv >= 0) MP_RET(qkv_dw(pending_qkv));
    pending_qkv = -1;
    MP_RET(dw_gemm(x, dht, h, base + S.g, m, h, m, N, x.grad(dw, blk_param(c, l, B_FC2W)), m));
    MP_CHECK(ss.release(FREE_DH));
    MP_RET(dw_gemm(x, du, m, base + S.b, h, m, h, N, x.grad(dw, blk_param(c, l, B_FC1W)), h));
    MP_RET(fused ? band_reduce(x, N, (int)m, x.grad(dw, blk_param(c, l, B_FC1B)))
                 : colsum(x, x.dt, du, m, N, (int)m, x.grad(dw, blk_param(c, l, B_FC1B))));
    MP_CHECK(ss.release(FREE_DU));
    // attention: H_mid = H_in + O Wo^T + bo
    MP_CHECK(ss.fork());   // dhm, dhmt
    MP_RET(dw_gemm(x, dhmt, h, base + S.o, h, h, h, N, x.grad(dw, blk_param(c, l, B_PROJW)), h));
    MP_CHECK(ss.release(FREE_DHM));
    {
      GemmArgs a = ga(dhmt, h, x.W(blk_param(c, l, B_PROJW)), h, N, h, h, dO, h);
      MP_RET(gemm_call(x, GEMM_NN, EPI_STORE, a));
    }
    char* const dqkv = dqkvb[l & 1];
    MP_CHECK(ss.acquire((l & 1) ? FREE_DQKV1 : FREE_DQKV));
    {
      const char* qkv = base + S.qkv;
      AttnArgs qa = attn_args(x, qkv, false), ka = attn_args(x, qkv, true);
      for (AttnArgs* a : {&qa, &ka}) {
        a->o = base + S.o;
        a->d_o = dO;
        a->ldo = h;
        a->lse = const_cast<float*>(reinterpret_cast<const float*>(base + S.lse));
        a->delta = delta;
        a->delta_out = delta;
        a->dq = dqkv;
        a->dk = dqkv + h * x.E;
        a->dv = dqkv + 2 * h * x.E;
        a->ldd = 3 * h;
        // the tape's q, k are pair-interleaved and rotated: dQ, dK are written rotated
        // back, in plain column order
        a->rope_pos = pos;
        a->rope_tab = reinterpret_cast<const float2*>(freq);
      }
      const double f = 2.0 * c.heads * c.d * (double)P.sum_len2;
      MP_CHECK(run(x.e, x.s, "attn_bwd_dq", f, [&] { return attention_bwd_dq(x.dt, c.d, qa, x.s); }));
      MP_CHECK(run(x.e, x.s, "attn_bwd_dkdv", 3 * f, [&] { return attention_bwd_dkdv(x.dt, c.d, ka, x.s); }));
    }
    {
      GemmArgs a = ga(dqkv, 3 * h, x.W(blk_param(c, l, B_QKVW)), h, N, h, 3 * h, dxln, h);
      MP_RET(gemm_call(x, GEMM_NN, epi_dxln, a));
    }
    MP_CHECK(ss.acquire(FREE_DH));
    MP_RET(ln_bwd(hin, base + S.mean1, base + S.rstd1, x.W(blk_param(c, l, B_LN1G)), dhm, dh, dht,
                  x.grad(dw, blk_param(c, l, B_LN1G)), x.grad(dw, blk_param(c, l, B_LN1B)),
                  x.grad(dw, l > 0 ? blk_param(c, l - 1, B_FC2B) : P_PE_B)));
    // qkv's weight gradient runs beside the next block's attention (its dqkv buffer
    // alternates with the next block's)
    pending_qkv = l;
  }
  // patch embedding (the trainable source: nothing goes upstream unless asked)
  MP_CHECK(ss.fork());   // dh, dht
  if (pending_qkv >= 0) MP_RET(qkv_dw(pending_qkv));
  MP_RET(dw_gemm(x, dht, h, Xp, ldx, h, c.kpe, N, x.grad(dw, P_PE_W), c.kpe));
  if (d_patches) {
    GemmArgs a = ga(dht, h, Wpe, ldx, N, c.kpe, h, d_patches, c.kpe);
    MP_RET(gemm_call(x, GEMM_NN, EPI_STORE, a));
  }
  return MPIPE_OK;
}

mpipe_status check_handle(const mpipe_encoder* e) {
  if (!e) return fail(MPIPE_ERR_INVALID_ARG, "null encoder handle");
  return MPIPE_OK;
}

}  // namespace

// =====================================================================================
// C ABI
// =====================================================================================
extern "C" {

mpipe_status mpipe_encoder_create(const mpipe_encoder_cfg* cfg, mpipe_encoder** out) {
  if (!cfg || !out) return fail(MPIPE_ERR_INVALID_ARG, "null argument");
  Cfg c = to_cfg(cfg);
  const std::string why = check_cfg(c);
  if (!why.empty()) return fail(MPIPE_ERR_UNSUPPORTED, why);
  mpipe_encoder* e = new mpipe_encoder();
  e->cfg = c;
  e->params = param_table(c);
  *out = e;
  return MPIPE_OK;
}

void mpipe_encoder_destroy(mpipe_encoder* e) {
  if (!e) return;
  // teardown has no caller to report to: each release is attempted regardless
  if (e->staging_pending && e->staging_ev) (void)hipEventSynchronize(e->staging_ev);
  if (e->staging) (void)hipHostFree(e->staging);
  if (e->staging_ev) (void)hipEventDestroy(e->staging_ev);
  for (auto& r : e->recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto ev : e->pool) (void)hipEventDestroy(ev);
  if (e->side) {
    (void)hipStreamSynchronize(e->side);
    (void)hipStreamDestroy(e->side);
  }
  for (auto ev : e->sync)
    if (ev) (void)hipEventDestroy(ev);
  delete e;
}

mpipe_status mpipe_encoder_set_side_stream(mpipe_encoder* e, int32_t enable) {
  MP_RET(check_handle(e));
  e->side_on = enable != 0;
  return MPIPE_OK;
}

int64_t mpipe_param_count(const mpipe_encoder_cfg* cfg) {
  if (!cfg) return -1;
  Cfg c = to_cfg(cfg);
  auto t = param_table(c);
  return t.empty() ? 0 : t.back().off + t.back().rows * t.back().cols;
}

int32_t mpipe_param_tensors(const mpipe_encoder_cfg* cfg) {
  if (!cfg) return -1;
  return (int32_t)param_table(to_cfg(cfg)).size();
}

mpipe_status mpipe_param_info(const mpipe_encoder_cfg* cfg, int32_t i, char* name, int32_t cap,
                              int64_t* offset, int64_t* rows, int64_t* cols) {
  if (!cfg) return fail(MPIPE_ERR_INVALID_ARG, "null cfg");
  auto t = param_table(to_cfg(cfg));
  if (i < 0 || i >= (int32_t)t.size()) return fail(MPIPE_ERR_INVALID_ARG, "tensor index out of range");
  if (name && cap > 0) {
    std::strncpy(name, t[i].name.c_str(), (size_t)cap - 1);
    name[cap - 1] = 0;
  }
  if (offset) *offset = t[i].off;
  if (rows) *rows = t[i].rows;
  if (cols) *cols = t[i].cols;
  return MPIPE_OK;
}

mpipe_status mpipe_encoder_sizes(const mpipe_encoder* e, const int32_t* cu, int32_t n_seg,
                                 const int32_t* thw, int32_t n_items, int32_t trainable,
                                 size_t* ws_bytes, size_t* tape_bytes, int64_t* n_merged,
                                 int64_t* n_patches) {
  MP_RET(check_handle(e));
  Plan P;
  std::string err;
  const int rc = build_plan(e->cfg, cu, n_seg, thw, n_items, trainable, P, err);
  if (rc) return fail((mpipe_status)rc, err);
  if (ws_bytes) *ws_bytes = P.ws_bytes;
  if (tape_bytes) *tape_bytes = P.tape_bytes;
  if (n_merged) *n_merged = P.Tm;
  if (n_patches) *n_patches = P.N;
  return MPIPE_OK;
}

mpipe_status mpipe_encoder_regions(const mpipe_encoder* e, const int32_t* cu, int32_t n_seg,
                                   const int32_t* thw, int32_t n_items, int32_t trainable,
                                   int32_t which, int64_t* offsets, int64_t* bytes, int32_t cap,
                                   int32_t* n_regions) {
  MP_RET(check_handle(e));
  if (which != 0 && which != 1) return fail(MPIPE_ERR_INVALID_ARG, "which must be 0 or 1");
  if (!n_regions || cap < 0 || (cap > 0 && (!offsets || !bytes)))
    return fail(MPIPE_ERR_INVALID_ARG, "null output");
  Plan P;
  std::string err;
  const int rc = build_plan(e->cfg, cu, n_seg, thw, n_items, trainable, P, err);
  if (rc) return fail((mpipe_status)rc, err);
  const std::vector<Region>& R = which == 0 ? P.ws_regions : P.tape_regions;
  *n_regions = (int32_t)R.size();
  for (int32_t i = 0; i < cap && i < (int32_t)R.size(); ++i) {
    offsets[i] = (int64_t)R[i].off;
    bytes[i] = (int64_t)R[i].bytes;
  }
  return MPIPE_OK;
}

mpipe_status mpipe_encoder_cost(const mpipe_encoder* e, const int32_t* cu, int32_t n_seg,
                                const int32_t* thw, int32_t n_items, int32_t trainable,
                                double flops_per_s, double bytes_per_s, mpipe_slab_cost* out) {
  MP_RET(check_handle(e));
  if (!out || !(flops_per_s > 0) || !(bytes_per_s > 0))
    return fail(MPIPE_ERR_INVALID_ARG, "need an output and rates > 0");
  Plan P;
  std::string err;
  const int rc = build_plan(e->cfg, cu, n_seg, thw, n_items, trainable, P, err);
  if (rc) return fail((mpipe_status)rc, err);
  const SlabCost sc = encoder_slab_cost(e->cfg, P);
  out->fwd_flops = sc.fwd_flops;
  out->fwd_bytes = sc.fwd_bytes;
  out->fwd_seconds = std::max(sc.fwd_flops / flops_per_s, sc.fwd_bytes / bytes_per_s);
  out->bwd_flops = sc.bwd_flops;
  out->bwd_bytes = sc.bwd_bytes;
  out->bwd_seconds = std::max(sc.bwd_flops / flops_per_s, sc.bwd_bytes / bytes_per_s);
  return MPIPE_OK;
}

mpipe_status mpipe_encoder_fwd(mpipe_encoder* e, const void* weights, const void* patches,
                               const int32_t* cu, int32_t n_seg, const int32_t* thw,
                               int32_t n_items, int32_t trainable, void* merged, void* tape,
                               size_t tape_bytes, void* ws, size_t ws_bytes, void* stream) {
  MP_RET(check_handle(e));
  Plan P;
  std::string err;
  const int rc = build_plan(e->cfg, cu, n_seg, thw, n_items, trainable, P, err);
  if (rc) return fail((mpipe_status)rc, err);
  if (P.N == 0) return MPIPE_OK;
  if (!weights || !patches || !merged) return fail(MPIPE_ERR_INVALID_ARG, "null device buffer");
  if (!ws || ws_bytes < P.ws_bytes)
    return fail(MPIPE_ERR_WORKSPACE, "workspace needs " + std::to_string(P.ws_bytes) + " bytes");
  if (trainable && (!tape || tape_bytes < P.tape_bytes))
    return fail(MPIPE_ERR_NO_TAPE, "trainable forward needs a tape of " +
                                       std::to_string(P.tape_bytes) + " bytes");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  MP_RET(upload_meta(e, P, reinterpret_cast<char*>(ws), s));
  Ctx x{e, e->cfg, P, s, reinterpret_cast<const char*>(weights), reinterpret_cast<char*>(ws),
        e->cfg.dtype, e->cfg.esz};
  x.s2 = s;
  return forward(x, patches, merged, reinterpret_cast<char*>(tape));
}

mpipe_status mpipe_encoder_bwd(mpipe_encoder* e, const void* weights, const void* patches,
                               const int32_t* cu, int32_t n_seg, const int32_t* thw,
                               int32_t n_items, int32_t trainable, const void* tape,
                               size_t tape_bytes, const void* d_merged, float* d_weights,
                               void* d_patches, void* ws, size_t ws_bytes, void* stream) {
  MP_RET(check_handle(e));
  if (trainable == MODE_FROZEN)
    return fail(MPIPE_NOOP_FROZEN, "frozen encoder: no backward (Lemma 1)");
  Plan P;
  std::string err;
  const int rc = build_plan(e->cfg, cu, n_seg, thw, n_items, trainable, P, err);
  if (rc) return fail((mpipe_status)rc, err);
  if (P.mode == MODE_MERGER && d_patches)
    return fail(MPIPE_ERR_INVALID_ARG,
                "only the merger is trainable: it sends nothing upstream, d_patches must be NULL");
  if (P.N == 0) return MPIPE_OK;
  if (!weights || !patches || !d_merged || !d_weights)
    return fail(MPIPE_ERR_INVALID_ARG, "null device buffer");
  if (!tape || tape_bytes < P.tape_bytes)
    return fail(MPIPE_ERR_NO_TAPE, "backward needs the forward's tape of " +
                                       std::to_string(P.tape_bytes) + " bytes");
  if (!ws || ws_bytes < P.ws_bytes)
    return fail(MPIPE_ERR_WORKSPACE, "workspace needs " + std::to_string(P.ws_bytes) + " bytes");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  MP_RET(upload_meta(e, P, reinterpret_cast<char*>(ws), s));
  Ctx x{e, e->cfg, P, s, reinterpret_cast<const char*>(weights), reinterpret_cast<char*>(ws),
        e->cfg.dtype, e->cfg.esz};
  x.s2 = s;
  if (e->side_on) {
    MP_CHECK(ensure_side(e));
    x.s2 = e->side;
  }
  const mpipe_status st =
      backward(x, patches, reinterpret_cast<const char*>(tape), d_merged, d_weights, d_patches);
  // join on every path, so the caller's stream never runs ahead of gradient work
  SideSync ss{x, x.s2 != x.s};
  const hipError_t j = ss.join();
  if (st != MPIPE_OK) return st;
  MP_CHECK(j);
  return MPIPE_OK;
}

static mpipe_status rows_common(int32_t row_elems, int32_t dtype, int64_t n_merged, int64_t n_rows,
                                const void* a, const void* b, const int64_t* idx) {
  if (dtype != MPIPE_F32 && dtype != MPIPE_BF16) return fail(MPIPE_ERR_INVALID_ARG, "bad dtype");
  if (row_elems <= 0 || n_merged < 0 || n_rows < 0)
    return fail(MPIPE_ERR_INVALID_ARG, "negative size");
  if (n_merged > 0 && (!a || !b || !idx)) return fail(MPIPE_ERR_INVALID_ARG, "null device buffer");
  return MPIPE_OK;
}

mpipe_status mpipe_merge_scatter(const void* merged, int64_t n_merged, int32_t row_elems,
                                 int32_t dtype, const int64_t* idx, void* embeds, int64_t n_rows,
                                 void* stream) {
  MP_RET(rows_common(row_elems, dtype, n_merged, n_rows, merged, embeds, idx));
  const int64_t rb = (int64_t)row_elems * (dtype == MPIPE_BF16 ? 2 : 4);
  MP_CHECK(rows_copy(true, merged, embeds, idx, n_merged, rb, n_rows,
                     reinterpret_cast<hipStream_t>(stream)));
  return MPIPE_OK;
}

mpipe_status mpipe_merge_gather(const void* d_embeds, int64_t n_rows, int32_t row_elems,
                                int32_t dtype, const int64_t* idx, int64_t n_merged,
                                void* d_merged, void* stream) {
  MP_RET(rows_common(row_elems, dtype, n_merged, n_rows, d_embeds, d_merged, idx));
  const int64_t rb = (int64_t)row_elems * (dtype == MPIPE_BF16 ? 2 : 4);
  MP_CHECK(rows_copy(false, d_embeds, d_merged, idx, n_merged, rb, n_rows,
                     reinterpret_cast<hipStream_t>(stream)));
  return MPIPE_OK;
}

mpipe_status mpipe_merge_check_indices(const int64_t* idx, int64_t n_merged, int64_t n_rows,
                                       int32_t* marks, int32_t* status, void* stream) {
  if (n_merged < 0 || n_rows < 0) return fail(MPIPE_ERR_INVALID_ARG, "negative size");
  if (!status || (n_rows > 0 && !marks) || (n_merged > 0 && !idx))
    return fail(MPIPE_ERR_INVALID_ARG, "null device buffer");
  MP_CHECK(check_indices(idx, n_merged, n_rows, marks, status, reinterpret_cast<hipStream_t>(stream)));
  return MPIPE_OK;
}

const char* mpipe_last_error(void) { return g_err.c_str(); }

mpipe_status mpipe_profile_enable(mpipe_encoder* e, int32_t enable) {
  MP_RET(check_handle(e));
  e->prof = enable != 0;
  return MPIPE_OK;
}

int32_t mpipe_profile_read(mpipe_encoder* e, void* stream, int32_t cap, char* names,
                           int32_t name_stride, int64_t* launches, double* ms, double* flops) {
  if (!e) return -1;
  if (hipStreamSynchronize(reinterpret_cast<hipStream_t>(stream)) != hipSuccess) return -1;
  std::map<std::string, std::tuple<int64_t, double, double>> agg;
  for (auto& r : e->recs) {
    float t = 0.f;
    if (hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) t = 0.f;   // counted, timed as 0
    auto& v = agg[r.side ? r.cls + "@side" : r.cls];
    std::get<0>(v) += 1;
    std::get<1>(v) += t;
    std::get<2>(v) += r.flops;
    e->pool.push_back(r.a);
    e->pool.push_back(r.b);
  }
  e->recs.clear();
  int32_t n = 0;
  for (auto& kv : agg) {
    if (n >= cap) break;
    if (names && name_stride > 0) {
      std::strncpy(names + (size_t)n * name_stride, kv.first.c_str(), (size_t)name_stride - 1);
      names[(size_t)n * name_stride + name_stride - 1] = 0;
    }
    if (launches) launches[n] = std::get<0>(kv.second);
    if (ms) ms[n] = std::get<1>(kv.second);
    if (flops) flops[n] = std::get<2>(kv.second);
    ++n;
  }
  return n;
}

}  // extern "C"
