// Kernel-level entry points of libmpipe (include/mpipe_ops.h).
#include "../../include/mpipe_ops.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "internal.h"
#include "plan.h"

using namespace mpipe;

extern "C" const char* mpipe_last_error(void);
namespace mpipe {
mpipe_status set_error(mpipe_status s, const std::string& m);
}

namespace {

#define OP_CHECK(expr)                                                                         \
  do {                                                                                         \
    hipError_t _e = (expr);                                                                    \
    if (_e != hipSuccess)                                                                      \
      return set_error(MPIPE_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(_e));      \
  } while (0)

size_t al(size_t x) { return (x + 255) / 256 * 256; }

// attention work lists (tiles of ATTN_TILE rows, longest segments first) into scratch
mpipe_status upload_work(const int32_t* cu, int n_seg, int64_t N, char* scratch, size_t bytes,
                         hipStream_t s, int& n_work, size_t& off_end) {
  if (n_seg < 0 || (n_seg > 0 && !cu)) return set_error(MPIPE_ERR_INVALID_ARG, "bad segments");
  if (n_seg == 0 || N == 0) {
    n_work = 0;
    off_end = 0;
    return MPIPE_OK;
  }
  if (cu[0] != 0 || cu[n_seg] != N) return set_error(MPIPE_ERR_BAD_METADATA, "cu_seqlens must span [0, N]");
  std::vector<int> order(n_seg);
  for (int i = 0; i < n_seg; ++i) {
    order[i] = i;
    if (cu[i + 1] <= cu[i]) return set_error(MPIPE_ERR_BAD_METADATA, "cu_seqlens not increasing");
  }
  std::stable_sort(order.begin(), order.end(),
                   [&](int a, int b) { return cu[a + 1] - cu[a] > cu[b + 1] - cu[b]; });
  std::vector<int32_t> w;
  for (int sg : order)
    for (int r = cu[sg]; r < cu[sg + 1]; r += ATTN_TILE) w.insert(w.end(), {r, cu[sg], cu[sg + 1], 0});
  n_work = (int)(w.size() / 4);
  off_end = al(w.size() * sizeof(int32_t));
  if (off_end > bytes) return set_error(MPIPE_ERR_WORKSPACE, "scratch too small");
  OP_CHECK(hipMemcpyAsync(scratch, w.data(), w.size() * sizeof(int32_t), hipMemcpyHostToDevice, s));
  OP_CHECK(hipStreamSynchronize(s));
  return MPIPE_OK;
}

}  // namespace

extern "C" {

size_t mpipe_op_scratch_bytes(int64_t N, int32_t heads, int32_t n, int32_t n_seg) {
  const size_t work = al(((size_t)(N + ATTN_TILE - 1) / ATTN_TILE + (size_t)n_seg + 1) * 16);
  const size_t delta = al((size_t)heads * N * 4);
  const size_t pos = al((size_t)N * 4) + al((size_t)65536 * 8);
  const size_t part = al((size_t)layernorm_bwd_partial_rows(N) * std::max(n, 1) * 4) * 3;
  return std::max(work + delta, pos) + part + 4096;
}

mpipe_status mpipe_op_gemm(int32_t dtype, int32_t layout, int32_t epi, int32_t M, int32_t N,
                           int32_t K, const void* A, int64_t lda, const void* B, int64_t ldb,
                           void* C, int64_t ldc, const void* bias, const void* aux, int64_t ld_aux,
                           void* C2, int64_t ldc2, int32_t beta, int32_t kps,
                           int64_t split_stride, void* stream) {
  if (dtype != 0 && dtype != 1) return set_error(MPIPE_ERR_INVALID_ARG, "bad dtype");
  if (layout < 0 || layout > 2 || epi < 0 || epi > 4) return set_error(MPIPE_ERR_INVALID_ARG, "bad layout/epilogue");
  if (M < 0 || N < 0 || K < 0) return set_error(MPIPE_ERR_INVALID_ARG, "negative size");
  const int vec = dtype == 1 ? 8 : 4;
  const bool a_km = layout == GEMM_TN, b_km = layout != GEMM_NT;
  if (!a_km && (K % vec || lda % vec)) return set_error(MPIPE_ERR_INVALID_ARG, "A: K and lda must be multiples of the vector width");
  if (a_km && (M % vec || lda % vec)) return set_error(MPIPE_ERR_INVALID_ARG, "A (K-major): M and lda must be multiples of the vector width");
  if (!b_km && (K % vec || ldb % vec)) return set_error(MPIPE_ERR_INVALID_ARG, "B: K and ldb must be multiples of the vector width");
  if (b_km && (ldb % vec || ((N + vec - 1) / vec * vec) > ldb)) return set_error(MPIPE_ERR_INVALID_ARG, "B (K-major): ldb must be a multiple of the vector width covering N");
  if (kps > 0 && (kps % 64 || epi != EPI_F32)) return set_error(MPIPE_ERR_INVALID_ARG, "k_per_split must be a multiple of 64 and needs epilogue 4");
  GemmArgs a;
  a.A = A; a.B = B; a.lda = lda; a.ldb = ldb; a.M = M; a.N = N; a.K = K; a.kps = kps;
  a.C = C; a.ldc = ldc; a.split_stride = split_stride; a.bias = bias; a.aux = aux;
  a.ld_aux = ld_aux; a.C2 = C2; a.ldc2 = ldc2; a.beta = beta;
  OP_CHECK(gemm(dtype, layout, epi, a, reinterpret_cast<hipStream_t>(stream)));
  return MPIPE_OK;
}

mpipe_status mpipe_op_splitk_reduce(const float* part, int32_t splits, int64_t M, int64_t N,
                                    float* out, int64_t ldo, void* stream) {
  if (splits < 1 || M < 0 || N < 0 || ldo < N)
    return set_error(MPIPE_ERR_INVALID_ARG, "need splits >= 1, M, N >= 0 and ldo >= N");
  if (M * N > 0 && (!part || !out)) return set_error(MPIPE_ERR_INVALID_ARG, "null device buffer");
  OP_CHECK(splitk_reduce(part, splits, M, N, out, ldo, reinterpret_cast<hipStream_t>(stream)));
  return MPIPE_OK;
}

int32_t mpipe_op_weight_grad_splits(int64_t M, int64_t N, int64_t K) {
  if (M < 0 || N < 0 || K < 0) return -1;
  return choose_split(M, N, K).splits;
}

mpipe_status mpipe_op_layernorm_fwd(int32_t dtype, const float* X, int64_t rows, int32_t n,
                                    const void* g, const void* b, float eps, void* Y, float* mean,
                                    float* rstd, void* stream) {
  if (n % 4 || n > 2048 || n <= 0) return set_error(MPIPE_ERR_UNSUPPORTED, "n must be a multiple of 4, <= 2048");
  OP_CHECK(layernorm_fwd(dtype, X, n, rows, n, g, b, eps, Y, n, mean, rstd,
                         reinterpret_cast<hipStream_t>(stream)));
  return MPIPE_OK;
}

mpipe_status mpipe_op_layernorm_bwd(int32_t dtype, const float* dY, const float* X,
                                    const float* mean, const float* rstd, const void* g,
                                    int64_t rows, int32_t n, const float* dres, float* dX,
                                    void* dXt, float* grad_g, float* grad_b, float* colsum_dx,
                                    void* scratch, size_t scratch_bytes, void* stream) {
  if (n % 4 || n > 2048 || n <= 0) return set_error(MPIPE_ERR_UNSUPPORTED, "n must be a multiple of 4, <= 2048");
  const size_t third = al((size_t)layernorm_bwd_partial_rows(rows) * n * 4);
  if (scratch_bytes < 3 * third) return set_error(MPIPE_ERR_WORKSPACE, "scratch too small");
  float* pg = reinterpret_cast<float*>(scratch);
  float* pb = reinterpret_cast<float*>(reinterpret_cast<char*>(scratch) + third);
  float* pc = reinterpret_cast<float*>(reinterpret_cast<char*>(scratch) + 2 * third);
  OP_CHECK(layernorm_bwd(dtype, dY, n, X, n, mean, rstd, g, rows, n, dres, dX, dXt, pg, pb, pc,
                         grad_g, grad_b, colsum_dx, reinterpret_cast<hipStream_t>(stream)));
  return MPIPE_OK;
}

mpipe_status mpipe_op_rope(int32_t dtype, void* qkv, int64_t rows, int32_t heads, int32_t d,
                           const int32_t* thw, int32_t n_items, float theta, int32_t inverse,
                           void* scratch, size_t scratch_bytes, void* stream) {
  if (d % 8) return set_error(MPIPE_ERR_UNSUPPORTED, "head_dim must be a multiple of 8");
  std::vector<int32_t> pos;
  int64_t n = 0;
  for (int i = 0; i < n_items; ++i) {
    const int t = thw[3 * i], gh = thw[3 * i + 1], gw = thw[3 * i + 2];
    if (t <= 0 || gh <= 0 || gw <= 0 || gh % 2 || gw % 2) return set_error(MPIPE_ERR_BAD_METADATA, "bad grid");
    for (int64_t r = 0; r < (int64_t)t * gh * gw; ++r) {
      const int64_t w = r >> 2;
      const int wb = (int)(w % (gw / 2)), hb = (int)((w / (gw / 2)) % (gh / 2));
      pos.push_back(((2 * hb + (int)((r >> 1) & 1)) << 16) | (2 * wb + (int)(r & 1)));
    }
    n += (int64_t)t * gh * gw;
  }
  if (n != rows) return set_error(MPIPE_ERR_BAD_METADATA, "grid does not match rows");
  int max_side = 1;
  for (int i = 0; i < n_items; ++i) max_side = std::max({max_side, thw[3 * i + 1], thw[3 * i + 2]});
  Cfg cf;
  cf.hidden = heads * d;
  cf.heads = heads;
  cf.theta = theta;
  derive_cfg(cf);
  std::vector<float> tab = rope_table(cf, max_side);
  const size_t need = al(pos.size() * 4) + al(tab.size() * 4);
  if (scratch_bytes < need) return set_error(MPIPE_ERR_WORKSPACE, "scratch too small");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* sc = reinterpret_cast<char*>(scratch);
  OP_CHECK(hipMemcpyAsync(sc, pos.data(), pos.size() * 4, hipMemcpyHostToDevice, s));
  OP_CHECK(hipMemcpyAsync(sc + al(pos.size() * 4), tab.data(), tab.size() * 4, hipMemcpyHostToDevice, s));
  OP_CHECK(rope(dtype, qkv, 3 * (int64_t)heads * d, rows, heads, d, heads * d,
                reinterpret_cast<const int32_t*>(sc),
                reinterpret_cast<const float*>(sc + al(pos.size() * 4)), inverse, s));
  OP_CHECK(hipStreamSynchronize(s));
  return MPIPE_OK;
}

mpipe_status mpipe_op_attention_fwd(int32_t dtype, const void* qkv, int64_t N, int32_t heads,
                                    int32_t d, const int32_t* cu, int32_t n_seg, void* o,
                                    float* lse, void* scratch, size_t scratch_bytes, void* stream) {
  if (!attention_supported(dtype, d)) return set_error(MPIPE_ERR_UNSUPPORTED, "head_dim not supported");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  int n_work = 0;
  size_t end = 0;
  mpipe_status st = upload_work(cu, n_seg, N, reinterpret_cast<char*>(scratch), scratch_bytes, s, n_work, end);
  if (st) return st;
  const int64_t E = dtype == 1 ? 2 : 4, h = (int64_t)heads * d;
  AttnArgs a;
  a.q = qkv;
  a.k = reinterpret_cast<const char*>(qkv) + h * E;
  a.v = reinterpret_cast<const char*>(qkv) + 2 * h * E;
  a.ld = 3 * h;
  a.out = o;
  a.ldo = h;
  a.lse = lse;
  a.work = reinterpret_cast<const int4*>(scratch);
  a.n_work = n_work;
  a.heads = heads;
  a.N = N;
  a.scale = 1.0f / std::sqrt((float)d);
  OP_CHECK(attention_fwd(dtype, d, a, s));
  return MPIPE_OK;
}

mpipe_status mpipe_op_attention_bwd(int32_t dtype, const void* qkv, const void* o, const void* d_o,
                                    const float* lse, int64_t N, int32_t heads, int32_t d,
                                    const int32_t* cu, int32_t n_seg, void* dqkv, void* scratch,
                                    size_t scratch_bytes, void* stream) {
  if (!attention_supported(dtype, d)) return set_error(MPIPE_ERR_UNSUPPORTED, "head_dim not supported");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  int n_work = 0;
  size_t end = 0;
  mpipe_status st = upload_work(cu, n_seg, N, reinterpret_cast<char*>(scratch), scratch_bytes, s, n_work, end);
  if (st) return st;
  const int64_t E = dtype == 1 ? 2 : 4, h = (int64_t)heads * d;
  if (end + al((size_t)heads * N * 4) > scratch_bytes) return set_error(MPIPE_ERR_WORKSPACE, "scratch too small");
  float* delta = reinterpret_cast<float*>(reinterpret_cast<char*>(scratch) + end);
  AttnArgs a;
  a.q = qkv;
  a.k = reinterpret_cast<const char*>(qkv) + h * E;
  a.v = reinterpret_cast<const char*>(qkv) + 2 * h * E;
  a.ld = 3 * h;
  a.o = o;
  a.d_o = d_o;
  a.ldo = h;
  a.lse = const_cast<float*>(lse);
  a.delta = delta;
  a.delta_out = delta;
  a.dq = dqkv;
  a.dk = reinterpret_cast<char*>(dqkv) + h * E;
  a.dv = reinterpret_cast<char*>(dqkv) + 2 * h * E;
  a.ldd = 3 * h;
  a.work = reinterpret_cast<const int4*>(scratch);
  a.n_work = n_work;
  a.heads = heads;
  a.N = N;
  a.scale = 1.0f / std::sqrt((float)d);
  OP_CHECK(attention_bwd_dq(dtype, d, a, s));
  OP_CHECK(attention_bwd_dkdv(dtype, d, a, s));
  return MPIPE_OK;
}

}  // extern "C"
