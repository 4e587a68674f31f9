// Row-wise and element-wise kernels of the encoder step: LayerNorm forward and
// backward (fp32 statistics, one wave64 per row, wavefront reductions), 2D
// rotary position, operand padding, deterministic column reductions for the
// bias / LayerNorm-affine gradients, the split-K reduction of weight
// gradients, and the bit-exact placeholder row scatter / gather.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "internal.h"
#include "plan.h"

namespace mpipe {
namespace {

constexpr int MAXC = 8;  // float4 chunks per lane: LayerNorm rows up to 64 * 4 * 8 = 2048 wide

template <class T> struct V4;
template <> struct V4<float> {
  static __device__ __forceinline__ float4 load(const float* p) {
    return *reinterpret_cast<const float4*>(p);
  }
  static __device__ __forceinline__ void store(float* p, float4 v) {
    *reinterpret_cast<float4*>(p) = v;
  }
};
template <> struct V4<bf16> {
  static __device__ __forceinline__ float4 load(const bf16* p) {
    uint2 u = *reinterpret_cast<const uint2*>(p);
    const bf16* b = reinterpret_cast<const bf16*>(&u);
    return make_float4((float)b[0], (float)b[1], (float)b[2], (float)b[3]);
  }
  static __device__ __forceinline__ void store(bf16* p, float4 v) {
    bf16 b[4] = {(bf16)v.x, (bf16)v.y, (bf16)v.z, (bf16)v.w};
    *reinterpret_cast<uint2*>(p) = *reinterpret_cast<uint2*>(b);
  }
};

// 8 consecutive elements as two float4 (one 16-byte access for bf16, two for fp32)
template <class T> struct V8;
template <> struct V8<float> {
  static __device__ __forceinline__ void load(const float* p, float4& a, float4& b) {
    a = *reinterpret_cast<const float4*>(p);
    b = *reinterpret_cast<const float4*>(p + 4);
  }
  static __device__ __forceinline__ void store(float* p, float4 a, float4 b) {
    *reinterpret_cast<float4*>(p) = a;
    *reinterpret_cast<float4*>(p + 4) = b;
  }
};
template <> struct V8<bf16> {
  static __device__ __forceinline__ void load(const bf16* p, float4& a, float4& b) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const bf16* e = reinterpret_cast<const bf16*>(&u);
    a = make_float4((float)e[0], (float)e[1], (float)e[2], (float)e[3]);
    b = make_float4((float)e[4], (float)e[5], (float)e[6], (float)e[7]);
  }
  static __device__ __forceinline__ void store(bf16* p, float4 a, float4 b) {
    bf16 e[8] = {(bf16)a.x, (bf16)a.y, (bf16)a.z, (bf16)a.w,
                 (bf16)b.x, (bf16)b.y, (bf16)b.z, (bf16)b.w};
    *reinterpret_cast<uint4*>(p) = *reinterpret_cast<const uint4*>(e);
  }
};

// ---- LayerNorm forward: y = (x - mean) * rstd * g + b, biased variance -------------
// MC = float4 chunks per lane (rows up to 256 MC wide): register arrays sized to the row
template <class T, int MC>
__global__ __launch_bounds__(256) void ln_fwd_kernel(const float* X, int64_t ldx, int64_t rows,
                                                     int n, const T* gam, const T* bet, float eps,
                                                     T* Y, int64_t ldy, float* mean, float* rstd) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int l = threadIdx.x & 63;
  if (row >= rows) return;
  const int nc = n / 4;
  const float* x = X + row * ldx;
  float4 v[MC];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < MC; ++i) {
    const int c = l + 64 * i;
    if (c < nc) {
      v[i] = V4<float>::load(x + 4 * c);
      s += v[i].x + v[i].y + v[i].z + v[i].w;
    }
  }
  const float mu = warp_sum(s) / (float)n;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < MC; ++i) {
    const int c = l + 64 * i;
    if (c < nc) {
      const float a = v[i].x - mu, b = v[i].y - mu, cc = v[i].z - mu, d = v[i].w - mu;
      q += a * a + b * b + cc * cc + d * d;
    }
  }
  const float var = warp_sum(q) / (float)n;
  const float rs = rsqrtf(var + eps);
  T* y = Y + row * ldy;
#pragma unroll
  for (int i = 0; i < MC; ++i) {
    const int c = l + 64 * i;
    if (c < nc) {
      const float4 gg = V4<T>::load(gam + 4 * c), bb = V4<T>::load(bet + 4 * c);
      float4 o;
      o.x = (v[i].x - mu) * rs * gg.x + bb.x;
      o.y = (v[i].y - mu) * rs * gg.y + bb.y;
      o.z = (v[i].z - mu) * rs * gg.z + bb.z;
      o.w = (v[i].w - mu) * rs * gg.w + bb.w;
      V4<T>::store(y + 4 * c, o);
    }
  }
  if (l == 0) {
    if (mean) mean[row] = mu;
    if (rstd) rstd[row] = rs;
  }
}

// ---- LayerNorm backward -------------------------------------------------------------
// dx = rstd * (g*dy - mean(g*dy) - xhat * mean(g*dy*xhat)) + dres, written in fp32
// (and optionally as T for the next GEMM).  Each block owns a contiguous chunk of
// rows (its four waves take every fourth row); the block's sums of dy*xhat and dy
// are combined in LDS in a fixed order and written to part_g / part_b
// [gridDim.x][n] for a deterministic reduction.  With part_c the block also sums the
// dx rows it writes (the bias gradient of the product that produced this residual-stream
// gradient), so no separate pass over dx is needed.
constexpr int LN_BWD_MAX_BLOCKS = 1024;
static_assert(LN_BWD_MAX_BLOCKS <= kPartialRowsMax, "partials must fit the workspace");

template <int MC>
__device__ __forceinline__ void combine_waves(const float4* red, int nc, float* out) {
  for (int c = threadIdx.x; c < nc; c += 256) {
    const int i = c / 64, ll = c % 64;
    float4 t = red[i * 64 + ll];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const float4 u = red[(w * MC + i) * 64 + ll];
      t.x += u.x; t.y += u.y; t.z += u.z; t.w += u.w;
    }
    *reinterpret_cast<float4*>(out + 4 * c) = t;
  }
}

// DY: the type of dY (fp32, or bf16 as the encoder's bf16 input-gradient GEMMs store it)
template <class T, int MC, class DY>
__global__ __launch_bounds__(256) void ln_bwd_kernel(const DY* dY, int64_t ldd, const float* X,
                                                     int64_t ldx, const float* mean,
                                                     const float* rstd, const T* gam, int64_t rows,
                                                     int n, int64_t rows_per_block,
                                                     const float* dres, float* dX, T* dXt,
                                                     float* part_g, float* part_b, float* part_c) {
  __shared__ float4 red[4 * MC * 64];
  __shared__ float4 gms[MC * 64];   // the gain, read from LDS per row (registers go to loads)
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int nc = n / 4;
  float4 ag[MC], ab[MC], ac[MC];
#pragma unroll
  for (int i = 0; i < MC; ++i) ag[i] = ab[i] = ac[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int c = threadIdx.x; c < nc; c += 256) gms[c] = V4<T>::load(gam + 4 * c);
  __syncthreads();
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = min(rows, r0 + rows_per_block);
  for (int64_t row = r0 + wave; row < r1; row += 4) {
    const float mu = mean[row], rs = rstd[row];
    // every operand of the row is requested before any is used
    float4 x[MC], dy[MC];
#pragma unroll
    for (int i = 0; i < MC; ++i) {
      const int c = l + 64 * i;
      if (c < nc) {
        x[i] = V4<float>::load(X + row * ldx + 4 * c);
        dy[i] = V4<DY>::load(dY + row * ldd + 4 * c);
      }
    }
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int i = 0; i < MC; ++i) {
      const int c = l + 64 * i;
      if (c < nc) {
        x[i] = make_float4((x[i].x - mu) * rs, (x[i].y - mu) * rs, (x[i].z - mu) * rs,
                           (x[i].w - mu) * rs);   // now xhat
        const float4 gm = gms[c];
        const float4 gd = make_float4(dy[i].x * gm.x, dy[i].y * gm.y, dy[i].z * gm.z,
                                      dy[i].w * gm.w);
        s1 += gd.x + gd.y + gd.z + gd.w;
        s2 += gd.x * x[i].x + gd.y * x[i].y + gd.z * x[i].z + gd.w * x[i].w;
        ag[i].x += dy[i].x * x[i].x; ag[i].y += dy[i].y * x[i].y;
        ag[i].z += dy[i].z * x[i].z; ag[i].w += dy[i].w * x[i].w;
        ab[i].x += dy[i].x; ab[i].y += dy[i].y; ab[i].z += dy[i].z; ab[i].w += dy[i].w;
      }
    }
    if (!dX) continue;   // affine gradients only (no input gradient wanted)
    s1 = warp_sum(s1) / (float)n;
    s2 = warp_sum(s2) / (float)n;
#pragma unroll
    for (int i = 0; i < MC; ++i) {
      const int c = l + 64 * i;
      if (c < nc) {
        const float4 gm = gms[c];
        const float4 dr =
            dres ? V4<float>::load(dres + row * ldx + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
        float4 o;
        o.x = rs * (dy[i].x * gm.x - s1 - x[i].x * s2) + dr.x;
        o.y = rs * (dy[i].y * gm.y - s1 - x[i].y * s2) + dr.y;
        o.z = rs * (dy[i].z * gm.z - s1 - x[i].z * s2) + dr.z;
        o.w = rs * (dy[i].w * gm.w - s1 - x[i].w * s2) + dr.w;
        V4<float>::store(dX + row * ldx + 4 * c, o);
        if (dXt) V4<T>::store(dXt + row * ldx + 4 * c, o);
        ac[i].x += o.x; ac[i].y += o.y; ac[i].z += o.z; ac[i].w += o.w;
      }
    }
  }
  // combine the four waves in a fixed order: gain sums, then shift sums
#pragma unroll
  for (int i = 0; i < MC; ++i) red[(wave * MC + i) * 64 + l] = ag[i];
  __syncthreads();
  combine_waves<MC>(red, nc, part_g + (int64_t)blockIdx.x * n);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MC; ++i) red[(wave * MC + i) * 64 + l] = ab[i];
  __syncthreads();
  combine_waves<MC>(red, nc, part_b + (int64_t)blockIdx.x * n);
  if (!part_c || !dX) return;   // uniform over the grid
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MC; ++i) red[(wave * MC + i) * 64 + l] = ac[i];
  __syncthreads();
  combine_waves<MC>(red, nc, part_c + (int64_t)blockIdx.x * n);
}

// ---- column sums: part[b][c] = sum of X[r][c] over row chunk b ----------------------
constexpr int COLSUM_MAX_CHUNKS = 256;
static_assert(COLSUM_MAX_CHUNKS <= kPartialRowsMax, "partials must fit the workspace");

template <class T>
__global__ void colsum_partial_kernel(const T* X, int64_t ld, int64_t rows, int n,
                                      int64_t rows_per_chunk, float* part) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= n) return;
  const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
  const int64_t r1 = min(rows, r0 + rows_per_chunk);
  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
  int64_t r = r0;
  for (; r + 4 <= r1; r += 4) {
    s0 += to_f(X[r * ld + c]);
    s1 += to_f(X[(r + 1) * ld + c]);
    s2 += to_f(X[(r + 2) * ld + c]);
    s3 += to_f(X[(r + 3) * ld + c]);
  }
  for (; r < r1; ++r) s0 += to_f(X[r * ld + c]);
  part[(int64_t)blockIdx.y * n + c] = (s0 + s1) + (s2 + s3);
}

// Vector form (n % 8 == 0, 16-byte aligned rows): lane l of a wave sums columns
// [8l, 8l + 8) of a 512-column strip over every fourth row of the block's row chunk
// (four of its rows in flight per iteration); the four waves are combined in LDS in a
// fixed order.
template <class T>
__global__ __launch_bounds__(256) void colsum_vec_kernel(const T* X, int64_t ld, int64_t rows,
                                                         int n, int64_t rows_per_chunk,
                                                         float* part) {
  __shared__ float red[4][512];
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int c = blockIdx.x * 512 + 8 * l;
  const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
  const int64_t r1 = min(rows, r0 + rows_per_chunk);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (c < n) {
    int64_t r = r0 + wave;
    for (; r + 12 < r1; r += 16) {
      const T* p0 = X + r * ld + c;
      float4 a0, b0, a1, b1, a2, b2, a3, b3;
      V8<T>::load(p0, a0, b0);
      V8<T>::load(p0 + 4 * ld, a1, b1);
      V8<T>::load(p0 + 8 * ld, a2, b2);
      V8<T>::load(p0 + 12 * ld, a3, b3);
      acc[0] += (a0.x + a1.x) + (a2.x + a3.x); acc[1] += (a0.y + a1.y) + (a2.y + a3.y);
      acc[2] += (a0.z + a1.z) + (a2.z + a3.z); acc[3] += (a0.w + a1.w) + (a2.w + a3.w);
      acc[4] += (b0.x + b1.x) + (b2.x + b3.x); acc[5] += (b0.y + b1.y) + (b2.y + b3.y);
      acc[6] += (b0.z + b1.z) + (b2.z + b3.z); acc[7] += (b0.w + b1.w) + (b2.w + b3.w);
    }
    for (; r < r1; r += 4) {
      float4 a, b;
      V8<T>::load(X + r * ld + c, a, b);
      acc[0] += a.x; acc[1] += a.y; acc[2] += a.z; acc[3] += a.w;
      acc[4] += b.x; acc[5] += b.y; acc[6] += b.z; acc[7] += b.w;
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[wave][8 * l + e] = acc[e];
  __syncthreads();
  for (int j = threadIdx.x; j < 512; j += 256) {
    const int cc = blockIdx.x * 512 + j;
    if (cc < n)
      part[(int64_t)blockIdx.y * n + cc] = (red[0][j] + red[1][j]) + (red[2][j] + red[3][j]);
  }
}

// out[c] += sum_b part[b][c], b < nb, for up to two (part, out) sets (blockIdx.z), in two
// fixed-order stages so that the result depends only on nb, never on timing.
// Stage 1: block (x, g) sums the partial rows of chunk g, [g * chunk, (g + 1) * chunk), for
// columns 64x..64x+63 (wave w takes rows w, w + 4, ..., four loads in flight; the four wave
// sums are added in order) and writes the chunk sum over the chunk's first row: only this
// block reads or writes that part of the buffer.  Stage 2 adds the chunk sums in chunk order.
struct PartialSet {
  float* part[3];
  float* out[3];
};
constexpr int RED_CHUNKS = 16;   // at most this many chunks per set

int64_t reduce_chunk_rows(int64_t nb) {
  const int64_t c = (nb + RED_CHUNKS - 1) / RED_CHUNKS;
  return c < 16 ? 16 : c;
}

__global__ __launch_bounds__(256) void reduce_partials_stage1(PartialSet ps, int64_t nb, int n,
                                                              int64_t chunk) {
  __shared__ float red[4][64];
  float* part = ps.part[blockIdx.z];
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int c = blockIdx.x * 64 + l;
  const int64_t r0 = (int64_t)blockIdx.y * chunk;
  const int64_t r1 = min(nb, r0 + chunk);
  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
  if (c < n) {
    int64_t b = r0 + w;
    for (; b + 12 < r1; b += 16) {
      s0 += part[b * n + c];
      s1 += part[(b + 4) * n + c];
      s2 += part[(b + 8) * n + c];
      s3 += part[(b + 12) * n + c];
    }
    for (; b < r1; b += 4) s0 += part[b * n + c];
  }
  red[w][l] = (s0 + s1) + (s2 + s3);
  __syncthreads();
  if (w == 0 && c < n) part[r0 * n + c] = (red[0][l] + red[1][l]) + (red[2][l] + red[3][l]);
}

__global__ __launch_bounds__(64) void reduce_partials_stage2(PartialSet ps, int64_t nb, int n,
                                                             int64_t chunk) {
  const float* part = ps.part[blockIdx.z];
  const int c = blockIdx.x * 64 + threadIdx.x;
  if (c >= n) return;
  float t = 0.f;
  for (int64_t r = 0; r < nb; r += chunk) t += part[r * n + c];
  ps.out[blockIdx.z][c] += t;
}

// Launch both stages for the non-null sets among (p0, o0), (p1, o1), (p2, o2).
void reduce_partials(float* p0, float* o0, float* p1, float* o1, float* p2, float* o2,
                     int64_t nb, int n, hipStream_t s) {
  PartialSet ps{};
  int z = 0;
  if (o0) ps.part[z] = p0, ps.out[z] = o0, ++z;
  if (o1) ps.part[z] = p1, ps.out[z] = o1, ++z;
  if (o2) ps.part[z] = p2, ps.out[z] = o2, ++z;
  if (!z || nb <= 0 || n <= 0) return;
  const int64_t chunk = reduce_chunk_rows(nb);
  const unsigned cx = (unsigned)((n + 63) / 64), g = (unsigned)((nb + chunk - 1) / chunk);
  hipLaunchKernelGGL(reduce_partials_stage1, dim3(cx, g, (unsigned)z), dim3(256), 0, s, ps, nb, n,
                     chunk);
  hipLaunchKernelGGL(reduce_partials_stage2, dim3(cx, 1, (unsigned)z), dim3(64), 0, s, ps, nb, n,
                     chunk);
}

// out[m][n] += sum_s part[s][m][n], four columns per thread (N % 4 == 0, ldo % 4 == 0,
// M * N / 4 < 2^31)
__global__ void splitk_reduce4_kernel(const float* part, int splits, int M, int N4, float* out,
                                      int64_t ldo) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= M * N4) return;
  const int m = i / N4, c = i - m * N4;
  const int64_t stride = (int64_t)M * N4;
  const float4* p = reinterpret_cast<const float4*>(part) + i;
  float4 acc = p[0];
  for (int k = 1; k < splits; ++k) {
    const float4 v = p[k * stride];
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  float4* o = reinterpret_cast<float4*>(out + (int64_t)m * ldo) + c;
  float4 r = *o;
  r.x += acc.x; r.y += acc.y; r.z += acc.z; r.w += acc.w;
  *o = r;
}

// out[m][n] += sum_s part[s][m][n]   (partials are dense [M][N])
__global__ void splitk_reduce_kernel(const float* part, int splits, int64_t M, int64_t N,
                                     float* out, int64_t ldo) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= M * N) return;
  const int64_t m = i / N, n = i % N;
  float s = 0.f;
  for (int k = 0; k < splits; ++k) s += part[(int64_t)k * M * N + i];
  out[m * ldo + n] += s;
}

// ---- padding copy: dst[r][c] = c < K ? src[r][c] : 0, for c < Kp --------------------
template <class T>
__global__ void pad_cols_kernel(const T* src, int64_t rows, int K, T* dst, int Kp) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * Kp) return;
  const int64_t r = i / Kp;
  const int c = (int)(i % Kp);
  dst[i] = c < K ? src[r * K + c] : from_f<T>(0.f);
}

// ---- batched transpose: dst[c][r] = src[r][c], element bits copied ------------------
// 64x64 tiles through LDS; block b takes tile b - first_tile of the job it falls in.
// VEC elements per 16-byte access when every job allows it (VEC = 1: scalar accesses).
struct TJobs {
  TJob j[kMaxTJobs];
  int64_t first[kMaxTJobs + 1];   // first tile of each job; first[n] = total tiles
  int n;
};

template <class U, int VEC>
__global__ __launch_bounds__(256) void transpose_kernel(TJobs jb) {
  __shared__ U tile[64][65];
  const int64_t b = blockIdx.x;
  int ji = 0;
  while (ji + 1 < jb.n && b >= jb.first[ji + 1]) ++ji;
  const TJob& J = jb.j[ji];
  const int64_t tix = b - jb.first[ji];
  const int tiles_c = (J.cols + 63) / 64;
  const int r0 = (int)(tix / tiles_c) * 64, c0 = (int)(tix % tiles_c) * 64;
  const U* src = reinterpret_cast<const U*>(J.src);
  U* dst = reinterpret_cast<U*>(J.dst);
  constexpr int TPR = 64 / VEC;          // threads per 64-element line
  constexpr int LPP = 256 / TPR;         // lines per pass
  const int t = threadIdx.x;
  const int li = t / TPR, ci = (t % TPR) * VEC;
  for (int rr = li; rr < 64; rr += LPP) {       // load src rows r0+rr, cols c0+ci..
    const int r = r0 + rr, c = c0 + ci;
    // the source row whose values land at stored row r
    const int rs = r < J.perm_rows ? r - r % J.perm_d + rope_component(r % J.perm_d, J.perm_d) : r;
    if constexpr (VEC > 1) {
      if (r < J.rows && c < J.cols) {
        const uint4 v = *reinterpret_cast<const uint4*>(src + (int64_t)rs * J.lds + c);
        const U* e = reinterpret_cast<const U*>(&v);
#pragma unroll
        for (int k = 0; k < VEC; ++k) tile[rr][ci + k] = e[k];
      }
    } else {
      if (r < J.rows && c < J.cols) tile[rr][ci] = src[(int64_t)rs * J.lds + c];
    }
  }
  __syncthreads();
  for (int cc = li; cc < 64; cc += LPP) {       // store dst rows c0+cc, cols r0+ci..
    const int c = c0 + cc, r = r0 + ci;
    if constexpr (VEC > 1) {
      if (c < J.cols && r < J.rows) {
        uint4 v;
        U* e = reinterpret_cast<U*>(&v);
#pragma unroll
        for (int k = 0; k < VEC; ++k) e[k] = tile[ci + k][cc];
        *reinterpret_cast<uint4*>(dst + (int64_t)c * J.ldd + r) = v;
      }
    } else {
      if (c < J.cols && r < J.rows) dst[(int64_t)c * J.ldd + r] = tile[ci][cc];
    }
  }
}

// ---- 2D rotary position, in place on the q and k column blocks -------------------
// pos[r] = y << 16 | x.  tab[p * q4 + k] = (cos, sin) of p * theta^(-4k/d) (k < q4 = d/4,
// computed on the host in double).  Pair (j, j + d/2) of each head rotates by the
// angle of y (j < d/4) or of x (j >= d/4).  Each thread rotates 4 consecutive pairs.
template <class T>
__global__ void rope_kernel(T* qk, int64_t ld, int64_t rows, int heads, int d, int kcol,
                            const int32_t* pos, const float2* tab, int inverse) {
  const int half = d / 2, quarter = d / 4;
  const int groups = half / 4;                       // 4-pair groups per head
  const int64_t per_row = (int64_t)2 * heads * groups;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * per_row) return;
  const int64_t r = i / per_row;
  int rem = (int)(i % per_row);
  const int which = rem / (heads * groups);
  rem %= heads * groups;
  const int hd = rem / groups, j0 = 4 * (rem % groups);
  const uint32_t pp = (uint32_t)pos[r];
  T* v = qk + r * ld + (which ? kcol : 0) + hd * d;
  const float4 a = V4<T>::load(v + j0), b = V4<T>::load(v + j0 + half);
  const float x1[4] = {a.x, a.y, a.z, a.w}, x2[4] = {b.x, b.y, b.z, b.w};
  float o1[4], o2[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int j = j0 + e;
    const int coord = (int)((j < quarter) ? (pp >> 16) : (pp & 0xFFFFu));
    const float2 cs = tab[coord * quarter + (j < quarter ? j : j - quarter)];
    const float sn = inverse ? -cs.y : cs.y;
    o1[e] = x1[e] * cs.x - x2[e] * sn;
    o2[e] = x2[e] * cs.x + x1[e] * sn;
  }
  V4<T>::store(v + j0, make_float4(o1[0], o1[1], o1[2], o1[3]));
  V4<T>::store(v + j0 + half, make_float4(o2[0], o2[1], o2[2], o2[3]));
}

// Eight consecutive pairs per thread (16-byte accesses; needs d % 16 == 0).
template <class T>
__global__ void rope8_kernel(T* qk, int64_t ld, int64_t rows, int heads, int d, int kcol,
                             const int32_t* pos, const float2* tab, int inverse) {
  const int half = d / 2, quarter = d / 4;
  const int groups = half / 8;                       // 8-pair groups per head
  const int per_row = 2 * heads * groups;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * per_row) return;
  const int64_t r = i / per_row;
  int rem = (int)(i - r * per_row);
  const int which = rem / (heads * groups);
  rem -= which * heads * groups;
  const int hd = rem / groups, j0 = 8 * (rem - hd * groups);
  const uint32_t pp = (uint32_t)pos[r];
  T* v = qk + r * ld + (which ? kcol : 0) + hd * d;
  float4 a0, a1, b0, b1;
  V8<T>::load(v + j0, a0, a1);
  V8<T>::load(v + j0 + half, b0, b1);
  const float x1[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
  const float x2[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
  float o1[8], o2[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int j = j0 + e;
    const int coord = (int)((j < quarter) ? (pp >> 16) : (pp & 0xFFFFu));
    const float2 cs = tab[coord * quarter + (j < quarter ? j : j - quarter)];
    const float sn = inverse ? -cs.y : cs.y;
    o1[e] = x1[e] * cs.x - x2[e] * sn;
    o2[e] = x2[e] * cs.x + x1[e] * sn;
  }
  V8<T>::store(v + j0, make_float4(o1[0], o1[1], o1[2], o1[3]),
               make_float4(o1[4], o1[5], o1[6], o1[7]));
  V8<T>::store(v + j0 + half, make_float4(o2[0], o2[1], o2[2], o2[3]),
               make_float4(o2[4], o2[5], o2[6], o2[7]));
}

// ---- bit-exact row scatter / gather ---------------------------------------------------
// dst row idx[j] <- src row j (scatter) or dst row j <- src row idx[j] (gather).
// Rows with an index outside [0, n_rows) are skipped.
template <class U, bool SCATTER>
__global__ void rows_copy_kernel(const U* __restrict__ src, U* __restrict__ dst,
                                 const int64_t* __restrict__ idx, int64_t n_idx, int64_t units,
                                 int64_t n_rows) {
  const int64_t total = n_idx * units;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t j = i / units, c = i % units;
    const int64_t t = idx[j];
    if (t < 0 || t >= n_rows) continue;
    if (SCATTER)
      dst[t * units + c] = src[j * units + c];
    else
      dst[j * units + c] = src[t * units + c];
  }
}

// range + uniqueness check of placeholder indices: marks[t] counts hits (int32,
// zero-initialised by the caller's stream), status[0] |= 1 out of range, 2 repeated.
__global__ void idx_mark_kernel(const int64_t* idx, int64_t n, int64_t n_rows, int32_t* marks,
                                int32_t* status) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  const int64_t t = idx[j];
  if (t < 0 || t >= n_rows) {
    atomicOr(status, 1);
    return;
  }
  if (atomicAdd(marks + t, 1) != 0) atomicOr(status, 2);
}

__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

inline int blocks_for(int64_t n, int t = 256) { return (int)((n + t - 1) / t); }

// Blocks of `kernel` resident on the whole device at once (one full round), from the
// occupancy calculator; computed once per (signature, TAG) -- TAG tells apart
// instantiations that share a signature.
template <int TAG, class K>
int64_t resident_blocks(K kernel, int threads) {
  static const int64_t n = [&] {
    int dev = 0, cus = 0, per = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, threads, 0) != hipSuccess)
      return (int64_t)1 << 30;   // unknown: no cap
    return (int64_t)(per > 0 ? per : 1) * (cus > 0 ? cus : 1);
  }();
  return n;
}

// calls f(integral_constant<int, MC>) for the float4-per-lane count of a LayerNorm row
template <class F>
bool dispatch_mc(int mc, F&& f) {
  static_assert(MAXC == 8, "one case per chunk count up to MAXC");
  switch (mc) {
    case 1: f(std::integral_constant<int, 1>{}); return true;
    case 2: f(std::integral_constant<int, 2>{}); return true;
    case 3: f(std::integral_constant<int, 3>{}); return true;
    case 4: f(std::integral_constant<int, 4>{}); return true;
    case 5: f(std::integral_constant<int, 5>{}); return true;
    case 6: f(std::integral_constant<int, 6>{}); return true;
    case 7: f(std::integral_constant<int, 7>{}); return true;
    case 8: f(std::integral_constant<int, 8>{}); return true;
  }
  return false;
}

}  // namespace

hipError_t layernorm_fwd(int dtype, const float* X, int64_t ldx, int64_t rows, int n,
                         const void* g, const void* b, float eps, void* Y, int64_t ldy,
                         float* mean, float* rstd, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 3) / 4));
  const int mc = (n / 4 + 63) / 64;
  auto go = [&](auto MCc) {
    constexpr int MC = decltype(MCc)::value;
    if (dtype == DT_BF16)
      hipLaunchKernelGGL((ln_fwd_kernel<bf16, MC>), grid, dim3(256), 0, s, X, ldx, rows, n,
                         (const bf16*)g, (const bf16*)b, eps, (bf16*)Y, ldy, mean, rstd);
    else
      hipLaunchKernelGGL((ln_fwd_kernel<float, MC>), grid, dim3(256), 0, s, X, ldx, rows, n,
                         (const float*)g, (const float*)b, eps, (float*)Y, ldy, mean, rstd);
  };
  if (!dispatch_mc(mc, go)) return hipErrorInvalidValue;
  return hipGetLastError();
}

int64_t layernorm_bwd_partial_rows(int64_t rows) {
  const int64_t b = (rows + 3) / 4;
  return b < LN_BWD_MAX_BLOCKS ? b : LN_BWD_MAX_BLOCKS;
}

hipError_t layernorm_bwd_partials(int dtype, const void* dY, int dy_dtype, int64_t ldd,
                                  const float* X, int64_t ldx, const float* mean, const float* rstd,
                                  const void* g, int64_t rows, int n, const float* dres, float* dX,
                                  void* dXt, float* part_g, float* part_b, float* part_c,
                                  int64_t* blocks, hipStream_t s) {
  *blocks = 0;
  if (rows == 0) return hipSuccess;
  // one round of resident blocks (never more than the partial rows the caller sized)
  const int mc = (n / 4 + 63) / 64;
  int64_t nblk = 0;
  float* pc = dX ? part_c : nullptr;
  auto go = [&](auto MCc) {
    constexpr int MC = decltype(MCc)::value;
    auto launch = [&](auto kern, auto dy, auto gptr, auto dxt) {
      nblk = std::min(layernorm_bwd_partial_rows(rows), resident_blocks<MC>(kern, 256));
      const int64_t rpb = (rows + nblk - 1) / nblk;
      hipLaunchKernelGGL(kern, dim3((unsigned)nblk), dim3(256), 0, s, dy, ldd, X, ldx, mean, rstd,
                         gptr, rows, n, rpb, dres, dX, dxt, part_g, part_b, pc);
    };
    if (dtype == DT_BF16 && dy_dtype == DT_BF16)
      launch(ln_bwd_kernel<bf16, MC, bf16>, (const bf16*)dY, (const bf16*)g, (bf16*)dXt);
    else if (dtype == DT_BF16)
      launch(ln_bwd_kernel<bf16, MC, float>, (const float*)dY, (const bf16*)g, (bf16*)dXt);
    else
      launch(ln_bwd_kernel<float, MC, float>, (const float*)dY, (const float*)g, (float*)dXt);
  };
  if (!dispatch_mc(mc, go)) return hipErrorInvalidValue;
  *blocks = nblk;
  return hipGetLastError();
}

hipError_t partials_reduce(float* part, float* out, int64_t rows, int n, hipStream_t s) {
  reduce_partials(part, out, nullptr, nullptr, nullptr, nullptr, rows, n, s);
  return hipGetLastError();
}

hipError_t layernorm_bwd_reduce(float* part_g, float* grad_g, float* part_b, float* grad_b,
                                float* part_c, float* grad_c, int64_t blocks, int n,
                                hipStream_t s) {
  reduce_partials(part_g, grad_g, part_b, grad_b, part_c, grad_c, blocks, n, s);
  return hipGetLastError();
}

hipError_t layernorm_bwd(int dtype, const float* dY, int64_t ldd, const float* X, int64_t ldx,
                         const float* mean, const float* rstd, const void* g, int64_t rows, int n,
                         const float* dres, float* dX, void* dXt, float* part_g, float* part_b,
                         float* part_c, float* grad_g, float* grad_b, float* grad_c,
                         hipStream_t s) {
  if (!dX || !grad_c) part_c = grad_c = nullptr;
  int64_t nb = 0;
  hipError_t r = layernorm_bwd_partials(dtype, dY, DT_F32, ldd, X, ldx, mean, rstd, g, rows, n,
                                        dres, dX, dXt, part_g, part_b, part_c, &nb, s);
  if (r != hipSuccess) return r;
  return layernorm_bwd_reduce(part_g, grad_g, part_b, grad_b, part_c, grad_c, nb, n, s);
}

int64_t colsum_partial_rows(int64_t rows) {
  const int64_t c = (rows + 31) / 32;
  return c < COLSUM_MAX_CHUNKS ? c : COLSUM_MAX_CHUNKS;
}

hipError_t colsum_accumulate(int dtype_in, const void* X, int64_t ld, int64_t rows, int n,
                             float* part, float* out, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const int64_t nb = colsum_partial_rows(rows);
  const int64_t rpc = (rows + nb - 1) / nb;
  const bool vec = n % 8 == 0 && ld % 8 == 0 && (reinterpret_cast<uintptr_t>(X) & 15) == 0;
  if (vec) {
    const dim3 grid((unsigned)((n + 511) / 512), (unsigned)nb);
    if (dtype_in == DT_BF16)
      hipLaunchKernelGGL(colsum_vec_kernel<bf16>, grid, dim3(256), 0, s, (const bf16*)X, ld, rows,
                         n, rpc, part);
    else
      hipLaunchKernelGGL(colsum_vec_kernel<float>, grid, dim3(256), 0, s, (const float*)X, ld,
                         rows, n, rpc, part);
  } else {
    const dim3 grid((unsigned)blocks_for(n), (unsigned)nb);
    if (dtype_in == DT_BF16)
      hipLaunchKernelGGL(colsum_partial_kernel<bf16>, grid, dim3(256), 0, s, (const bf16*)X, ld,
                         rows, n, rpc, part);
    else
      hipLaunchKernelGGL(colsum_partial_kernel<float>, grid, dim3(256), 0, s, (const float*)X, ld,
                         rows, n, rpc, part);
  }
  reduce_partials(part, out, nullptr, nullptr, nullptr, nullptr, nb, n, s);
  return hipGetLastError();
}

hipError_t splitk_reduce(const float* part, int splits, int64_t M, int64_t N, float* out,
                         int64_t ldo, hipStream_t s) {
  if (M * N == 0) return hipSuccess;
  if (N % 4 == 0 && ldo % 4 == 0 && M * N / 4 < (int64_t)1 << 31 &&
      (reinterpret_cast<uintptr_t>(part) & 15) == 0 && (reinterpret_cast<uintptr_t>(out) & 15) == 0) {
    hipLaunchKernelGGL(splitk_reduce4_kernel, dim3(blocks_for(M * N / 4)), dim3(256), 0, s, part,
                       splits, (int)M, (int)(N / 4), out, ldo);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks_for(M * N)), dim3(256), 0, s, part, splits,
                     M, N, out, ldo);
  return hipGetLastError();
}

hipError_t pad_cols(int dtype, const void* src, int64_t rows, int K, void* dst, int Kp,
                    hipStream_t s) {
  const int64_t n = rows * Kp;
  if (n == 0) return hipSuccess;
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(pad_cols_kernel<bf16>, dim3(blocks_for(n)), dim3(256), 0, s,
                       (const bf16*)src, rows, K, (bf16*)dst, Kp);
  else
    hipLaunchKernelGGL(pad_cols_kernel<float>, dim3(blocks_for(n)), dim3(256), 0, s,
                       (const float*)src, rows, K, (float*)dst, Kp);
  return hipGetLastError();
}

hipError_t transpose_batch(int dtype, const TJob* jobs, int n, hipStream_t s) {
  if (n < 0 || n > kMaxTJobs) return hipErrorInvalidValue;
  TJobs jb{};
  jb.n = 0;
  int64_t tiles = 0;
  const int esz = dtype == DT_BF16 ? 2 : 4;
  const int vec = 16 / esz;
  bool vok = true;
  for (int i = 0; i < n; ++i) {
    const TJob& J = jobs[i];
    if (J.rows <= 0 || J.cols <= 0) continue;
    if (J.lds < J.cols || J.ldd < J.rows) return hipErrorInvalidValue;
    if (J.perm_rows > 0 && (J.perm_d <= 0 || J.perm_d % 2 || J.perm_rows % J.perm_d ||
                            J.perm_rows > J.rows))
      return hipErrorInvalidValue;
    jb.j[jb.n] = J;
    jb.first[jb.n] = tiles;
    tiles += (int64_t)((J.rows + 63) / 64) * ((J.cols + 63) / 64);
    ++jb.n;
    vok = vok && J.rows % vec == 0 && J.cols % vec == 0 && J.lds % vec == 0 && J.ldd % vec == 0 &&
          (reinterpret_cast<uintptr_t>(J.src) & 15) == 0 && (reinterpret_cast<uintptr_t>(J.dst) & 15) == 0;
  }
  jb.first[jb.n] = tiles;
  if (tiles == 0) return hipSuccess;
  const dim3 grid((unsigned)tiles);
  if (dtype == DT_BF16) {
    if (vok) hipLaunchKernelGGL((transpose_kernel<uint16_t, 8>), grid, dim3(256), 0, s, jb);
    else hipLaunchKernelGGL((transpose_kernel<uint16_t, 1>), grid, dim3(256), 0, s, jb);
  } else {
    if (vok) hipLaunchKernelGGL((transpose_kernel<uint32_t, 4>), grid, dim3(256), 0, s, jb);
    else hipLaunchKernelGGL((transpose_kernel<uint32_t, 1>), grid, dim3(256), 0, s, jb);
  }
  return hipGetLastError();
}

hipError_t rope(int dtype, void* qk, int64_t ld, int64_t rows, int heads, int d, int kcol,
                const int32_t* pos, const float* tab, int inverse, hipStream_t s) {
  const int64_t n = rows * 2 * heads * (d / 8);  // (q and k) x heads x 4-pair groups
  if (n == 0) return hipSuccess;
  const float2* t = reinterpret_cast<const float2*>(tab);
  const int esz = dtype == DT_BF16 ? 2 : 4;
  if (d % 16 == 0 && (ld * esz) % 16 == 0 && (kcol * esz) % 16 == 0 &&
      (reinterpret_cast<uintptr_t>(qk) & 15) == 0) {   // eight pairs per thread
    const int64_t n8 = rows * 2 * heads * (d / 16);
    if (dtype == DT_BF16)
      hipLaunchKernelGGL(rope8_kernel<bf16>, dim3(blocks_for(n8)), dim3(256), 0, s, (bf16*)qk, ld,
                         rows, heads, d, kcol, pos, t, inverse);
    else
      hipLaunchKernelGGL(rope8_kernel<float>, dim3(blocks_for(n8)), dim3(256), 0, s, (float*)qk,
                         ld, rows, heads, d, kcol, pos, t, inverse);
    return hipGetLastError();
  }
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(rope_kernel<bf16>, dim3(blocks_for(n)), dim3(256), 0, s, (bf16*)qk, ld,
                       rows, heads, d, kcol, pos, t, inverse);
  else
    hipLaunchKernelGGL(rope_kernel<float>, dim3(blocks_for(n)), dim3(256), 0, s, (float*)qk, ld,
                       rows, heads, d, kcol, pos, t, inverse);
  return hipGetLastError();
}

hipError_t rows_copy(bool scatter, const void* src, void* dst, const int64_t* idx, int64_t n_idx,
                     int64_t row_bytes, int64_t n_rows, hipStream_t s) {
  if (n_idx == 0 || row_bytes == 0) return hipSuccess;
  const uintptr_t al = (uintptr_t)src | (uintptr_t)dst | (uintptr_t)row_bytes;
  int unit = (al % 16 == 0) ? 16 : (al % 8 == 0) ? 8 : (al % 4 == 0) ? 4 : (al % 2 == 0) ? 2 : 1;
  const int64_t units = row_bytes / unit;
  const int64_t total = n_idx * units;
  const int grid = (int)(blocks_for(total) < 4096 ? blocks_for(total) : 4096);
#define MPIPE_RC(U)                                                                              \
  if (scatter)                                                                                  \
    hipLaunchKernelGGL((rows_copy_kernel<U, true>), dim3(grid), dim3(256), 0, s, (const U*)src, \
                       (U*)dst, idx, n_idx, units, n_rows);                                      \
  else                                                                                          \
    hipLaunchKernelGGL((rows_copy_kernel<U, false>), dim3(grid), dim3(256), 0, s, (const U*)src,\
                       (U*)dst, idx, n_idx, units, n_rows);
  switch (unit) {
    case 16: MPIPE_RC(uint4) break;
    case 8: MPIPE_RC(uint2) break;
    case 4: MPIPE_RC(uint32_t) break;
    case 2: MPIPE_RC(uint16_t) break;
    default: MPIPE_RC(uint8_t) break;
  }
#undef MPIPE_RC
  return hipGetLastError();
}

hipError_t check_indices(const int64_t* idx, int64_t n, int64_t n_rows, int32_t* marks,
                         int32_t* status, hipStream_t s) {
  hipLaunchKernelGGL(fill_i32_kernel, dim3(blocks_for(n_rows + 1)), dim3(256), 0, s, marks,
                     n_rows, 0);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(32), 0, s, status, (int64_t)1, 0);
  if (n > 0)
    hipLaunchKernelGGL(idx_mark_kernel, dim3(blocks_for(n)), dim3(256), 0, s, idx, n, n_rows,
                       marks, status);
  return hipGetLastError();
}

}  // namespace mpipe
