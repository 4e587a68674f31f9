// Row-wise and element-wise kernels of the encoder step: LayerNorm forward and
// backward (fp32 statistics, one wave64 per row, wavefront reductions), 2D
// rotary position, operand padding, deterministic column reductions for the
// bias / LayerNorm-affine gradients, the split-K reduction of weight
// gradients, and the bit-exact placeholder row scatter / gather.
#include "common.h"
#include "internal.h"

namespace mpipe {
namespace {

constexpr int MAXC = 8;  // float4 chunks per lane: rows up to 64 * 4 * 8 = 2048 wide

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

// ---- LayerNorm forward: y = (x - mean) * rstd * g + b, biased variance -------------
template <class T>
__global__ __launch_bounds__(256) void ln_fwd_kernel(const float* X, int64_t ldx, int64_t rows,
                                                     int n, const T* gam, const T* bet, float eps,
                                                     T* Y, int64_t ldy, float* mean, float* rstd) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int l = threadIdx.x & 63;
  if (row >= rows) return;
  const int nc = n / 4;
  const float* x = X + row * ldx;
  float4 v[MAXC];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = l + 64 * i;
    if (c < nc) {
      v[i] = V4<float>::load(x + 4 * c);
      s += v[i].x + v[i].y + v[i].z + v[i].w;
    }
  }
  const float mu = warp_sum(s) / (float)n;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
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
  for (int i = 0; i < MAXC; ++i) {
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
// [gridDim.x][n] for a deterministic reduction.
constexpr int LN_BWD_MAX_BLOCKS = 512;

__device__ __forceinline__ void combine_waves(const float4* red, int nc, float* out) {
  for (int c = threadIdx.x; c < nc; c += 256) {
    const int i = c / 64, ll = c % 64;
    float4 t = red[i * 64 + ll];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const float4 u = red[(w * MAXC + i) * 64 + ll];
      t.x += u.x; t.y += u.y; t.z += u.z; t.w += u.w;
    }
    *reinterpret_cast<float4*>(out + 4 * c) = t;
  }
}

template <class T>
__global__ __launch_bounds__(256) void ln_bwd_kernel(const float* dY, int64_t ldd, const float* X,
                                                     int64_t ldx, const float* mean,
                                                     const float* rstd, const T* gam, int64_t rows,
                                                     int n, int64_t rows_per_block,
                                                     const float* dres, float* dX, T* dXt,
                                                     float* part_g, float* part_b) {
  __shared__ float4 red[4 * MAXC * 64];
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int nc = n / 4;
  float4 ag[MAXC], ab[MAXC], gm[MAXC];
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    ag[i] = ab[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    const int c = l + 64 * i;
    if (c < nc) gm[i] = V4<T>::load(gam + 4 * c);
  }
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = min(rows, r0 + rows_per_block);
  for (int64_t row = r0 + wave; row < r1; row += 4) {
    const float mu = mean[row], rs = rstd[row];
    float4 xh[MAXC], dy[MAXC];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = l + 64 * i;
      if (c < nc) {
        const float4 x = V4<float>::load(X + row * ldx + 4 * c);
        dy[i] = V4<float>::load(dY + row * ldd + 4 * c);
        xh[i] = make_float4((x.x - mu) * rs, (x.y - mu) * rs, (x.z - mu) * rs, (x.w - mu) * rs);
        const float4 gd = make_float4(dy[i].x * gm[i].x, dy[i].y * gm[i].y, dy[i].z * gm[i].z,
                                      dy[i].w * gm[i].w);
        s1 += gd.x + gd.y + gd.z + gd.w;
        s2 += gd.x * xh[i].x + gd.y * xh[i].y + gd.z * xh[i].z + gd.w * xh[i].w;
        ag[i].x += dy[i].x * xh[i].x; ag[i].y += dy[i].y * xh[i].y;
        ag[i].z += dy[i].z * xh[i].z; ag[i].w += dy[i].w * xh[i].w;
        ab[i].x += dy[i].x; ab[i].y += dy[i].y; ab[i].z += dy[i].z; ab[i].w += dy[i].w;
      }
    }
    s1 = warp_sum(s1) / (float)n;
    s2 = warp_sum(s2) / (float)n;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = l + 64 * i;
      if (c < nc) {
        float4 o;
        o.x = rs * (dy[i].x * gm[i].x - s1 - xh[i].x * s2);
        o.y = rs * (dy[i].y * gm[i].y - s1 - xh[i].y * s2);
        o.z = rs * (dy[i].z * gm[i].z - s1 - xh[i].z * s2);
        o.w = rs * (dy[i].w * gm[i].w - s1 - xh[i].w * s2);
        if (dres) {
          const float4 d = V4<float>::load(dres + row * ldx + 4 * c);
          o.x += d.x; o.y += d.y; o.z += d.z; o.w += d.w;
        }
        V4<float>::store(dX + row * ldx + 4 * c, o);
        if (dXt) V4<T>::store(dXt + row * ldx + 4 * c, o);
      }
    }
  }
  // combine the four waves in a fixed order: gain sums, then shift sums
#pragma unroll
  for (int i = 0; i < MAXC; ++i) red[(wave * MAXC + i) * 64 + l] = ag[i];
  __syncthreads();
  combine_waves(red, nc, part_g + (int64_t)blockIdx.x * n);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MAXC; ++i) red[(wave * MAXC + i) * 64 + l] = ab[i];
  __syncthreads();
  combine_waves(red, nc, part_b + (int64_t)blockIdx.x * n);
}

// ---- column sums: part[b][c] = sum of X[r][c] over row chunk b ----------------------
constexpr int COLSUM_MAX_CHUNKS = 256;

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

// out[c] += sum_b part[b][c], b < nb.  One block per 64 columns; its four waves
// take every fourth partial row and are combined in a fixed order.
__global__ void reduce_partials_kernel(const float* part, int64_t nb, int n, float* out) {
  __shared__ float red[4][64];
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int c = blockIdx.x * 64 + l;
  float s = 0.f;
  if (c < n)
    for (int64_t b = w; b < nb; b += 4) s += part[b * n + c];
  red[w][l] = s;
  __syncthreads();
  if (w == 0 && c < n) out[c] += (red[0][l] + red[1][l]) + (red[2][l] + red[3][l]);
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
  const int32_t pp = pos[r];
  T* v = qk + r * ld + (which ? kcol : 0) + hd * d;
  const float4 a = V4<T>::load(v + j0), b = V4<T>::load(v + j0 + half);
  const float x1[4] = {a.x, a.y, a.z, a.w}, x2[4] = {b.x, b.y, b.z, b.w};
  float o1[4], o2[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int j = j0 + e;
    const int coord = (j < quarter) ? (pp >> 16) : (pp & 0xFFFF);
    const float2 cs = tab[coord * quarter + (j < quarter ? j : j - quarter)];
    const float sn = inverse ? -cs.y : cs.y;
    o1[e] = x1[e] * cs.x - x2[e] * sn;
    o2[e] = x2[e] * cs.x + x1[e] * sn;
  }
  V4<T>::store(v + j0, make_float4(o1[0], o1[1], o1[2], o1[3]));
  V4<T>::store(v + j0 + half, make_float4(o2[0], o2[1], o2[2], o2[3]));
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

}  // namespace

hipError_t layernorm_fwd(int dtype, const float* X, int64_t ldx, int64_t rows, int n,
                         const void* g, const void* b, float eps, void* Y, int64_t ldy,
                         float* mean, float* rstd, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 3) / 4));
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(ln_fwd_kernel<bf16>, grid, dim3(256), 0, s, X, ldx, rows, n,
                       (const bf16*)g, (const bf16*)b, eps, (bf16*)Y, ldy, mean, rstd);
  else
    hipLaunchKernelGGL(ln_fwd_kernel<float>, grid, dim3(256), 0, s, X, ldx, rows, n,
                       (const float*)g, (const float*)b, eps, (float*)Y, ldy, mean, rstd);
  return hipGetLastError();
}

int64_t layernorm_bwd_partial_rows(int64_t rows) {
  const int64_t b = (rows + 3) / 4;
  return b < LN_BWD_MAX_BLOCKS ? b : LN_BWD_MAX_BLOCKS;
}

hipError_t layernorm_bwd(int dtype, const float* dY, int64_t ldd, const float* X, int64_t ldx,
                         const float* mean, const float* rstd, const void* g, int64_t rows, int n,
                         const float* dres, float* dX, void* dXt, float* part_g, float* part_b,
                         float* grad_g, float* grad_b, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const int64_t nblk = layernorm_bwd_partial_rows(rows);
  const int64_t rpb = (rows + nblk - 1) / nblk;
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(ln_bwd_kernel<bf16>, dim3((unsigned)nblk), dim3(256), 0, s, dY, ldd, X, ldx,
                       mean, rstd, (const bf16*)g, rows, n, rpb, dres, dX, (bf16*)dXt, part_g,
                       part_b);
  else
    hipLaunchKernelGGL(ln_bwd_kernel<float>, dim3((unsigned)nblk), dim3(256), 0, s, dY, ldd, X,
                       ldx, mean, rstd, (const float*)g, rows, n, rpb, dres, dX, (float*)dXt,
                       part_g, part_b);
  const dim3 rg((unsigned)((n + 63) / 64));
  if (grad_g)
    hipLaunchKernelGGL(reduce_partials_kernel, rg, dim3(256), 0, s, part_g, nblk, n, grad_g);
  if (grad_b)
    hipLaunchKernelGGL(reduce_partials_kernel, rg, dim3(256), 0, s, part_b, nblk, n, grad_b);
  return hipGetLastError();
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
  const dim3 grid((unsigned)blocks_for(n), (unsigned)nb);
  if (dtype_in == DT_BF16)
    hipLaunchKernelGGL(colsum_partial_kernel<bf16>, grid, dim3(256), 0, s, (const bf16*)X, ld,
                       rows, n, rpc, part);
  else
    hipLaunchKernelGGL(colsum_partial_kernel<float>, grid, dim3(256), 0, s, (const float*)X, ld,
                       rows, n, rpc, part);
  hipLaunchKernelGGL(reduce_partials_kernel, dim3((unsigned)((n + 63) / 64)), dim3(256), 0, s,
                     part, nb, n, out);
  return hipGetLastError();
}

hipError_t splitk_reduce(const float* part, int splits, int64_t M, int64_t N, float* out,
                         int64_t ldo, hipStream_t s) {
  if (M * N == 0) return hipSuccess;
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

hipError_t rope(int dtype, void* qk, int64_t ld, int64_t rows, int heads, int d, int kcol,
                const int32_t* pos, const float* tab, int inverse, hipStream_t s) {
  const int64_t n = rows * 2 * heads * (d / 8);  // (q and k) x heads x 4-pair groups
  if (n == 0) return hipSuccess;
  const float2* t = reinterpret_cast<const float2*>(tab);
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
