// LayerNorm forward/backward and deterministic column reductions.
//
// These kernels are bound by HBM bandwidth.  A wave owns a row: each lane
// moves 16-byte chunks (8 elements) with consecutive lanes on consecutive
// chunks, so every wave-wide access is one contiguous span; row statistics are
// wave64 butterfly reductions in fp32.
//
// Parameter/bias gradients are sums over all tokens.  They are formed in two
// fixed-order phases (no floating-point atomics): a workgroup owns a segment of
// kReduceRows rows and a 512-column slice, its 4 waves take every 4th row of
// the segment, and their register sums are added in wave order into one
// partial row; reduce_partials then adds the partials in segment order.
#include "common.h"
#include "kernels.h"

namespace merak {

constexpr int kRowsPerBlock = 4;  // waves per 256-thread workgroup

// Rows of a launch may come from `members` equal groups of mrows rows, group m
// starting m * mstride rows after the pointers given: logical row r is
// physical row (r / mrows) * mstride + r % mrows.
__device__ __forceinline__ int member_row(int r, int mrows, int mstride) {
  return (r / mrows) * mstride + r % mrows;
}

template <typename T, int CH>
__global__ void __launch_bounds__(256) ln_fwd_kernel(int rows, int mrows, int mstride, int h, float eps,
                                                     const T* __restrict__ x,
                                                     const T* __restrict__ gamma, const T* __restrict__ beta,
                                                     T* __restrict__ y, float* __restrict__ mean,
                                                     float* __restrict__ rstd) {
  const int lrow = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (lrow >= rows) return;
  const int row = member_row(lrow, mrows, mstride);
  const T* xr = x + (size_t)row * h;
  float v[CH][8];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int c = (lane + 64 * i) * 8;
    if (c < h) {
      load8(xr + c, v[i]);
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[i][e];
    }
  }
  const float mu = wave_sum(s) / (float)h;
  float q = 0.0f;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int c = (lane + 64 * i) * 8;
    if (c < h) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = v[i][e] - mu;
        q += d * d;
      }
    }
  }
  const float var = wave_sum(q) / (float)h;  // biased variance
  const float rs = 1.0f / sqrtf(var + eps);
  T* yr = y + (size_t)row * h;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int c = (lane + 64 * i) * 8;
    if (c < h) {
      float g[8], b[8], o[8];
      load8(gamma + c, g);
      load8(beta + c, b);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (v[i][e] - mu) * rs * g[e] + b[e];
      store8(yr + c, o);
    }
  }
  if (lane == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

// dx = dres + rstd * (dxhat - mean(dxhat) - xhat * mean(dxhat * xhat)),
// dxhat = dout * gamma.  One wave per row; the row stays in registers.
template <typename T, int CH>
__global__ void __launch_bounds__(256) ln_bwd_kernel(int rows, int mrows, int mstride, int h,
                                                     const T* __restrict__ dout,
                                                     const T* __restrict__ x, const float* __restrict__ mean,
                                                     const float* __restrict__ rstd, const T* __restrict__ gamma,
                                                     const T* __restrict__ dres, T* __restrict__ dx) {
  const int lrow = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (lrow >= rows) return;
  const int row = member_row(lrow, mrows, mstride);
  const float mu = mean[row], rs = rstd[row];
  const T* xr = x + (size_t)row * h;
  const T* dr = dout + (size_t)row * h;
  float xh[CH][8], dxh[CH][8];
  float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int c = (lane + 64 * i) * 8;
    if (c < h) {
      float xv[8], dv[8], g[8];
      load8(xr + c, xv);
      load8(dr + c, dv);
      load8(gamma + c, g);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        xh[i][e] = (xv[e] - mu) * rs;
        dxh[i][e] = dv[e] * g[e];
        s1 += dxh[i][e];
        s2 += dxh[i][e] * xh[i][e];
      }
    }
  }
  const float m1 = wave_sum(s1) / (float)h;
  const float m2 = wave_sum(s2) / (float)h;
  const T* rr = dres + (size_t)row * h;
  T* outr = dx + (size_t)row * h;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int c = (lane + 64 * i) * 8;
    if (c < h) {
      float res[8], o[8];
      load8(rr + c, res);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = res[e] + rs * (dxh[i][e] - m1 - xh[i][e] * m2);
      store8(outr + c, o);
    }
  }
}

// Segment/slice partial sums.  MODE 0: part0 = sum x.  MODE 1 (LayerNorm
// parameters): part0 = sum dout * xhat, part1 = sum dout, with xhat rebuilt from
// x, mean and rstd.
template <typename T, int MODE>
__global__ void __launch_bounds__(256) segment_partials_kernel(int rows, int cols, const T* __restrict__ a,
                                                               const T* __restrict__ x,
                                                               const float* __restrict__ mean,
                                                               const float* __restrict__ rstd,
                                                               float* __restrict__ part0,
                                                               float* __restrict__ part1) {
  constexpr int NQ = MODE == 0 ? 1 : 2;
  __shared__ float red[NQ][kRowsPerBlock][64 * 8];
  const int w = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int seg = blockIdx.y;
  const int c = (blockIdx.x * 64 + lane) * 8;
  const int r0 = seg * kReduceRows;
  const int r1 = min(r0 + kReduceRows, rows);
  float acc[NQ][8];
#pragma unroll
  for (int q = 0; q < NQ; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[q][e] = 0.0f;
  if (c < cols) {
    for (int r = r0 + w; r < r1; r += kRowsPerBlock) {
      float v[8];
      load8(a + (size_t)r * cols + c, v);
      if constexpr (MODE == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[0][e] += v[e];
      } else {
        float xv[8];
        load8(x + (size_t)r * cols + c, xv);
        const float mu = mean[r], rs = rstd[r];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          acc[0][e] += v[e] * ((xv[e] - mu) * rs);
          acc[1][e] += v[e];
        }
      }
    }
  }
#pragma unroll
  for (int q = 0; q < NQ; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) red[q][w][lane * 8 + e] = acc[q][e];
  __syncthreads();
  // 256 threads finish 64 lanes x 8 columns x NQ quantities; wave order fixed.
  for (int idx = threadIdx.x; idx < NQ * 64 * 8; idx += 256) {
    const int q = idx / (64 * 8);
    const int j = idx % (64 * 8);
    const int col = blockIdx.x * 64 * 8 + j;
    if (col < cols) {
      float t = 0.0f;
#pragma unroll
      for (int i = 0; i < kRowsPerBlock; ++i) t += red[q][i][j];
      (q == 0 ? part0 : part1)[(size_t)seg * cols + col] = t;
    }
  }
}

// out[c] (= or +=) sum_g part[g, c].  16 waves split the groups round-robin and
// their sums are added in wave order, so the result does not depend on timing.
constexpr int kReduceWaves = 16;
__global__ void __launch_bounds__(64 * kReduceWaves) reduce_partials_kernel(int groups, int cols,
                                                                           const float* __restrict__ part,
                                                                           float* __restrict__ out,
                                                                           int accumulate) {
  __shared__ float red[kReduceWaves][64];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  float s = 0.0f;
  if (c < cols)
    for (int g = w; g < groups; g += kReduceWaves) s += part[(size_t)g * cols + c];
  red[w][lane] = s;
  __syncthreads();
  if (w == 0 && c < cols) {
    float t = 0.0f;
#pragma unroll
    for (int i = 0; i < kReduceWaves; ++i) t += red[i][lane];
    out[c] = accumulate ? out[c] + t : t;
  }
}

// ---------------------------------------------------------------------------
// Host launchers
// ---------------------------------------------------------------------------
// Rows of one launch: `rows` logical rows in groups of mrows, mstride apart.
struct RowMap {
  int rows, mrows, mstride;
};

template <typename T, int CH>
static hipError_t ln_fwd_t(RowMap rm, int h, float eps, const void* x, const void* g, const void* b, void* y,
                           float* mean, float* rstd, hipStream_t s) {
  dim3 grid((rm.rows + kRowsPerBlock - 1) / kRowsPerBlock);
  hipLaunchKernelGGL((ln_fwd_kernel<T, CH>), grid, dim3(256), 0, s, rm.rows, rm.mrows, rm.mstride, h, eps,
                     (const T*)x, (const T*)g, (const T*)b, (T*)y, mean, rstd);
  return hipGetLastError();
}

template <typename T>
static hipError_t ln_fwd_dispatch(RowMap rm, int h, float eps, const void* x, const void* g, const void* b,
                                  void* y, float* mean, float* rstd, hipStream_t s) {
  const int ch = (h + 511) / 512;
  if (ch <= 1) return ln_fwd_t<T, 1>(rm, h, eps, x, g, b, y, mean, rstd, s);
  if (ch <= 2) return ln_fwd_t<T, 2>(rm, h, eps, x, g, b, y, mean, rstd, s);
  if (ch <= 4) return ln_fwd_t<T, 4>(rm, h, eps, x, g, b, y, mean, rstd, s);
  if (ch <= 6) return ln_fwd_t<T, 6>(rm, h, eps, x, g, b, y, mean, rstd, s);
  if (ch <= 8) return ln_fwd_t<T, 8>(rm, h, eps, x, g, b, y, mean, rstd, s);
  if (ch <= 12) return ln_fwd_t<T, 12>(rm, h, eps, x, g, b, y, mean, rstd, s);
  if (ch <= 16) return ln_fwd_t<T, 16>(rm, h, eps, x, g, b, y, mean, rstd, s);
  return hipErrorInvalidValue;
}

static bool row_map(int rows, int members, int member_stride, RowMap* rm) {
  if (members < 1 || (members > 1 && member_stride < rows)) return false;
  if ((long long)rows * members > 0x7fffffffLL || (long long)member_stride * (members - 1) + rows > 0x7fffffffLL)
    return false;
  *rm = {rows * members, rows, members > 1 ? member_stride : rows};
  return true;
}

hipError_t launch_layernorm_fwd(int dtype, int rows, int h, float eps, const void* x, const void* gamma,
                                const void* beta, void* y, float* mean, float* rstd, hipStream_t stream,
                                int members, int member_stride) {
  if (rows <= 0) return hipSuccess;
  RowMap rm;
  if (h % 8 != 0 || !row_map(rows, members, member_stride, &rm)) return hipErrorInvalidValue;
  return dtype == DT_BF16 ? ln_fwd_dispatch<bf16_t>(rm, h, eps, x, gamma, beta, y, mean, rstd, stream)
                          : ln_fwd_dispatch<float>(rm, h, eps, x, gamma, beta, y, mean, rstd, stream);
}

template <typename T, int CH>
static hipError_t ln_bwd_t(RowMap rm, int h, const void* dout, const void* x, const float* mean,
                           const float* rstd, const void* g, const void* dres, void* dx, hipStream_t s) {
  dim3 grid((rm.rows + kRowsPerBlock - 1) / kRowsPerBlock);
  hipLaunchKernelGGL((ln_bwd_kernel<T, CH>), grid, dim3(256), 0, s, rm.rows, rm.mrows, rm.mstride, h,
                     (const T*)dout, (const T*)x, mean, rstd, (const T*)g, (const T*)dres, (T*)dx);
  return hipGetLastError();
}

template <typename T>
static hipError_t ln_bwd_dispatch(RowMap rm, int h, const void* dout, const void* x, const float* mean,
                                  const float* rstd, const void* g, const void* dres, void* dx, hipStream_t s) {
  const int ch = (h + 511) / 512;
  if (ch <= 1) return ln_bwd_t<T, 1>(rm, h, dout, x, mean, rstd, g, dres, dx, s);
  if (ch <= 2) return ln_bwd_t<T, 2>(rm, h, dout, x, mean, rstd, g, dres, dx, s);
  if (ch <= 4) return ln_bwd_t<T, 4>(rm, h, dout, x, mean, rstd, g, dres, dx, s);
  if (ch <= 6) return ln_bwd_t<T, 6>(rm, h, dout, x, mean, rstd, g, dres, dx, s);
  if (ch <= 8) return ln_bwd_t<T, 8>(rm, h, dout, x, mean, rstd, g, dres, dx, s);
  if (ch <= 12) return ln_bwd_t<T, 12>(rm, h, dout, x, mean, rstd, g, dres, dx, s);
  if (ch <= 16) return ln_bwd_t<T, 16>(rm, h, dout, x, mean, rstd, g, dres, dx, s);
  return hipErrorInvalidValue;
}

hipError_t launch_layernorm_bwd(int dtype, int rows, int h, const void* dout, const void* x, const float* mean,
                                const float* rstd, const void* gamma, const void* dres, void* dx,
                                hipStream_t stream, int members, int member_stride) {
  if (rows <= 0) return hipSuccess;
  RowMap rm;
  if (h % 8 != 0 || !row_map(rows, members, member_stride, &rm)) return hipErrorInvalidValue;
  return dtype == DT_BF16 ? ln_bwd_dispatch<bf16_t>(rm, h, dout, x, mean, rstd, gamma, dres, dx, stream)
                          : ln_bwd_dispatch<float>(rm, h, dout, x, mean, rstd, gamma, dres, dx, stream);
}

template <int MODE>
static hipError_t partials_launch(int dtype, int rows, int cols, const void* a, const void* x,
                                  const float* mean, const float* rstd, float* p0, float* p1, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (cols % 8 != 0) return hipErrorInvalidValue;
  dim3 grid((cols / 8 + 63) / 64, (unsigned)reduce_groups(rows));
  if (dtype == DT_BF16)
    hipLaunchKernelGGL((segment_partials_kernel<bf16_t, MODE>), grid, dim3(256), 0, s, rows, cols,
                       (const bf16_t*)a, (const bf16_t*)x, mean, rstd, p0, p1);
  else
    hipLaunchKernelGGL((segment_partials_kernel<float, MODE>), grid, dim3(256), 0, s, rows, cols,
                       (const float*)a, (const float*)x, mean, rstd, p0, p1);
  return hipGetLastError();
}

hipError_t launch_column_partials(int dtype, int rows, int cols, const void* x, float* part, hipStream_t stream) {
  return partials_launch<0>(dtype, rows, cols, x, nullptr, nullptr, nullptr, part, nullptr, stream);
}

hipError_t launch_layernorm_param_partials(int dtype, int rows, int h, const void* dout, const void* x,
                                           const float* mean, const float* rstd, float* part_g, float* part_b,
                                           hipStream_t stream) {
  return partials_launch<1>(dtype, rows, h, dout, x, mean, rstd, part_g, part_b, stream);
}

hipError_t launch_reduce_partials(int groups, int cols, const float* part, float* out, int accumulate,
                                  hipStream_t stream) {
  if (cols <= 0) return hipSuccess;
  dim3 grid((cols + 63) / 64);
  hipLaunchKernelGGL(reduce_partials_kernel, grid, dim3(64 * kReduceWaves), 0, stream, groups, cols, part, out,
                     accumulate);
  return hipGetLastError();
}

}  // namespace merak
