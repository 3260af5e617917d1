// Internal launch interface of the gfx950 kernels (host side).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace merak {

enum DType { DT_BF16 = 0, DT_F32 = 1 };

enum Epi {
  EPI_STORE = 0,       // C = acc
  EPI_BIAS = 1,        // C = acc + bias[n]
  EPI_BIAS_GELU = 2,   // aux = u = acc + bias[n]; C = gelu(u)
  EPI_BIAS_RESID = 3,  // aux = acc (if non-null); C = resid + acc + bias[n]
  EPI_GELU_BWD = 4,    // C = acc * gelu'(aux)
  EPI_F32 = 5,         // fp32 C = acc (or += acc when accumulate)
  EPI_COUNT = 6
};

// One GEMM problem: C[M,N] = op(A)[M,K] op(B)[K,N] with the layout flags of the
// launch (a_t: A[m,k] at a[k*lda+m]; b_t: B[k,n] at b[k*ldb+n], else b[n*ldb+k]).
struct GemmProblem {
  int M, N, K;
  const void* a; int lda;
  const void* b; int ldb;
  void* c; int ldc;
  const void* bias;   // [N], element type of the launch (EPI_BIAS*, nullptr otherwise)
  const void* resid;  // [M, ldc] (EPI_BIAS_RESID)
  void* aux;          // [M, ldc] (EPI_BIAS_GELU out, EPI_BIAS_RESID optional out, EPI_GELU_BWD in)
  int accumulate;     // EPI_F32
};

constexpr int kMaxGroup = 4;

// Launch 1..kMaxGroup independent problems sharing layout, epilogue and dtype
// as one grid.
hipError_t launch_gemm(int dtype, bool a_t, bool b_t, int epi, const GemmProblem* probs, int n_probs,
                       hipStream_t stream);
// Whether the bf16 kernel can address both operands of `q`: it uses 32-bit
// byte offsets, counting the rows of a partial edge tile (up to 256 past M or
// N).  launch_gemm refuses a problem that does not fit.
inline bool gemm_bf16_offsets_fit(const GemmProblem& q, bool a_t, bool b_t) {
  const long long ea = (long long)(a_t ? q.K : q.M + 256) * q.lda + (a_t ? q.M + 256 : q.K);
  const long long eb = (long long)(b_t ? q.K : q.N + 256) * q.ldb + (b_t ? q.N + 256 : q.K);
  return 2 * ea < (1LL << 31) && 2 * eb < (1LL << 31);
}

// LayerNorm over rows of width h (h % 8 == 0).  Like attention, one launch may
// cover `members` groups of `rows` rows, member m starting m * member_stride
// rows after every row-indexed pointer given (member_stride >= rows).
hipError_t launch_layernorm_fwd(int dtype, int rows, int h, float eps, const void* x, const void* gamma,
                                const void* beta, void* y, float* mean, float* rstd, hipStream_t stream,
                                int members = 1, int member_stride = 0);

// Rows per partial-sum segment of the deterministic column reductions.
constexpr int kReduceRows = 64;
inline size_t reduce_groups(int rows) { return (size_t)(rows + kReduceRows - 1) / kReduceRows; }

// dx = dres + LN'(dout) (input gradient of LayerNorm plus the residual gradient).
hipError_t launch_layernorm_bwd(int dtype, int rows, int h, const void* dout, const void* x,
                                const float* mean, const float* rstd, const void* gamma,
                                const void* dres, void* dx, hipStream_t stream, int members = 1,
                                int member_stride = 0);

// Partials [reduce_groups(rows), h] of sum(dout * xhat) and sum(dout).
hipError_t launch_layernorm_param_partials(int dtype, int rows, int h, const void* dout, const void* x,
                                           const float* mean, const float* rstd, float* part_g, float* part_b,
                                           hipStream_t stream);

// Column partial sums of x [rows, cols] into part [groups, cols] fp32.
hipError_t launch_column_partials(int dtype, int rows, int cols, const void* x, float* part,
                                  hipStream_t stream);

// out[c] (=|+=) sum over groups g of part[g, c], in increasing g.
hipError_t launch_reduce_partials(int groups, int cols, const float* part, float* out, int accumulate,
                                  hipStream_t stream);

// Batched forms: up to kMaxColJobs independent reductions in one launch, with
// the same per-job results as the single calls above.
constexpr int kMaxColJobs = 6;
struct ColPartialJob {
  int mode;  // 0: p0 = column partials of a; 1: LayerNorm parameter partials (a = dout)
  int rows, cols;
  const void* a;
  const void* x;  // mode 1: LayerNorm input, with mean and rstd
  const float* mean;
  const float* rstd;
  float* p0;
  float* p1;  // mode 1: partials of sum dout
};
hipError_t launch_column_partials_batch(int dtype, const ColPartialJob* jobs, int n, hipStream_t stream);
struct ReduceJob {
  int groups, cols;
  const float* part;
  float* out;
  int accumulate;
};
hipError_t launch_reduce_partials_batch(const ReduceJob* jobs, int n, hipStream_t stream);

// Count of the NaN and +-Inf elements among x[0 .. n) into *count (device,
// 64-bit; the first kernel sets it to zero, so no memset node is needed under
// graph capture).  x is 16-byte aligned.
hipError_t launch_count_nonfinite(int dtype, const void* x, long long n, unsigned long long* count,
                                  hipStream_t stream);

// Library-owned scratch of the allocation-free LayerNorm backward
// (merak_layernorm_bwd_noalloc): kNoAllocScratchFloats fp32 elements per GPU.
// noalloc_scratch returns its device address on the current device, taking it
// with hipGetSymbolAddress on the first call per device.
constexpr size_t kNoAllocScratchFloats = (size_t)4 << 20;  // 16 MiB
hipError_t noalloc_scratch(float** out);

// Causal attention on packed qkv [batch, seq, 3, heads, d].  One launch may
// cover `members` groups of `batch` sequences each, member m starting
// m * member_stride sequences after the pointers given (so the sub-micro-
// batches that share a stream form one grid); member_stride >= batch.
hipError_t launch_attention_fwd(int dtype, int batch, int seq, int heads, int d, const void* qkv, void* o,
                                float* lse, hipStream_t stream, int members = 1, int member_stride = 0);
hipError_t launch_attention_bwd(int dtype, int batch, int seq, int heads, int d, const void* qkv,
                                const void* o, const float* lse, const void* dout, void* dqkv,
                                float* delta, hipStream_t stream, int members = 1, int member_stride = 0);

}  // namespace merak
