// GEMM kernels for the shard's linear layers.
//
//   forward   X W^T      (A row-major [M,K], B = weight [N,K])          a_t=0 b_t=0
//   backward  dY W       (A row-major [M,K], B = weight [K,N])          a_t=0 b_t=1
//   weights   dY^T X     (A = dY [K,M] read transposed, B = X [K,N])    a_t=1 b_t=1
//
// bf16 path: v_mfma_f32_32x32x16_bf16 on LDS-staged tiles (BK = 64), fp32
// accumulation in registers, double-buffered LDS with one barrier per K step,
// register prefetch of the next K tile while the current one is multiplied.
// Both operands are kept K-contiguous in LDS (rows padded by 8 elements so the
// 16-byte fragment reads of 8 consecutive rows hit distinct banks); an operand
// that is contiguous along M or N in memory is loaded as 8x8 blocks and
// transposed in registers on its way into LDS.  The MFMA is issued with the B
// tile as its first operand so each lane ends up owning one output row and 4
// consecutive output columns per group, which the fused epilogues store as one
// vector.
//
// fp32 check mode: a plain LDS-tiled FMA kernel with the same layouts and
// epilogues.
#include "common.h"
#include "kernels.h"

namespace merak {

struct GemmBatch {
  GemmProblem p[kMaxGroup];
  int tile_start[kMaxGroup + 1];
  int n_probs;
};

// ---------------------------------------------------------------------------
// Epilogue on 4 consecutive columns n..n+3 of row m.
// ---------------------------------------------------------------------------
template <typename T, int EPI>
__device__ __forceinline__ void epilogue4(const GemmProblem& p, int m, int n, float v[4]) {
  const size_t off = (size_t)m * p.ldc + n;
  if constexpr (EPI == EPI_F32) {
    float* c = reinterpret_cast<float*>(p.c) + off;
    if (p.accumulate) {
      float o[4];
      load4(c, o);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += o[e];
    }
    store4(c, v);
  } else {
    T* c = reinterpret_cast<T*>(p.c) + off;
    if constexpr (EPI == EPI_STORE) {
      store4(c, v);
    } else if constexpr (EPI == EPI_BIAS) {
      float b[4];
      load4(reinterpret_cast<const T*>(p.bias) + n, b);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += b[e];
      store4(c, v);
    } else if constexpr (EPI == EPI_BIAS_GELU) {
      float b[4], g[4];
      load4(reinterpret_cast<const T*>(p.bias) + n, b);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] += b[e];
        g[e] = gelu_f(v[e]);
      }
      store4(reinterpret_cast<T*>(p.aux) + off, v);
      store4(c, g);
    } else if constexpr (EPI == EPI_BIAS_RESID) {
      float b[4], r[4];
      if (p.aux) store4(reinterpret_cast<T*>(p.aux) + off, v);
      load4(reinterpret_cast<const T*>(p.bias) + n, b);
      load4(reinterpret_cast<const T*>(p.resid) + off, r);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = r[e] + v[e] + b[e];
      store4(c, v);
    } else if constexpr (EPI == EPI_GELU_BWD) {
      float u[4];
      load4(reinterpret_cast<const T*>(p.aux) + off, u);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] *= gelu_grad_f(u[e]);
      store4(c, v);
    }
  }
}

// Problem owning workgroup `bid`, copied out with uniform selects (a dynamic
// index into the kernel-argument struct would go through scratch memory).
__device__ __forceinline__ GemmProblem select_problem(const GemmBatch& b, int bid, int* start) {
  GemmProblem p = b.p[0];
  int s = 0;
#pragma unroll
  for (int i = 1; i < kMaxGroup; ++i)
    if (i < b.n_probs && bid >= b.tile_start[i]) { p = b.p[i]; s = b.tile_start[i]; }
  *start = s;
  return p;
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------
constexpr int kBK = 64;
constexpr int kLDK = kBK + 8;  // padded LDS row, elements

// Global -> register -> LDS staging of one BK-wide K tile of an operand with R
// rows (R = BM for A, BN for B).  Each thread owns kRegs 16-byte registers.
//
// K-contiguous operand (element (r, k) at base[r*ld + k]): 16-byte chunks,
// 8 per row; consecutive threads read consecutive chunks of a row.
//
// R-contiguous operand (element (r, k) at base[k*ld + r]): 8x8 blocks (8 k rows
// x 8 contiguous r), transposed in registers so LDS stays K-contiguous.
template <bool TRANS, int R, int NT>
struct Stage {
  static constexpr int kChunks = R * kBK / 8;             // K-contiguous: 16-byte chunks
  static constexpr int kBlocks = (R / 8) * (kBK / 8);     // R-contiguous: 8x8 blocks
  static constexpr int kBlocksPer = (kBlocks + NT - 1) / NT;
  static_assert(TRANS || kChunks % NT == 0, "tile/thread mismatch");
  static constexpr int kRegs = TRANS ? kBlocksPer * 8 : kChunks / NT;
};

template <bool TRANS, int R, int NT, int NR>
__device__ __forceinline__ void stage_load(u32x4_t (&r)[NR], const bf16_t* base, int ld, int r0, int rtot,
                                           int k0, int tid) {
  if constexpr (!TRANS) {
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const int c = tid + i * NT;
      const int row = min(r0 + (c >> 3), rtot - 1);
      r[i] = *reinterpret_cast<const u32x4_t*>(base + (size_t)row * ld + k0 + (c & 7) * 8);
    }
  } else {
    constexpr int kBlocks = Stage<TRANS, R, NT>::kBlocks;
#pragma unroll
    for (int i = 0; i < NR / 8; ++i) {
      const int c = tid + i * NT;
      if (kBlocks % NT == 0 || c < kBlocks) {
        const int kg = c & 7;
        const int rs = min(r0 + (c >> 3) * 8, rtot - 8);
        const bf16_t* p = base + (size_t)(k0 + kg * 8) * ld + rs;
#pragma unroll
        for (int j = 0; j < 8; ++j) r[i * 8 + j] = *reinterpret_cast<const u32x4_t*>(p + (size_t)j * ld);
      }
    }
  }
}

__device__ __forceinline__ uint32_t u4_word(const u32x4_t& v, int w) { return v[w]; }

template <bool TRANS, int R, int NT, int NR>
__device__ __forceinline__ void stage_store(const u32x4_t (&r)[NR], bf16_t* s, int tid) {
  if constexpr (!TRANS) {
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const int c = tid + i * NT;
      *reinterpret_cast<u32x4_t*>(s + (c >> 3) * kLDK + (c & 7) * 8) = r[i];
    }
  } else {
    constexpr int kBlocks = Stage<TRANS, R, NT>::kBlocks;
#pragma unroll
    for (int i = 0; i < NR / 8; ++i) {
      const int c = tid + i * NT;
      if (kBlocks % NT == 0 || c < kBlocks) {
        const int kg = c & 7;
        const int rb = (c >> 3) * 8;
        // Output row rb+e holds k = kg*8 + 0..7, i.e. element e of r[i*8 + 0..7].
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          uint32_t o[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t lo = u4_word(r[i * 8 + 2 * q], e >> 1);
            const uint32_t hi = u4_word(r[i * 8 + 2 * q + 1], e >> 1);
            o[q] = (e & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
          }
          *reinterpret_cast<u32x4_t*>(s + (rb + e) * kLDK + kg * 8) = u32x4_t{o[0], o[1], o[2], o[3]};
        }
      }
    }
  }
}

template <int BM, int BN, int WM, int WN, bool A_T, bool B_T, int EPI>
__global__ void __launch_bounds__(WM * WN * 64) gemm_mfma_kernel(GemmBatch batch) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM / 32;
  constexpr int TN = BN / WN / 32;
  extern __shared__ __align__(16) bf16_t smem[];
  bf16_t* As = smem;                      // [2][BM][kLDK]
  bf16_t* Bs = smem + 2 * BM * kLDK;      // [2][BN][kLDK]

  const int bid = blockIdx.x;
  int tile0;
  const GemmProblem p = select_problem(batch, bid, &tile0);
  const int tile = bid - tile0;
  const int tiles_n = (p.N + BN - 1) / BN;
  const int m0 = (tile / tiles_n) * BM;
  const int n0 = (tile % tiles_n) * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  const bf16_t* A = reinterpret_cast<const bf16_t*>(p.a);
  const bf16_t* B = reinterpret_cast<const bf16_t*>(p.b);

  u32x4_t ra[Stage<A_T, BM, NT>::kRegs];
  u32x4_t rb[Stage<B_T, BN, NT>::kRegs];

  f32x16_t acc[TN][TM];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[j][i][e] = 0.0f;

  const int KT = p.K / kBK;
  stage_load<A_T, BM, NT>(ra, A, p.lda, m0, p.M, 0, tid);
  stage_load<B_T, BN, NT>(rb, B, p.ldb, n0, p.N, 0, tid);
  stage_store<A_T, BM, NT>(ra, As, tid);
  stage_store<B_T, BN, NT>(rb, Bs, tid);
  __syncthreads();

  const int arow = wm * TM * 32 + (lane & 31);
  const int brow = wn * TN * 32 + (lane & 31);
  const int kofs = (lane >> 5) * 8;

  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) {
      stage_load<A_T, BM, NT>(ra, A, p.lda, m0, p.M, (kt + 1) * kBK, tid);
      stage_load<B_T, BN, NT>(rb, B, p.ldb, n0, p.N, (kt + 1) * kBK, tid);
    }
    const bf16_t* as = As + buf * BM * kLDK;
    const bf16_t* bs = Bs + buf * BN * kLDK;
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      bf16x8_t af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(as + (arow + i * 32) * kLDK + ks * 16 + kofs);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(bs + (brow + j * 32) * kLDK + ks * 16 + kofs);
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int i = 0; i < TM; ++i)
          acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[j][i], 0, 0, 0);
    }
    if (kt + 1 < KT) {
      stage_store<A_T, BM, NT>(ra, As + (buf ^ 1) * BM * kLDK, tid);
      stage_store<B_T, BN, NT>(rb, Bs + (buf ^ 1) * BN * kLDK, tid);
    }
    __syncthreads();
  }

  // acc[j][i][r]: output row m = m0 + wm*TM*32 + i*32 + lane%32,
  // column n = n0 + wn*TN*32 + j*32 + (r/4)*8 + (lane/32)*4 + r%4.
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + wm * TM * 32 + i * 32 + (lane & 31);
      if (m >= p.M) continue;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn * TN * 32 + j * 32 + g * 8 + (lane >> 5) * 4;
        if (n < p.N) {
          float v[4] = {acc[j][i][4 * g], acc[j][i][4 * g + 1], acc[j][i][4 * g + 2], acc[j][i][4 * g + 3]};
          epilogue4<bf16_t, EPI>(p, m, n, v);
        }
      }
    }
}

// ---------------------------------------------------------------------------
// fp32 check-mode kernel: 64x64 tile, BK = 16, 4x4 outputs per thread.
// ---------------------------------------------------------------------------
template <bool A_T, bool B_T, int EPI>
__global__ void __launch_bounds__(256) gemm_f32_kernel(GemmBatch batch) {
  __shared__ float As[16][64 + 4];
  __shared__ float Bs[16][64 + 4];
  const int bid = blockIdx.x;
  int tile0;
  const GemmProblem p = select_problem(batch, bid, &tile0);
  const int tile = bid - tile0;
  const int tiles_n = (p.N + 63) / 64;
  const int m0 = (tile / tiles_n) * 64;
  const int n0 = (tile % tiles_n) * 64;
  const float* A = reinterpret_cast<const float*>(p.a);
  const float* B = reinterpret_cast<const float*>(p.b);
  const int tid = threadIdx.x;
  const int ty = tid >> 4, tx = tid & 15;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < p.K; k0 += 16) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      int idx = tid + e * 256;
      int m, k, n, kb;
      if (!A_T) { m = idx >> 4; k = idx & 15; } else { k = idx >> 6; m = idx & 63; }
      int gm = min(m0 + m, p.M - 1);
      As[k][m] = A_T ? A[(size_t)(k0 + k) * p.lda + gm] : A[(size_t)gm * p.lda + k0 + k];
      if (!B_T) { n = idx >> 4; kb = idx & 15; } else { kb = idx >> 6; n = idx & 63; }
      int gn = min(n0 + n, p.N - 1);
      Bs[kb][n] = B_T ? B[(size_t)(k0 + kb) * p.ldb + gn] : B[(size_t)gn * p.ldb + k0 + kb];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      float a[4], b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) { a[r] = As[k][ty * 4 + r]; b[r] = Bs[k][tx * 4 + r]; }
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(a[r], b[c], acc[r][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int m = m0 + ty * 4 + r;
    const int n = n0 + tx * 4;
    if (m < p.M && n < p.N) epilogue4<float, EPI>(p, m, n, acc[r]);
  }
}

// ---------------------------------------------------------------------------
// Host dispatch
// ---------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN, bool AT, bool BT, int EPI>
static hipError_t run_mfma(GemmBatch& batch, hipStream_t stream) {
  int tiles = 0;
  for (int i = 0; i < batch.n_probs; ++i) {
    batch.tile_start[i] = tiles;
    tiles += ((batch.p[i].M + BM - 1) / BM) * ((batch.p[i].N + BN - 1) / BN);
  }
  for (int i = batch.n_probs; i <= kMaxGroup; ++i) batch.tile_start[i] = tiles;
  if (tiles == 0) return hipSuccess;
  constexpr size_t lds = (size_t)2 * (BM + BN) * kLDK * sizeof(bf16_t);
  auto kern = gemm_mfma_kernel<BM, BN, WM, WN, AT, BT, EPI>;
  static bool attr_set = false;  // per instantiation
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3(tiles), dim3(WM * WN * 64), lds, stream, batch);
  return hipGetLastError();
}

template <bool AT, bool BT, int EPI>
static hipError_t run_f32(GemmBatch& batch, hipStream_t stream) {
  int tiles = 0;
  for (int i = 0; i < batch.n_probs; ++i) {
    batch.tile_start[i] = tiles;
    tiles += ((batch.p[i].M + 63) / 64) * ((batch.p[i].N + 63) / 64);
  }
  for (int i = batch.n_probs; i <= kMaxGroup; ++i) batch.tile_start[i] = tiles;
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_f32_kernel<AT, BT, EPI>), dim3(tiles), dim3(256), 0, stream, batch);
  return hipGetLastError();
}

template <bool AT, bool BT, int EPI>
static hipError_t run_bf16(GemmBatch& batch, hipStream_t stream) {
  long long big_tiles = 0;
  for (int i = 0; i < batch.n_probs; ++i)
    big_tiles += (long long)((batch.p[i].M + 255) / 256) * ((batch.p[i].N + 255) / 256);
  if (big_tiles >= 240) return run_mfma<256, 256, 2, 2, AT, BT, EPI>(batch, stream);
  return run_mfma<128, 128, 2, 2, AT, BT, EPI>(batch, stream);
}

template <bool AT, bool BT>
static hipError_t dispatch_epi(int dtype, int epi, GemmBatch& batch, hipStream_t s) {
#define MERAK_EPI_CASE(E)                                                             \
  case E:                                                                             \
    return dtype == DT_BF16 ? run_bf16<AT, BT, E>(batch, s) : run_f32<AT, BT, E>(batch, s);
  switch (epi) {
    MERAK_EPI_CASE(EPI_STORE)
    MERAK_EPI_CASE(EPI_BIAS)
    MERAK_EPI_CASE(EPI_BIAS_GELU)
    MERAK_EPI_CASE(EPI_BIAS_RESID)
    MERAK_EPI_CASE(EPI_GELU_BWD)
    MERAK_EPI_CASE(EPI_F32)
    default:
      return hipErrorInvalidValue;
  }
#undef MERAK_EPI_CASE
}

hipError_t launch_gemm(int dtype, bool a_t, bool b_t, int epi, const GemmProblem* probs, int n_probs,
                       hipStream_t stream) {
  if (n_probs < 1 || n_probs > kMaxGroup) return hipErrorInvalidValue;
  GemmBatch batch;
  for (int i = 0; i < n_probs; ++i) batch.p[i] = probs[i];
  batch.n_probs = n_probs;
  if (!a_t && !b_t) return dispatch_epi<false, false>(dtype, epi, batch, stream);
  if (!a_t && b_t) return dispatch_epi<false, true>(dtype, epi, batch, stream);
  if (a_t && !b_t) return dispatch_epi<true, false>(dtype, epi, batch, stream);
  return dispatch_epi<true, true>(dtype, epi, batch, stream);
}

}  // namespace merak
