// Causal self-attention on a rank's local heads, forward and backward.
//
// Layout: packed qkv [batch, seq, 3, heads, d] (row stride 3*heads*d), output
// o [batch, seq, heads, d], log-sum-exp lse [batch, heads, seq] (natural log of
// sum_j exp(s_ij), s = q k^T / sqrt(d)).  Keys j > i are masked.
//
// bf16 path (v_mfma_f32_32x32x16_bf16, fp32 softmax): flash-style tiling so the
// seq x seq score matrix never reaches HBM (the method published as
// FlashAttention, Dao et al. 2022; the gfx950 tiling below is our own).
//   * forward: a workgroup owns 32*NW query rows of one (batch, head), a wave 32
//     of them.  It computes the transposed score tile S^T = K Q^T so that each
//     lane owns one query column; the online softmax then needs only a lane-half
//     exchange, and the probabilities P^T stay in registers as the second
//     operand of the O^T += V^T P^T product (K/V tiles of 64 keys in LDS, V
//     stored transposed).
//   * backward, deterministic (no atomics): a KV-parallel kernel (a wave owns
//     32 keys, loops over 64-query tiles) accumulates dK and dV; a Q-parallel
//     kernel (a wave owns 32 queries, loops over 64-key tiles) accumulates dQ.
//     Both rebuild P from the stored lse.  delta_i = rowsum(dO_i * O_i) comes
//     from a small preprocessing kernel.
// The 32x32 accumulator layout is: lane l holds column l%32 and rows
// (r/4)*8 + (l/32)*4 + r%4 for r = 0..15.  When such an accumulator feeds the
// next MFMA as its 16-deep operand, the MFMA's k index 8*(l/32)+e is taken to
// mean row (e/4)*8 + (l/32)*4 + e%4 of that 16-row group; the other operand is
// read from a transposed LDS copy with the same key order (two 8-byte reads).
//
// fp32 check mode: one thread per query (or key) row, fp32 throughout.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace merak {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t cvt8(const f32x16_t& a, int base) {
  bf16x8_t r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (__bf16)a[base + e];
  return r;
}

// Operand of 8 elements from a transposed LDS tile (rows = MFMA i index, row
// contiguous along the 16-deep group): elements e=0..3 at cols kb+4*hf+0..3,
// e=4..7 at cols kb+8+4*hf+0..3.
__device__ __forceinline__ bf16x8_t frag_t(const bf16_t* row, int kb, int hf) {
  const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(row + kb + 4 * hf);
  const u32x2_t hi = *reinterpret_cast<const u32x2_t*>(row + kb + 8 + 4 * hf);
  u32x4_t v = {lo[0], lo[1], hi[0], hi[1]};
  return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ bf16x8_t frag_kc(const bf16_t* p) { return *reinterpret_cast<const bf16x8_t*>(p); }

// Copy a [64 rows][D] tile (global row stride gs) into LDS [64][LD] (LD % 8 == 0).
template <int D, int LD, int NT>
__device__ __forceinline__ void tile_to_lds(bf16_t* dst, const bf16_t* src, size_t gs, int tid) {
  constexpr int CPR = D / 8;
  for (int c = tid; c < 64 * CPR; c += NT) {
    const int row = c / CPR, ch = c % CPR;
    *reinterpret_cast<u32x4_t*>(dst + row * LD + ch * 8) =
        *reinterpret_cast<const u32x4_t*>(src + (size_t)row * gs + ch * 8);
  }
}

// Copy a [64 rows][D] tile transposed into LDS [D][LDT] (LDT % 4 == 0):
// 8x8 blocks through registers, written as two 8-byte halves.
template <int D, int LDT, int NT>
__device__ __forceinline__ void tile_to_lds_t(bf16_t* dst, const bf16_t* src, size_t gs, int tid) {
  constexpr int CPR = D / 8;
  for (int c = tid; c < 8 * CPR; c += NT) {
    const int dc = c % CPR, rg = c / CPR;
    u32x4_t r[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      r[j] = *reinterpret_cast<const u32x4_t*>(src + (size_t)(rg * 8 + j) * gs + dc * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint32_t o[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t lo = r[2 * q][e >> 1], hi = r[2 * q + 1][e >> 1];
        o[q] = (e & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
      }
      bf16_t* d = dst + (dc * 8 + e) * LDT + rg * 8;
      *reinterpret_cast<u32x2_t*>(d) = u32x2_t{o[0], o[1]};
      *reinterpret_cast<u32x2_t*>(d + 4) = u32x2_t{o[2], o[3]};
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 forward
// ---------------------------------------------------------------------------
template <int D, int NW>
__global__ void __launch_bounds__(NW * 64) attn_fwd_bf16(int S, int H, const bf16_t* __restrict__ qkv,
                                                         bf16_t* __restrict__ o, float* __restrict__ lse,
                                                         float scale_log2) {
  constexpr int NT = NW * 64;
  constexpr int LDK = D + 8;
  constexpr int LDV = 64 + 4;
  constexpr int KS = D / 16;
  constexpr int DT = D / 32;
  __shared__ __align__(16) bf16_t Ks[64 * LDK];
  __shared__ __align__(16) bf16_t Vt[D * LDV];

  const int b = blockIdx.z, hh = blockIdx.y;
  const int qb = gridDim.x - 1 - blockIdx.x;  // longest rows first
  const int qblk0 = qb * 32 * NW;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int q0 = qblk0 + wave * 32;
  const size_t rs = (size_t)3 * H * D;
  const bf16_t* base = qkv + (size_t)b * S * rs;
  const bf16_t* Qp = base + hh * D;
  const bf16_t* Kp = base + (size_t)H * D + hh * D;
  const bf16_t* Vp = base + (size_t)2 * H * D + hh * D;

  const int myq = min(q0 + l32, S - 1);
  bf16x8_t qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = frag_kc(Qp + (size_t)myq * rs + ks * 16 + hf * 8);

  f32x16_t oacc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[t][r] = 0.0f;
  float m = -INFINITY, l = 0.0f;

  const int qlast_wg = min(qblk0 + 32 * NW, S) - 1;
  const int n_kb = qlast_wg / 64 + 1;
  const int q = q0 + l32;
  for (int kb = 0; kb < n_kb; ++kb) {
    const int k0 = kb * 64;
    __syncthreads();
    tile_to_lds<D, LDK, NT>(Ks, Kp + (size_t)k0 * rs, rs, tid);
    tile_to_lds_t<D, LDV, NT>(Vt, Vp + (size_t)k0 * rs, rs, tid);
    __syncthreads();
    if (q0 >= S || k0 > q0 + 31) continue;

    f32x16_t s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[t][r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_kc(Ks + (t * 32 + l32) * LDK + ks * 16 + hf * 8),
                                                       qf[ks], s[t], 0, 0, 0);
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + t * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
        const float v = key > q ? -INFINITY : s[t][r] * scale_log2;
        s[t][r] = v;
        mloc = fmaxf(mloc, v);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float mnew = fmaxf(m, mloc);
    const float alpha = exp2f(m - mnew);
    m = mnew;
    l *= alpha;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[t][r] *= alpha;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2f(s[t][r] - mnew);
        s[t][r] = p;
        l += p;
      }
    bf16x8_t pb[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) pb[g] = cvt8(s[g >> 1], (g & 1) * 8);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_t(Vt + (dt * 32 + l32) * LDV, g * 16, hf), pb[g],
                                                           oacc[dt], 0, 0, 0);
  }
  if (q0 >= S) return;
  l += __shfl_xor(l, 32, 64);
  const float inv = 1.0f / l;
  if (q < S) {
    bf16_t* orow = o + ((size_t)b * S + q) * H * D + hh * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v[4] = {oacc[dt][4 * g] * inv, oacc[dt][4 * g + 1] * inv, oacc[dt][4 * g + 2] * inv,
                      oacc[dt][4 * g + 3] * inv};
        store4(orow + dt * 32 + g * 8 + hf * 4, v);
      }
    if (hf == 0) lse[((size_t)b * H + hh) * S + q] = (m + log2f(l)) * kLn2;
  }
}

// ---------------------------------------------------------------------------
// delta[b, h, i] = sum_d dO[b, i, h, d] * O[b, i, h, d]
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(256) attn_delta_kernel(int B, int S, int H, const T* __restrict__ o,
                                                         const T* __restrict__ dout, float* __restrict__ delta) {
  const int row = blockIdx.x * 256 + threadIdx.x;  // (b, i, h) flattened
  if (row >= B * S * H) return;
  const T* orow = o + (size_t)row * D;
  const T* drow = dout + (size_t)row * D;
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < D; c += 8) {
    float a[8], d[8];
    load8(orow + c, a);
    load8(drow + c, d);
#pragma unroll
    for (int e = 0; e < 8; ++e) s += a[e] * d[e];
  }
  const int hh = row % H;
  const int bi = row / H;
  const int i = bi % S, b = bi / S;
  delta[((size_t)b * H + hh) * S + i] = s;
}

// ---------------------------------------------------------------------------
// bf16 backward: dK, dV (KV-parallel)
// ---------------------------------------------------------------------------
template <int D, int NW>
__global__ void __launch_bounds__(NW * 64) attn_bwd_dkdv_bf16(int S, int H, const bf16_t* __restrict__ qkv,
                                                              const bf16_t* __restrict__ dout,
                                                              const float* __restrict__ lse,
                                                              const float* __restrict__ delta,
                                                              bf16_t* __restrict__ dqkv, float scale_log2,
                                                              float scale) {
  constexpr int NT = NW * 64;
  constexpr int LDK = D + 8;
  constexpr int LDT = 64 + 4;
  constexpr int KS = D / 16;
  constexpr int DT = D / 32;
  __shared__ __align__(16) bf16_t Qs[64 * LDK];
  __shared__ __align__(16) bf16_t Qt[D * LDT];
  __shared__ __align__(16) bf16_t dOs[64 * LDK];
  __shared__ __align__(16) bf16_t dOt[D * LDT];
  __shared__ float lse_s[64], del_s[64];

  const int b = blockIdx.z, hh = blockIdx.y;
  const int kblk0 = blockIdx.x * 32 * NW;  // early keys see the most queries: dispatched first
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int kw0 = kblk0 + wave * 32;
  const size_t rs = (size_t)3 * H * D;
  const size_t ors = (size_t)H * D;
  const bf16_t* base = qkv + (size_t)b * S * rs;
  const bf16_t* Qp = base + hh * D;
  const bf16_t* Kp = base + (size_t)H * D + hh * D;
  const bf16_t* Vp = base + (size_t)2 * H * D + hh * D;
  const bf16_t* dOp = dout + (size_t)b * S * ors + hh * D;
  const float* lse_p = lse + ((size_t)b * H + hh) * S;
  const float* del_p = delta + ((size_t)b * H + hh) * S;

  const int mykey = min(kw0 + l32, S - 1);
  bf16x8_t kf[KS], vf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    kf[ks] = frag_kc(Kp + (size_t)mykey * rs + ks * 16 + hf * 8);
    vf[ks] = frag_kc(Vp + (size_t)mykey * rs + ks * 16 + hf * 8);
  }
  f32x16_t dk[DT], dv[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[t][r] = dv[t][r] = 0.0f;

  const int key = kw0 + l32;
  for (int qs = (kblk0 / 64) * 64; qs < S; qs += 64) {
    __syncthreads();
    tile_to_lds<D, LDK, NT>(Qs, Qp + (size_t)qs * rs, rs, tid);
    tile_to_lds_t<D, LDT, NT>(Qt, Qp + (size_t)qs * rs, rs, tid);
    tile_to_lds<D, LDK, NT>(dOs, dOp + (size_t)qs * ors, ors, tid);
    tile_to_lds_t<D, LDT, NT>(dOt, dOp + (size_t)qs * ors, ors, tid);
    if (tid < 64) {
      lse_s[tid] = lse_p[qs + tid] * kLog2e;
      del_s[tid] = del_p[qs + tid];
    }
    __syncthreads();
    if (kw0 >= S || qs + 63 < kw0) continue;

    f32x16_t p[2], dp[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) p[t][r] = dp[t][r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        p[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_kc(Qs + (t * 32 + l32) * LDK + ks * 16 + hf * 8),
                                                       kf[ks], p[t], 0, 0, 0);
        dp[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_kc(dOs + (t * 32 + l32) * LDK + ks * 16 + hf * 8),
                                                        vf[ks], dp[t], 0, 0, 0);
      }
    }
    // p[t][r]: query qs + t*32 + (r/4)*8 + 4*hf + r%4, key `key`.
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qi = t * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
        const float pv = (key > qs + qi) ? 0.0f : exp2f(p[t][r] * scale_log2 - lse_s[qi]);
        p[t][r] = pv;
        dp[t][r] = pv * (dp[t][r] - del_s[qi]);
      }
    bf16x8_t pb[4], sb[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      pb[g] = cvt8(p[g >> 1], (g & 1) * 8);
      sb[g] = cvt8(dp[g >> 1], (g & 1) * 8);
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        dv[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_t(dOt + (dt * 32 + l32) * LDT, g * 16, hf), pb[g],
                                                         dv[dt], 0, 0, 0);
        dk[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_t(Qt + (dt * 32 + l32) * LDT, g * 16, hf), sb[g],
                                                         dk[dt], 0, 0, 0);
      }
  }
  if (kw0 >= S || key >= S) return;
  bf16_t* krow = dqkv + ((size_t)b * S + key) * rs + (size_t)H * D + hh * D;
  bf16_t* vrow = krow + (size_t)H * D;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float a[4], c[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[e] = dk[dt][4 * g + e] * scale;
        c[e] = dv[dt][4 * g + e];
      }
      store4(krow + dt * 32 + g * 8 + hf * 4, a);
      store4(vrow + dt * 32 + g * 8 + hf * 4, c);
    }
}

// ---------------------------------------------------------------------------
// bf16 backward: dQ (Q-parallel)
// ---------------------------------------------------------------------------
template <int D, int NW>
__global__ void __launch_bounds__(NW * 64) attn_bwd_dq_bf16(int S, int H, const bf16_t* __restrict__ qkv,
                                                            const bf16_t* __restrict__ dout,
                                                            const float* __restrict__ lse,
                                                            const float* __restrict__ delta,
                                                            bf16_t* __restrict__ dqkv, float scale_log2,
                                                            float scale) {
  constexpr int NT = NW * 64;
  constexpr int LDK = D + 8;
  constexpr int LDT = 64 + 4;
  constexpr int KS = D / 16;
  constexpr int DT = D / 32;
  __shared__ __align__(16) bf16_t Ks[64 * LDK];
  __shared__ __align__(16) bf16_t Kt[D * LDT];
  __shared__ __align__(16) bf16_t Vs[64 * LDK];

  const int b = blockIdx.z, hh = blockIdx.y;
  const int qb = gridDim.x - 1 - blockIdx.x;
  const int qblk0 = qb * 32 * NW;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int q0 = qblk0 + wave * 32;
  const size_t rs = (size_t)3 * H * D;
  const size_t ors = (size_t)H * D;
  const bf16_t* base = qkv + (size_t)b * S * rs;
  const bf16_t* Qp = base + hh * D;
  const bf16_t* Kp = base + (size_t)H * D + hh * D;
  const bf16_t* Vp = base + (size_t)2 * H * D + hh * D;
  const bf16_t* dOp = dout + (size_t)b * S * ors + hh * D;

  const int myq = min(q0 + l32, S - 1);
  bf16x8_t qf[KS], of[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qf[ks] = frag_kc(Qp + (size_t)myq * rs + ks * 16 + hf * 8);
    of[ks] = frag_kc(dOp + (size_t)myq * ors + ks * 16 + hf * 8);
  }
  const float lse2 = lse[((size_t)b * H + hh) * S + myq] * kLog2e;
  const float del = delta[((size_t)b * H + hh) * S + myq];
  f32x16_t dq[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[t][r] = 0.0f;

  const int qlast_wg = min(qblk0 + 32 * NW, S) - 1;
  const int n_kb = qlast_wg / 64 + 1;
  const int q = q0 + l32;
  for (int kb = 0; kb < n_kb; ++kb) {
    const int k0 = kb * 64;
    __syncthreads();
    tile_to_lds<D, LDK, NT>(Ks, Kp + (size_t)k0 * rs, rs, tid);
    tile_to_lds_t<D, LDT, NT>(Kt, Kp + (size_t)k0 * rs, rs, tid);
    tile_to_lds<D, LDK, NT>(Vs, Vp + (size_t)k0 * rs, rs, tid);
    __syncthreads();
    if (q0 >= S || k0 > q0 + 31) continue;
    f32x16_t p[2], dp[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) p[t][r] = dp[t][r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        p[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_kc(Ks + (t * 32 + l32) * LDK + ks * 16 + hf * 8),
                                                       qf[ks], p[t], 0, 0, 0);
        dp[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_kc(Vs + (t * 32 + l32) * LDK + ks * 16 + hf * 8),
                                                        of[ks], dp[t], 0, 0, 0);
      }
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + t * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
        const float pv = key > q ? 0.0f : exp2f(p[t][r] * scale_log2 - lse2);
        dp[t][r] = pv * (dp[t][r] - del);
      }
    bf16x8_t sb[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) sb[g] = cvt8(dp[g >> 1], (g & 1) * 8);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        dq[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_t(Kt + (dt * 32 + l32) * LDT, g * 16, hf), sb[g],
                                                         dq[dt], 0, 0, 0);
  }
  if (q0 >= S || q >= S) return;
  bf16_t* qrow = dqkv + ((size_t)b * S + q) * rs + hh * D;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float a[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) a[e] = dq[dt][4 * g + e] * scale;
      store4(qrow + dt * 32 + g * 8 + hf * 4, a);
    }
}

// ---------------------------------------------------------------------------
// fp32 check mode
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(128) attn_fwd_f32(int B, int S, int H, const float* __restrict__ qkv,
                                                    float* __restrict__ o, float* __restrict__ lse, float scale) {
  const int idx = blockIdx.x * 128 + threadIdx.x;  // (b, h, i), i fastest
  if (idx >= B * H * S) return;
  const int i = idx % S, hh = (idx / S) % H, b = idx / (S * H);
  const size_t rs = (size_t)3 * H * D;
  const float* base = qkv + (size_t)b * S * rs;
  const float* qr = base + (size_t)i * rs + hh * D;
  float acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) acc[d] = 0.0f;
  float m = -INFINITY, l = 0.0f;
  for (int j = 0; j <= i; ++j) {
    const float* kr = base + (size_t)j * rs + (size_t)H * D + hh * D;
    const float* vr = kr + (size_t)H * D;
    float s = 0.0f;
#pragma unroll
    for (int d = 0; d < D; ++d) s += qr[d] * kr[d];
    s *= scale;
    const float mn = fmaxf(m, s);
    const float a = expf(m - mn), p = expf(s - mn);
    l = l * a + p;
#pragma unroll
    for (int d = 0; d < D; ++d) acc[d] = acc[d] * a + p * vr[d];
    m = mn;
  }
  float* orow = o + ((size_t)b * S + i) * H * D + hh * D;
#pragma unroll
  for (int d = 0; d < D; ++d) orow[d] = acc[d] / l;
  lse[((size_t)b * H + hh) * S + i] = m + logf(l);
}

template <int D>
__global__ void __launch_bounds__(128) attn_bwd_dq_f32(int B, int S, int H, const float* __restrict__ qkv,
                                                       const float* __restrict__ dout, const float* __restrict__ lse,
                                                       const float* __restrict__ delta, float* __restrict__ dqkv,
                                                       float scale) {
  const int idx = blockIdx.x * 128 + threadIdx.x;
  if (idx >= B * H * S) return;
  const int i = idx % S, hh = (idx / S) % H, b = idx / (S * H);
  const size_t rs = (size_t)3 * H * D;
  const float* base = qkv + (size_t)b * S * rs;
  const float* qr = base + (size_t)i * rs + hh * D;
  const float* dor = dout + ((size_t)b * S + i) * H * D + hh * D;
  const float L = lse[((size_t)b * H + hh) * S + i];
  const float del = delta[((size_t)b * H + hh) * S + i];
  float acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) acc[d] = 0.0f;
  for (int j = 0; j <= i; ++j) {
    const float* kr = base + (size_t)j * rs + (size_t)H * D + hh * D;
    const float* vr = kr + (size_t)H * D;
    float s = 0.0f, dp = 0.0f;
#pragma unroll
    for (int d = 0; d < D; ++d) {
      s += qr[d] * kr[d];
      dp += dor[d] * vr[d];
    }
    const float p = expf(s * scale - L);
    const float ds = p * (dp - del);
#pragma unroll
    for (int d = 0; d < D; ++d) acc[d] += ds * kr[d];
  }
  float* out = dqkv + ((size_t)b * S + i) * rs + hh * D;
#pragma unroll
  for (int d = 0; d < D; ++d) out[d] = acc[d] * scale;
}

template <int D>
__global__ void __launch_bounds__(128) attn_bwd_dkdv_f32(int B, int S, int H, const float* __restrict__ qkv,
                                                         const float* __restrict__ dout,
                                                         const float* __restrict__ lse,
                                                         const float* __restrict__ delta,
                                                         float* __restrict__ dqkv, float scale) {
  const int idx = blockIdx.x * 128 + threadIdx.x;
  if (idx >= B * H * S) return;
  const int j = idx % S, hh = (idx / S) % H, b = idx / (S * H);
  const size_t rs = (size_t)3 * H * D;
  const float* base = qkv + (size_t)b * S * rs;
  const float* kr = base + (size_t)j * rs + (size_t)H * D + hh * D;
  const float* vr = kr + (size_t)H * D;
  float dk[D], dv[D];
#pragma unroll
  for (int d = 0; d < D; ++d) dk[d] = dv[d] = 0.0f;
  for (int i = j; i < S; ++i) {
    const float* qr = base + (size_t)i * rs + hh * D;
    const float* dor = dout + ((size_t)b * S + i) * H * D + hh * D;
    float s = 0.0f, dp = 0.0f;
#pragma unroll
    for (int d = 0; d < D; ++d) {
      s += qr[d] * kr[d];
      dp += dor[d] * vr[d];
    }
    const float p = expf(s * scale - lse[((size_t)b * H + hh) * S + i]);
    const float ds = p * (dp - delta[((size_t)b * H + hh) * S + i]);
#pragma unroll
    for (int d = 0; d < D; ++d) {
      dv[d] += p * dor[d];
      dk[d] += ds * qr[d];
    }
  }
  float* ko = dqkv + ((size_t)b * S + j) * rs + (size_t)H * D + hh * D;
  float* vo = ko + (size_t)H * D;
#pragma unroll
  for (int d = 0; d < D; ++d) {
    ko[d] = dk[d] * scale;
    vo[d] = dv[d];
  }
}

// ---------------------------------------------------------------------------
// Host launchers
// ---------------------------------------------------------------------------
constexpr int kAttnWaves = 4;

template <int D>
static hipError_t fwd_d(int dtype, int B, int S, int H, const void* qkv, void* o, float* lse, hipStream_t st) {
  const float scale = 1.0f / sqrtf((float)D);
  if (dtype == DT_BF16) {
    constexpr int QB = 32 * kAttnWaves;
    dim3 grid((S + QB - 1) / QB, H, B);
    hipLaunchKernelGGL((attn_fwd_bf16<D, kAttnWaves>), grid, dim3(64 * kAttnWaves), 0, st, S, H,
                       (const bf16_t*)qkv, (bf16_t*)o, lse, scale * kLog2e);
  } else {
    dim3 grid((B * H * S + 127) / 128);
    hipLaunchKernelGGL((attn_fwd_f32<D>), grid, dim3(128), 0, st, B, S, H, (const float*)qkv, (float*)o, lse,
                       scale);
  }
  return hipGetLastError();
}

template <int D>
static hipError_t bwd_d(int dtype, int B, int S, int H, const void* qkv, const void* o, const float* lse,
                        const void* dout, void* dqkv, float* delta, hipStream_t st) {
  const float scale = 1.0f / sqrtf((float)D);
  const int rows = B * S * H;
  if (dtype == DT_BF16) {
    hipLaunchKernelGGL((attn_delta_kernel<bf16_t, D>), dim3((rows + 255) / 256), dim3(256), 0, st, B, S, H,
                       (const bf16_t*)o, (const bf16_t*)dout, delta);
    constexpr int BLK = 32 * kAttnWaves;
    dim3 grid((S + BLK - 1) / BLK, H, B);
    hipLaunchKernelGGL((attn_bwd_dkdv_bf16<D, kAttnWaves>), grid, dim3(64 * kAttnWaves), 0, st, S, H,
                       (const bf16_t*)qkv, (const bf16_t*)dout, lse, delta, (bf16_t*)dqkv, scale * kLog2e, scale);
    hipLaunchKernelGGL((attn_bwd_dq_bf16<D, kAttnWaves>), grid, dim3(64 * kAttnWaves), 0, st, S, H,
                       (const bf16_t*)qkv, (const bf16_t*)dout, lse, delta, (bf16_t*)dqkv, scale * kLog2e, scale);
  } else {
    hipLaunchKernelGGL((attn_delta_kernel<float, D>), dim3((rows + 255) / 256), dim3(256), 0, st, B, S, H,
                       (const float*)o, (const float*)dout, delta);
    dim3 grid((B * H * S + 127) / 128);
    hipLaunchKernelGGL((attn_bwd_dkdv_f32<D>), grid, dim3(128), 0, st, B, S, H, (const float*)qkv,
                       (const float*)dout, lse, delta, (float*)dqkv, scale);
    hipLaunchKernelGGL((attn_bwd_dq_f32<D>), grid, dim3(128), 0, st, B, S, H, (const float*)qkv,
                       (const float*)dout, lse, delta, (float*)dqkv, scale);
  }
  return hipGetLastError();
}

hipError_t launch_attention_fwd(int dtype, int batch, int seq, int heads, int d, const void* qkv, void* o,
                                float* lse, hipStream_t stream) {
  if (batch <= 0 || seq <= 0 || heads <= 0) return hipSuccess;
  if (seq % 64 != 0) return hipErrorInvalidValue;
  switch (d) {
    case 64: return fwd_d<64>(dtype, batch, seq, heads, qkv, o, lse, stream);
    case 96: return fwd_d<96>(dtype, batch, seq, heads, qkv, o, lse, stream);
    case 128: return fwd_d<128>(dtype, batch, seq, heads, qkv, o, lse, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attention_bwd(int dtype, int batch, int seq, int heads, int d, const void* qkv, const void* o,
                                const float* lse, const void* dout, void* dqkv, float* delta, hipStream_t stream) {
  if (batch <= 0 || seq <= 0 || heads <= 0) return hipSuccess;
  if (seq % 64 != 0) return hipErrorInvalidValue;
  switch (d) {
    case 64: return bwd_d<64>(dtype, batch, seq, heads, qkv, o, lse, dout, dqkv, delta, stream);
    case 96: return bwd_d<96>(dtype, batch, seq, heads, qkv, o, lse, dout, dqkv, delta, stream);
    case 128: return bwd_d<128>(dtype, batch, seq, heads, qkv, o, lse, dout, dqkv, delta, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace merak
