// Causal self-attention on a rank's local heads, forward and backward.
//
// Layout: packed qkv [batch, seq, 3, heads, d] (row stride 3*heads*d), output
// o [batch, seq, heads, d], log-sum-exp lse [batch, heads, seq] (natural log of
// sum_j exp(s_ij), s = q k^T / sqrt(d)).  Keys j > i are masked.
//
// bf16 path (v_mfma_f32_32x32x16_bf16, fp32 softmax): flash-style tiling so the
// seq x seq score matrix never reaches HBM (the method published as
// FlashAttention, Dao et al. 2022; the gfx950 tiling below is our own).
//   * forward: a workgroup owns 64 query rows of one (batch, head); its four
//     waves are two groups of 32 rows times the even and odd 64-key blocks,
//     merged at the end with the online-softmax merge.  A wave computes the
//     transposed score tile S^T = K Q^T so that each lane owns one query
//     column; the softmax then needs only a lane-half exchange, and P^T stays
//     in registers as the second operand of O^T += V^T P^T.  K and V tiles sit
//     in LDS in their natural [key][d] layout; V^T fragments come from
//     transposing LDS reads.
//   * backward, deterministic (no atomics): a Q-parallel kernel accumulates dQ
//     and also forms delta_i = rowsum(dO_i * O_i) for its rows; a KV-parallel
//     kernel, run after it, accumulates dK and dV.  Both rebuild P from the
//     stored lse.
// The 32x32 accumulator layout is: lane l holds column l%32 and rows
// (r/4)*8 + (l/32)*4 + r%4 for r = 0..15.  When such an accumulator feeds the
// next MFMA as its 16-deep operand, the MFMA's k index 8*(l/32)+e is taken to
// mean row (e/4)*8 + (l/32)*4 + e%4 of that 16-row group; the other operand is
// read with transposing LDS reads in the same key order (two 8-byte reads).
//
// fp32 check mode: one thread per query (or key) row, fp32 throughout.
#include <math.h>

#include <atomic>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace merak {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));
#define MERAK_LDS __attribute__((address_space(3)))

// Eight accumulator values narrowed to an MFMA operand, four packed
// conversion instructions.
__device__ __forceinline__ bf16x8_t cvt8(const f32x16_t& a, int base) {
  typedef float f32x8_t __attribute__((ext_vector_type(8)));
  f32x8_t v;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = a[base + e];
  return __builtin_convertvector(v, bf16x8_t);
}

// A [64 rows][D] bf16 tile in LDS with rows padded to LD elements: 16-byte
// reads of 16 consecutive rows hit distinct banks, the transposing reads of 4
// consecutive rows at most two-way.  LD * 2 is a multiple of 16, so the tile is
// exactly CPR wave-instructions of 16-byte-per-lane direct loads.
template <int D>
struct AttnTile {
  static constexpr int LD = D == 128 ? D + 24 : D + 8;
  static constexpr int CPR = LD / 8;         // 16-byte chunks per padded row
  static constexpr int DC = D / 8;           // data chunks per row
  static constexpr int BYTES = 64 * LD * 2;  // = CPR * 1024
};

// One wave's plan for copying rows 0..63 of a tensor (row stride gs
// elements) into the padded tile with loads that write LDS directly: lane i of
// instruction q fills chunk 64 q + i (padding chunks re-read a data chunk).
// The per-lane element offsets are computed once.
template <int D>
struct TileLoad {
  using TT = AttnTile<D>;
  uint32_t off[TT::CPR];
  __device__ __forceinline__ void init(size_t gs, int lane) {
#pragma unroll
    for (int q = 0; q < TT::CPR; ++q) {
      const int c = q * 64 + lane;
      const int row = c / TT::CPR, ch = c % TT::CPR;
      off[q] = (uint32_t)(row * gs) + (uint32_t)(ch < TT::DC ? ch : 0) * 8u;
    }
  }
  __device__ __forceinline__ void issue(char* lds, const bf16_t* src) const {
#pragma unroll
    for (int q = 0; q < TT::CPR; ++q)
      __builtin_amdgcn_global_load_lds(src + off[q], (MERAK_LDS void*)(lds + q * 1024), 16, 0, 0);
  }
};

// 64 floats (one per lane) into LDS with a direct load.
__device__ __forceinline__ void wave_vec_load(char* lds, const float* src, int lane) {
  __builtin_amdgcn_global_load_lds(src + lane, (MERAK_LDS void*)lds, 4, 0, 0);
}

// 8 consecutive elements of row `row` from column `col` of a padded tile.
template <int LD>
__device__ __forceinline__ bf16x8_t frag_row(const char* tile, int row, int col) {
  return *reinterpret_cast<const bf16x8_t*>(tile + (row * LD + col) * 2);
}

// MFMA operand of X^T taken from a natural tile X[row][col]: lane l gets
// column col0 + l % 32 and rows kb + 4 (l / 32) + 0..3 (elements 0..3) and
// kb + 8 + 4 (l / 32) + 0..3 (elements 4..7), the key order of an accumulator
// reused as the 16-deep operand.  Two transposing LDS reads: in each 16-lane
// group, lane j fetches 4 columns of row (j / 4) and lane i receives column i of
// the 4 rows.
template <int LD>
__device__ __forceinline__ bf16x8_t frag_tr(const char* tile, int kb, int col0, int lane) {
  const int row = kb + (lane >> 5) * 4 + ((lane & 15) >> 2);
  const int col = col0 + ((lane >> 4) & 1) * 16 + (lane & 3) * 4;
  const char* p = tile + (row * LD + col) * 2;
  const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((MERAK_LDS s16x4_t*)p);
  const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((MERAK_LDS s16x4_t*)(p + 8 * LD * 2));
  const s16x8_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ bf16x8_t frag_kc(const bf16_t* p) { return *reinterpret_cast<const bf16x8_t*>(p); }

// Sequence index of launch batch z when a launch covers several members (for
// example the sub-micro-batches that share a stream), each of Bm consecutive
// sequences, members mstride sequences apart.  Every tensor is addressed by
// sequence (rows b * S + i, lse and delta rows (b * H + h) * S + i), so the
// kernels need nothing else to work on such a group.
__device__ __forceinline__ int seq_index(int z, int Bm, int mstride) { return (z / Bm) * mstride + z % Bm; }

// LDS stages of the bf16 kernels (each four tiles: two 64-row blocks of two
// tensors).  One stage keeps a workgroup small enough (53 KB at d = 96) to share
// a CU with a GEMM workgroup of the other stream; the loads of the next block
// pair are then issued after the current pair has been used.
#ifndef MERAK_ATTN_STAGES
#define MERAK_ATTN_STAGES 1
#endif
constexpr int kAttnStages = MERAK_ATTN_STAGES;
static_assert(kAttnStages == 1 || kAttnStages == 2, "one or two LDS stages");

template <int D>
constexpr size_t attn_lds_bytes() { return (size_t)kAttnStages * 4 * AttnTile<D>::BYTES; }

// ---------------------------------------------------------------------------
// bf16 forward.  A workgroup owns 64 query rows of one (batch, head); wave w
// takes the 32 rows of group w % 2 against the even (w < 2) or odd 64-key
// blocks, and the two halves are merged at the end (online-softmax merge).
// Each stage holds the K and V tiles of two key blocks.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(256) attn_fwd_bf16(int S, int H, int Bm, int mstride, const bf16_t* __restrict__ qkv,
                                                     bf16_t* __restrict__ o, float* __restrict__ lse,
                                                     float scale_log2) {
  using TT = AttnTile<D>;
  constexpr int LD = TT::LD, KS = D / 16, DT = D / 32, TB = TT::BYTES;
  extern __shared__ __align__(16) char smem[];  // [stage][K blk a, K blk b, V blk a, V blk b]

  // Grid (heads, sequences, row blocks), row block slowest: the whole grid
  // runs longest rows first.
  const int b = seq_index(blockIdx.y, Bm, mstride), hh = blockIdx.x;
  const int qt = gridDim.z - 1 - blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int qg = wave & 1, kh = wave >> 1;
  const int q0 = qt * 64 + qg * 32;
  const int q = q0 + l32;
  const size_t rs = (size_t)3 * H * D;
  const bf16_t* base = qkv + (size_t)b * S * rs;
  const bf16_t* Qp = base + hh * D;
  const bf16_t* Kp = base + (size_t)H * D + hh * D;
  const bf16_t* Vp = base + (size_t)2 * H * D + hh * D;

  bf16x8_t qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = frag_kc(Qp + (size_t)q * rs + ks * 16 + hf * 8);

  const int n_kb = qt + 1;  // key blocks 0..qt reach the tile's last row
  const int n_it = (n_kb + 1) / 2;
  TileLoad<D> tl;
  tl.init(rs, lane);
  const bf16_t* lsrc = (wave >> 1) ? Vp : Kp;
  auto load_stage = [&](int it, int stage) {  // wave w: tile w of the stage
    const int blk = 2 * it + (wave & 1);
    if (blk < n_kb) tl.issue(smem + (stage * 4 + wave) * TB, lsrc + (size_t)blk * 64 * rs);
  };

  f32x16_t oacc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[t][r] = 0.0f;
  float m = -INFINITY, l = 0.0f;

  // S = K Q^T of key block kb (LDS tile Kt) for this wave's 32 queries.
  auto scores = [&](const char* Kt, f32x16_t (&s)[2]) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[t][r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_row<LD>(Kt, t * 32 + l32, ks * 16 + hf * 8), qf[ks],
                                                       s[t], 0, 0, 0);
    }
  };
  // Causal mask, online softmax and O^T += V^T P^T with key block kb (tile Vt).
  auto softmax_pv = [&](const char* Vt, int k0, f32x16_t (&s)[2]) {
    // s[t][r]: key k0 + t*32 + (r/4)*8 + 4*hf + r%4, query q.  Only a block
    // that reaches past the wave's first query needs the causal mask.
    float mloc = -INFINITY;
    if (k0 + 63 > q0) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + t * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
          const float v = key > q ? -INFINITY : s[t][r] * scale_log2;
          s[t][r] = v;
          mloc = fmaxf(mloc, v);
        }
    } else {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[t][r] *= scale_log2;
          mloc = fmaxf(mloc, s[t][r]);
        }
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float mnew = fmaxf(m, mloc);
    if (__ballot(mnew > m)) {  // rescale only when some row's maximum grew
      const float alpha = __builtin_amdgcn_exp2f(m - mnew);
      l *= alpha;
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[t][r] *= alpha;
      m = mnew;
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(s[t][r] - m);
        s[t][r] = p;
        l += p;
      }
    bf16x8_t pb[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) pb[g] = cvt8(s[g >> 1], (g & 1) * 8);
    // O^T[d][q] += V^T[d][key] P^T[key][q]
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_tr<LD>(Vt, g * 16, dt * 32, lane), pb[g], oacc[dt],
                                                           0, 0, 0);
  };

  if constexpr (kAttnStages == 1 && D <= 96) {
    // One LDS stage, with K and V on separate schedules: the next block
    // pair's K tiles are fetched while this pair's softmax and P.V run, and
    // its V tiles while the next S = K Q^T runs.  Waves 0-1 load the K tiles
    // and waves 2-3 the V tiles; before a barrier that publishes tiles, only
    // the waves that loaded them wait for their own loads.  (At d = 128 the
    // scores held across the middle barrier would cost a wave per SIMD.)
    auto barrier = [&](bool wait_own_loads) {
      if (wait_own_loads) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    };
    load_stage(0, 0);
    for (int it = 0; it < n_it; ++it) {
      const int kb = 2 * it + kh, k0 = kb * 64;
      const bool active = kb < n_kb && k0 <= q0 + 31;
      f32x16_t s[2];
      barrier(wave < 2);  // K tiles of this pair landed
      if (active) scores(smem + kh * TB, s);
      barrier(wave >= 2);  // every wave is done with the K tiles; V tiles landed
      if (wave < 2 && it + 1 < n_it) load_stage(it + 1, 0);
      if (active) softmax_pv(smem + (2 + kh) * TB, k0, s);
      barrier(false);  // every wave is done with the V tiles
      if (wave >= 2 && it + 1 < n_it) load_stage(it + 1, 0);
    }
  } else {
    if (kAttnStages == 2) load_stage(0, 0);
    for (int it = 0; it < n_it; ++it) {
      const int cur = it % kAttnStages;
      if (kAttnStages == 1) {
        __syncthreads();  // every wave is done with the previous block pair
        load_stage(it, 0);
      }
      __syncthreads();  // this block pair landed (and, with two stages, the other stage is free)
      if (kAttnStages == 2 && it + 1 < n_it) load_stage(it + 1, (it + 1) % kAttnStages);
      const int kb = 2 * it + kh, k0 = kb * 64;
      if (kb >= n_kb || k0 > q0 + 31) continue;
      f32x16_t s[2];
      scores(smem + (cur * 4 + kh) * TB, s);
      softmax_pv(smem + (cur * 4 + 2 + kh) * TB, k0, s);
    }
  }

  // Merge the two key halves of each query group (partial m, l, O^T).
  constexpr int XS = 2 + DT * 16;
  static_assert((size_t)128 * XS * 4 <= (size_t)kAttnStages * 4 * TB, "merge buffer fits the tiles");
  float* xch = reinterpret_cast<float*>(smem) + (size_t)(qg * 64 + lane) * XS;
  __syncthreads();
  if (kh == 1) {
    xch[0] = m;
    xch[1] = l;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) xch[2 + t * 16 + r] = oacc[t][r];
  }
  __syncthreads();
  if (kh == 1) return;
  const float m1 = xch[0], l1 = xch[1];
  const float mt = fmaxf(m, m1);
  const float a0 = __builtin_amdgcn_exp2f(m - mt), a1 = __builtin_amdgcn_exp2f(m1 - mt);
  float lt = l * a0 + l1 * a1;
  lt += __shfl_xor(lt, 32, 64);
  const float inv = 1.0f / lt;
  bf16_t* orow = o + ((size_t)b * S + q) * H * D + hh * D;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        v[e] = (oacc[dt][4 * g + e] * a0 + xch[2 + dt * 16 + 4 * g + e] * a1) * inv;
      store4(orow + dt * 32 + g * 8 + hf * 4, v);
    }
  if (hf == 0) lse[((size_t)b * H + hh) * S + q] = (mt + log2f(lt)) * kLn2;
}

// ---------------------------------------------------------------------------
// delta[b, h, i] = sum_d dO[b, i, h, d] * O[b, i, h, d] (fp32 check mode; the
// bf16 dQ kernel forms it itself)
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(256) attn_delta_kernel(int B, int S, int H, int Bm, int mstride,
                                                         const T* __restrict__ o, const T* __restrict__ dout,
                                                         float* __restrict__ delta) {
  const int row = blockIdx.x * 256 + threadIdx.x;  // (launch batch, i, h) flattened
  if (row >= B * S * H) return;
  const int hh = row % H;
  const int bi = row / H;
  const int i = bi % S, b = seq_index(bi / S, Bm, mstride);
  const size_t trow = ((size_t)b * S + i) * H + hh;
  const T* orow = o + trow * D;
  const T* drow = dout + trow * D;
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < D; c += 8) {
    float a[8], d[8];
    load8(orow + c, a);
    load8(drow + c, d);
#pragma unroll
    for (int e = 0; e < 8; ++e) s += a[e] * d[e];
  }
  delta[((size_t)b * H + hh) * S + i] = s;
}

// ---------------------------------------------------------------------------
// bf16 backward: dK, dV (KV-parallel).  A workgroup owns 64 keys of one
// (batch, head); wave w takes the 32 keys of group w % 2 against the even
// (w < 2) or odd 64-query blocks from the diagonal on, and the two partial sums
// are added at the end.  Each stage holds the Q and dO tiles (and lse, delta)
// of two query blocks.  P is rebuilt from lse.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(256) attn_bwd_dkdv_bf16(int S, int H, int Bm, int mstride,
                                                          const bf16_t* __restrict__ qkv,
                                                          const bf16_t* __restrict__ dout,
                                                          const float* __restrict__ lse,
                                                          const float* __restrict__ delta,
                                                          bf16_t* __restrict__ dqkv, float scale_log2,
                                                          float scale) {
  using TT = AttnTile<D>;
  constexpr int LD = TT::LD, KS = D / 16, DT = D / 32, TB = TT::BYTES;
  extern __shared__ __align__(16) char smem[];  // [stage][Q a, Q b, dO a, dO b], then lse/delta
  float* vecs = reinterpret_cast<float*>(smem + kAttnStages * 4 * TB);  // [stage][lse a|b, delta a|b]

  // Grid (heads, sequences, key blocks), key block slowest: early keys see the
  // most queries, so the whole grid runs longest columns first.
  const int b = seq_index(blockIdx.y, Bm, mstride), hh = blockIdx.x;
  const int kt = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int kg = wave & 1, qh = wave >> 1;
  const int kw0 = kt * 64 + kg * 32;
  const int key = kw0 + l32;
  const size_t rs = (size_t)3 * H * D;
  const size_t ors = (size_t)H * D;
  const bf16_t* base = qkv + (size_t)b * S * rs;
  const bf16_t* Qp = base + hh * D;
  const bf16_t* Kp = base + (size_t)H * D + hh * D;
  const bf16_t* Vp = base + (size_t)2 * H * D + hh * D;
  const bf16_t* dOp = dout + (size_t)b * S * ors + hh * D;
  const float* lse_p = lse + ((size_t)b * H + hh) * S;
  const float* del_p = delta + ((size_t)b * H + hh) * S;

  bf16x8_t kf[KS], vf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    kf[ks] = frag_kc(Kp + (size_t)key * rs + ks * 16 + hf * 8);
    vf[ks] = frag_kc(Vp + (size_t)key * rs + ks * 16 + hf * 8);
  }
  f32x16_t dk[DT], dv[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[t][r] = dv[t][r] = 0.0f;

  const int n_qb = S / 64 - kt;  // query blocks kt .. S/64-1
  const int n_it = (n_qb + 1) / 2;
  const bool is_do = (wave >> 1) != 0;
  const size_t lgs = is_do ? ors : rs;
  TileLoad<D> tl;
  tl.init(lgs, lane);
  const bf16_t* lsrc = is_do ? dOp : Qp;
  const float* vsrc = is_do ? del_p : lse_p;
  auto load_stage = [&](int it, int stage) {
    const int blk = kt + 2 * it + (wave & 1);
    if (2 * it + (wave & 1) < n_qb) {
      tl.issue(smem + (stage * 4 + wave) * TB, lsrc + (size_t)blk * 64 * lgs);
      float* v = vecs + stage * 256 + (wave & 1) * 64 + (is_do ? 128 : 0);
      if (is_do) wave_vec_load(reinterpret_cast<char*>(v), vsrc + (size_t)blk * 64, lane);
      else v[lane] = vsrc[(size_t)blk * 64 + lane] * kLog2e;  // lse staged in log2 units
    }
  };

  if (kAttnStages == 2) load_stage(0, 0);
  for (int it = 0; it < n_it; ++it) {
    const int cur = it % kAttnStages;
    if (kAttnStages == 1) {
      __syncthreads();
      load_stage(it, 0);
    }
    __syncthreads();
    if (kAttnStages == 2 && it + 1 < n_it) load_stage(it + 1, (it + 1) % kAttnStages);
    const int qb = kt + 2 * it + qh, qs = qb * 64;
    if (2 * it + qh >= n_qb || qs + 63 < kw0) continue;
    const char* Qt = smem + (cur * 4 + qh) * TB;
    const char* dOt = smem + (cur * 4 + 2 + qh) * TB;
    const float* lse_s = vecs + cur * 256 + qh * 64;
    const float* del_s = lse_s + 128;

    // The two 32-query halves of the block one after the other (smaller live
    // register set); each dK/dV accumulator still takes its four 16-query
    // groups in order 0..3, so the sums are those of the whole block.
    const bool diag = qs < kw0 + 32;  // some query of the block precedes some key of the wave
    // Query qs + qi precedes this lane's key iff qi < key - qs.  With the lane's
    // part of qi (4 hf) folded in, one compare against a constant per score
    // decides; off the diagonal the limit is below every qi and masks nothing.
    const int mlim = (diag ? key - qs : -1) - hf * 4;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      f32x16_t p, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) p[r] = dp[r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        p = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_row<LD>(Qt, t * 32 + l32, ks * 16 + hf * 8), kf[ks], p, 0,
                                                    0, 0);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_row<LD>(dOt, t * 32 + l32, ks * 16 + hf * 8), vf[ks], dp,
                                                     0, 0, 0);
      }
      // p[r]: query qs + t*32 + (r/4)*8 + 4*hf + r%4, key `key`.
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qc = t * 32 + (r >> 2) * 8 + (r & 3);
        const int qi = qc + hf * 4;
        float pv = __builtin_amdgcn_exp2f(fmaf(p[r], scale_log2, -lse_s[qi]));
        if (qc < mlim) pv = 0.0f;
        p[r] = pv;
        dp[r] = pv * (dp[r] - del_s[qi]);
      }
      const bf16x8_t pb[2] = {cvt8(p, 0), cvt8(p, 8)};
      const bf16x8_t sb[2] = {cvt8(dp, 0), cvt8(dp, 8)};
      // dV^T[d][key] += dO^T[d][q] P[q][key];  dK^T[d][key] += Q^T[d][q] dS[q][key]
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int gg = 0; gg < 2; ++gg) {
          const int g = 2 * t + gg;
          dv[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_tr<LD>(dOt, g * 16, dt * 32, lane), pb[gg], dv[dt],
                                                           0, 0, 0);
          dk[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_tr<LD>(Qt, g * 16, dt * 32, lane), sb[gg], dk[dt],
                                                           0, 0, 0);
        }
    }
  }

  // Add the two query halves.
  constexpr int XS = 2 * DT * 16;
  static_assert((size_t)128 * XS * 4 <= (size_t)kAttnStages * 4 * TB, "merge buffer fits the tiles");
  float* xch = reinterpret_cast<float*>(smem) + (size_t)(kg * 64 + lane) * XS;
  __syncthreads();
  if (qh == 1) {
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        xch[t * 16 + r] = dk[t][r];
        xch[DT * 16 + t * 16 + r] = dv[t][r];
      }
  }
  __syncthreads();
  if (qh == 1) return;
  bf16_t* krow = dqkv + ((size_t)b * S + key) * rs + (size_t)H * D + hh * D;
  bf16_t* vrow = krow + (size_t)H * D;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float a[4], c[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[e] = (dk[dt][4 * g + e] + xch[dt * 16 + 4 * g + e]) * scale;
        c[e] = dv[dt][4 * g + e] + xch[DT * 16 + dt * 16 + 4 * g + e];
      }
      store4(krow + dt * 32 + g * 8 + hf * 4, a);
      store4(vrow + dt * 32 + g * 8 + hf * 4, c);
    }
}

// ---------------------------------------------------------------------------
// bf16 backward: dQ (Q-parallel), the forward's layout: 64 query rows per
// workgroup, 2 query groups x 2 key halves, K and V tiles of two key blocks per
// stage, partial dQ sums added at the end.  It also writes delta for its rows,
// which the dK/dV kernel launched after it reads.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(256) attn_bwd_dq_bf16(int S, int H, int Bm, int mstride,
                                                        const bf16_t* __restrict__ qkv,
                                                        const bf16_t* __restrict__ o,
                                                        const bf16_t* __restrict__ dout,
                                                        const float* __restrict__ lse,
                                                        float* __restrict__ delta,
                                                        bf16_t* __restrict__ dqkv, float scale_log2, float scale) {
  using TT = AttnTile<D>;
  constexpr int LD = TT::LD, KS = D / 16, DT = D / 32, TB = TT::BYTES;
  extern __shared__ __align__(16) char smem[];

  const int b = seq_index(blockIdx.y, Bm, mstride), hh = blockIdx.x;  // grid as in the forward
  const int qt = gridDim.z - 1 - blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int qg = wave & 1, kh = wave >> 1;
  const int q0 = qt * 64 + qg * 32;
  const int q = q0 + l32;
  const size_t rs = (size_t)3 * H * D;
  const size_t ors = (size_t)H * D;
  const bf16_t* base = qkv + (size_t)b * S * rs;
  const bf16_t* Qp = base + hh * D;
  const bf16_t* Kp = base + (size_t)H * D + hh * D;
  const bf16_t* Vp = base + (size_t)2 * H * D + hh * D;
  const bf16_t* dOp = dout + (size_t)b * S * ors + hh * D;

  bf16x8_t qf[KS], of[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qf[ks] = frag_kc(Qp + (size_t)q * rs + ks * 16 + hf * 8);
    of[ks] = frag_kc(dOp + (size_t)q * ors + ks * 16 + hf * 8);
  }
  const float lse2 = lse[((size_t)b * H + hh) * S + q] * kLog2e;
  // delta = dO . O over the head dimension for this query: the lane holds
  // half of the row's elements (the fragments above), lane ^ 32 the other
  // half.  Written out for the dK/dV kernel, which runs after this one.
  float del;
  {
    const bf16_t* Op = o + (size_t)b * S * ors + hh * D;
    float part = 0.0f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      float ov[8], dv[8];
      load8(Op + (size_t)q * ors + ks * 16 + hf * 8, ov);
      load8(dOp + (size_t)q * ors + ks * 16 + hf * 8, dv);
#pragma unroll
      for (int e = 0; e < 8; ++e) part += dv[e] * ov[e];
    }
    del = part + __shfl_xor(part, 32, 64);
    if (kh == 0 && hf == 0) delta[((size_t)b * H + hh) * S + q] = del;
  }
  f32x16_t dq[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[t][r] = 0.0f;

  const int n_kb = qt + 1;
  const int n_it = (n_kb + 1) / 2;
  TileLoad<D> tl;
  tl.init(rs, lane);
  const bf16_t* lsrc = (wave >> 1) ? Vp : Kp;
  auto load_stage = [&](int it, int stage) {
    const int blk = 2 * it + (wave & 1);
    if (blk < n_kb) tl.issue(smem + (stage * 4 + wave) * TB, lsrc + (size_t)blk * 64 * rs);
  };

  if (kAttnStages == 2) load_stage(0, 0);
  for (int it = 0; it < n_it; ++it) {
    const int cur = it % kAttnStages;
    if (kAttnStages == 1) {
      __syncthreads();
      load_stage(it, 0);
    }
    __syncthreads();
    if (kAttnStages == 2 && it + 1 < n_it) load_stage(it + 1, (it + 1) % kAttnStages);
    const int kb = 2 * it + kh, k0 = kb * 64;
    if (kb >= n_kb || k0 > q0 + 31) continue;
    const char* Kt = smem + (cur * 4 + kh) * TB;
    const char* Vt = smem + (cur * 4 + 2 + kh) * TB;
    f32x16_t p[2], dp[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) p[t][r] = dp[t][r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        p[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_row<LD>(Kt, t * 32 + l32, ks * 16 + hf * 8), qf[ks], p[t],
                                                       0, 0, 0);
        dp[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_row<LD>(Vt, t * 32 + l32, ks * 16 + hf * 8), of[ks],
                                                        dp[t], 0, 0, 0);
      }
    }
    // the causal mask only on a block that reaches past the wave's first query
    auto probs = [&](auto diag_c) {
      constexpr bool DIAG = decltype(diag_c)::value;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kk = k0 + t * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
          float pv = __builtin_amdgcn_exp2f(fmaf(p[t][r], scale_log2, -lse2));
          if (DIAG && kk > q) pv = 0.0f;
          dp[t][r] = pv * (dp[t][r] - del);
        }
    };
    if (k0 + 63 > q0) probs(std::true_type{});
    else probs(std::false_type{});
    bf16x8_t sb[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) sb[g] = cvt8(dp[g >> 1], (g & 1) * 8);
    // dQ^T[d][q] += K^T[d][key] dS^T[key][q]
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        dq[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_tr<LD>(Kt, g * 16, dt * 32, lane), sb[g], dq[dt], 0, 0, 0);
  }

  constexpr int XS = DT * 16;
  static_assert((size_t)128 * XS * 4 <= (size_t)kAttnStages * 4 * TB, "merge buffer fits the tiles");
  float* xch = reinterpret_cast<float*>(smem) + (size_t)(qg * 64 + lane) * XS;
  __syncthreads();
  if (kh == 1) {
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) xch[t * 16 + r] = dq[t][r];
  }
  __syncthreads();
  if (kh == 1) return;
  bf16_t* qrow = dqkv + ((size_t)b * S + q) * rs + hh * D;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float a[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) a[e] = (dq[dt][4 * g + e] + xch[dt * 16 + 4 * g + e]) * scale;
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
// Explicit instantiations of the bf16 kernels (the host pass then always emits
// their launch stubs).
#define MERAK_ATTN_INST(D)                                                                                        \
  template __global__ void attn_fwd_bf16<D>(int, int, int, int, const bf16_t* __restrict__, bf16_t* __restrict__, \
                                            float* __restrict__, float);                                         \
  template __global__ void attn_bwd_dkdv_bf16<D>(int, int, int, int, const bf16_t* __restrict__,                 \
                                                 const bf16_t* __restrict__, const float* __restrict__,          \
                                                 const float* __restrict__, bf16_t* __restrict__, float, float); \
  template __global__ void attn_bwd_dq_bf16<D>(int, int, int, int, const bf16_t* __restrict__,                   \
                                               const bf16_t* __restrict__, const bf16_t* __restrict__,           \
                                               const float* __restrict__, float* __restrict__,                   \
                                               bf16_t* __restrict__, float, float);
MERAK_ATTN_INST(64)
MERAK_ATTN_INST(96)
MERAK_ATTN_INST(128)
#undef MERAK_ATTN_INST

// Allow a kernel's dynamic LDS beyond the default limit on the current device.
template <typename K>
static hipError_t allow_lds(K kern, size_t bytes, std::atomic<uint64_t>& done) {
  return allow_dynamic_lds(reinterpret_cast<const void*>(kern), bytes, done);
}

template <int D>
static hipError_t fwd_d(int dtype, int B, int S, int H, int G, int mstride, const void* qkv, void* o, float* lse,
                        hipStream_t st) {
  const float scale = 1.0f / sqrtf((float)D);
  if (dtype == DT_BF16) {
    constexpr size_t lds = attn_lds_bytes<D>();
    static std::atomic<uint64_t> ok{0};
    hipError_t e = allow_lds(attn_fwd_bf16<D>, lds, ok);
    if (e != hipSuccess) return e;
    dim3 grid(H, G * B, S / 64);
    hipLaunchKernelGGL((attn_fwd_bf16<D>), grid, dim3(256), lds, st, S, H, B, mstride, (const bf16_t*)qkv,
                       (bf16_t*)o, lse, scale * kLog2e);
  } else {
    const size_t rs = (size_t)3 * H * D, seq_rows = (size_t)mstride * S;
    for (int m = 0; m < G; ++m) {
      dim3 grid((B * H * S + 127) / 128);
      hipLaunchKernelGGL((attn_fwd_f32<D>), grid, dim3(128), 0, st, B, S, H,
                         (const float*)qkv + m * seq_rows * rs, (float*)o + m * seq_rows * H * D,
                         lse + m * seq_rows * H, scale);
    }
  }
  return hipGetLastError();
}

template <int D>
static hipError_t bwd_d(int dtype, int B, int S, int H, int G, int mstride, const void* qkv, const void* o,
                        const float* lse, const void* dout, void* dqkv, float* delta, hipStream_t st) {
  const float scale = 1.0f / sqrtf((float)D);
  const int rows = G * B * S * H;
  if (dtype == DT_BF16) {
    constexpr size_t lds_q = attn_lds_bytes<D>();
    constexpr size_t lds_k = attn_lds_bytes<D>() + kAttnStages * 256 * sizeof(float);
    static_assert(lds_k <= 160 * 1024, "LDS budget");
    static std::atomic<uint64_t> ok_k{0}, ok_q{0};
    hipError_t e = allow_lds(attn_bwd_dkdv_bf16<D>, lds_k, ok_k);
    if (e == hipSuccess) e = allow_lds(attn_bwd_dq_bf16<D>, lds_q, ok_q);
    if (e != hipSuccess) return e;
    // dQ first: it also forms delta, which dK/dV reads.
    dim3 grid(H, G * B, S / 64);
    hipLaunchKernelGGL((attn_bwd_dq_bf16<D>), grid, dim3(256), lds_q, st, S, H, B, mstride, (const bf16_t*)qkv,
                       (const bf16_t*)o, (const bf16_t*)dout, lse, delta, (bf16_t*)dqkv, scale * kLog2e, scale);
    hipLaunchKernelGGL((attn_bwd_dkdv_bf16<D>), grid, dim3(256), lds_k, st, S, H, B, mstride, (const bf16_t*)qkv,
                       (const bf16_t*)dout, lse, delta, (bf16_t*)dqkv, scale * kLog2e, scale);
  } else {
    hipLaunchKernelGGL((attn_delta_kernel<float, D>), dim3((rows + 255) / 256), dim3(256), 0, st, G * B, S, H, B,
                       mstride, (const float*)o, (const float*)dout, delta);
    const size_t rs = (size_t)3 * H * D, seq_rows = (size_t)mstride * S;
    for (int m = 0; m < G; ++m) {
      const float* q_m = (const float*)qkv + m * seq_rows * rs;
      const float* do_m = (const float*)dout + m * seq_rows * H * D;
      const float* lse_m = lse + m * seq_rows * H;
      const float* del_m = delta + m * seq_rows * H;
      float* dq_m = (float*)dqkv + m * seq_rows * rs;
      dim3 grid((B * H * S + 127) / 128);
      hipLaunchKernelGGL((attn_bwd_dkdv_f32<D>), grid, dim3(128), 0, st, B, S, H, q_m, do_m, lse_m, del_m, dq_m,
                         scale);
      hipLaunchKernelGGL((attn_bwd_dq_f32<D>), grid, dim3(128), 0, st, B, S, H, q_m, do_m, lse_m, del_m, dq_m,
                         scale);
    }
  }
  return hipGetLastError();
}

hipError_t launch_attention_fwd(int dtype, int batch, int seq, int heads, int d, const void* qkv, void* o,
                                float* lse, hipStream_t stream, int members, int member_stride) {
  if (batch <= 0 || seq <= 0 || heads <= 0 || members <= 0) return hipSuccess;
  if (seq % 64 != 0 || (members > 1 && member_stride < batch)) return hipErrorInvalidValue;
  switch (d) {
    case 64: return fwd_d<64>(dtype, batch, seq, heads, members, member_stride, qkv, o, lse, stream);
    case 96: return fwd_d<96>(dtype, batch, seq, heads, members, member_stride, qkv, o, lse, stream);
    case 128: return fwd_d<128>(dtype, batch, seq, heads, members, member_stride, qkv, o, lse, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attention_bwd(int dtype, int batch, int seq, int heads, int d, const void* qkv, const void* o,
                                const float* lse, const void* dout, void* dqkv, float* delta, hipStream_t stream,
                                int members, int member_stride) {
  if (batch <= 0 || seq <= 0 || heads <= 0 || members <= 0) return hipSuccess;
  if (seq % 64 != 0 || (members > 1 && member_stride < batch)) return hipErrorInvalidValue;
  switch (d) {
    case 64: return bwd_d<64>(dtype, batch, seq, heads, members, member_stride, qkv, o, lse, dout, dqkv, delta, stream);
    case 96: return bwd_d<96>(dtype, batch, seq, heads, members, member_stride, qkv, o, lse, dout, dqkv, delta, stream);
    case 128:
      return bwd_d<128>(dtype, batch, seq, heads, members, member_stride, qkv, o, lse, dout, dqkv, delta, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace merak
