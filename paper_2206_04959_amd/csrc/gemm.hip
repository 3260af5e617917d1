// GEMM kernels for the shard's linear layers.
//
//   forward   X W^T      (A row-major [M,K], B = weight [N,K])          a_t=0 b_t=0
//   backward  dY W       (A row-major [M,K], B = weight [K,N])          a_t=0 b_t=1
//   weights   dY^T X     (A = dY [K,M] read transposed, B = X [K,N])    a_t=1 b_t=1
//
// bf16 path: v_mfma_f32_32x32x16_bf16 with fp32 accumulation.  Operand tiles
// (BK = 64) go from global memory straight into an LDS ring (buffer loads that
// write LDS, no register staging) in XOR-swizzled layouts chosen for the 64
// banks of gfx950 LDS; operands contiguous along M or N stay that way in LDS
// and are read with the transposing LDS read, so no operand is transposed in
// registers.  Each wave reads the fragments of the next K sub-step while the
// MFMAs of the current one run, with one workgroup barrier per K stage; the
// fragment reads and the loads of later stages are issued one at a time
// between the MFMAs rather than in bursts.  The
// MFMA takes the B tile as its first operand so each lane owns one output row
// and 4 consecutive columns per group, which the fused epilogues store as one
// vector.  Workgroups are mapped to tiles so that each of the 8 XCDs works on
// a compact block of neighbouring tiles (operand reuse in its own L2).
//
// fp32 check mode: a plain LDS-tiled FMA kernel with the same layouts and
// epilogues.
#include <atomic>
#include <type_traits>

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
      if (p.aux) store4(reinterpret_cast<T*>(p.aux) + off, v);
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

// ---------------------------------------------------------------------------
// Epilogue on 8 consecutive columns n..n+7 of row m (16-byte bf16 / 32-byte
// fp32 accesses).
// ---------------------------------------------------------------------------
// `pre`, when given, holds the [M, N] operand the epilogue reads (the residual,
// or the stored GeLU input), fetched ahead of time.
template <typename T, int EPI>
__device__ __forceinline__ void epilogue8(const GemmProblem& p, int m, int n, float v[8],
                                          const u32x4_t* pre = nullptr) {
  const size_t off = (size_t)m * p.ldc + n;
  if constexpr (EPI == EPI_F32) {
    float* c = reinterpret_cast<float*>(p.c) + off;
    if (p.accumulate) {
      float o[8];
      load8(c, o);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += o[e];
    }
    store8(c, v);
  } else {
    T* c = reinterpret_cast<T*>(p.c) + off;
    if constexpr (EPI == EPI_STORE) {
      store8(c, v);
    } else if constexpr (EPI == EPI_BIAS) {
      float b[8];
      load8(reinterpret_cast<const T*>(p.bias) + n, b);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += b[e];
      store8(c, v);
    } else if constexpr (EPI == EPI_BIAS_GELU) {
      float b[8], g[8];
      load8(reinterpret_cast<const T*>(p.bias) + n, b);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[e] += b[e];
        g[e] = gelu_f(v[e]);
      }
      if (p.aux) store8(reinterpret_cast<T*>(p.aux) + off, v);
      store8(c, g);
    } else if constexpr (EPI == EPI_BIAS_RESID) {
      float b[8], r[8];
      if (p.aux) store8(reinterpret_cast<T*>(p.aux) + off, v);
      load8(reinterpret_cast<const T*>(p.bias) + n, b);
      if (pre) unpack8(*pre, r);
      else load8(reinterpret_cast<const T*>(p.resid) + off, r);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = r[e] + v[e] + b[e];
      store8(c, v);
    } else if constexpr (EPI == EPI_GELU_BWD) {
      float u[8];
      if (pre) unpack8(*pre, u);
      else load8(reinterpret_cast<const T*>(p.aux) + off, u);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] *= gelu_grad_f(u[e]);
      store8(c, v);
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
//
// LDS stage (one BK = 64 slice of K) of an operand with R tile rows (R = BM
// for A, BN for B) occupies R * 128 bytes, in one of two layouts:
//   K-contiguous operand: [R][64 k]; the 16-byte chunk c of row r is stored in
//     slot c ^ ((r >> 1) & 7), so the 16 rows read by one 256-byte pass of a
//     fragment read land in distinct banks (gfx950 LDS: 64 banks of 4 bytes);
//   MN-contiguous operand: [64 k][R]; chunk c of k-row k is stored in slot
//     (c + 4 * (k & 3)) mod (R / 8), so the four k-rows of a transposing read
//     pass land in distinct quarters of the 256-byte bank space (R = 128, 192
//     or 256).
// Tiles move global -> LDS with buffer loads that write LDS directly (no VGPR
// staging); each wave instruction fills 1 KiB of LDS, lane i writing bytes
// [16 i, 16 i + 16), and the swizzle is applied by choosing which global
// chunk each lane fetches.  Rows or columns past the operand's extent read as
// zero (buffer range check) or as in-range data whose products land only in
// discarded outputs.  MN-contiguous fragments are read with the gfx950
// transposing LDS read (ds_read_b64_tr_b16), which hands lane i of each
// 16-lane group the i-th column of the 4 x 16 block its group fetched.
// ---------------------------------------------------------------------------
constexpr int kBK = 64;

typedef short s16x4_t __attribute__((ext_vector_type(4)));
#define MERAK_LDS __attribute__((address_space(3)))

__device__ __forceinline__ __amdgpu_buffer_rsrc_t operand_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// Workgroup id -> tile id such that each of the 8 XCDs (which receive
// workgroups round-robin) works on one contiguous range of tiles.
__device__ __forceinline__ int xcd_remap(int bid, int n) {
  const int per = n >> 3, rem = n & 7, x = bid & 7, idx = bid >> 3;
  return (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + idx;
}

// One 16-byte-per-lane global -> LDS load: lane i writes LDS bytes
// [lds_addr + 16 i, lds_addr + 16 i + 16).  Issued as inline assembly: the
// compiler would otherwise treat every later LDS read that it cannot prove
// disjoint from this store (the transposing reads among them) as dependent on
// it and wait for all outstanding loads before that read, which would serialise
// the prefetch of the next K stage with the MFMAs of the current one.  The
// kernels order these loads themselves (wait_vm_barrier).  An M0 write needs
// one wait state before an LDS-DMA load.
typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ i32x4_t operand_rsrc_words(const void* p, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  return i32x4_t{(int32_t)(uint32_t)a, (int32_t)(uint32_t)((a >> 32) & 0xffffu), (int32_t)bytes, 0x00020000};
}

__device__ __forceinline__ void lds_dma16(i32x4_t rsrc, uint32_t lds_addr, uint32_t voff) {
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(voff), "s"(rsrc), "{m0}"(lds_addr)
               : "memory");
}

__device__ __forceinline__ uint32_t lds_address(const char* p) {
  return (uint32_t)(uintptr_t)(const MERAK_LDS char*)p;
}

// Global -> LDS loader of one operand.  Each wave issues kInst 16-byte-per-lane
// loads per K stage.
template <bool TRANS, int R, int NW>
struct TileLoader {
  static constexpr int kInst = R / 8 / NW;
  static_assert(R / 8 % NW == 0, "tile rows must split evenly over the waves");
  static_assert(!TRANS || (R % 32 == 0 && R >= 128), "MN-contiguous tiles: width a multiple of 32, at least 128");
  uint32_t voff[kInst];
  uint32_t step;  // bytes to advance per K stage

  __device__ __forceinline__ void init(int r0, int ld, int wave, int lane) {
#pragma unroll
    for (int q = 0; q < kInst; ++q) {
      if constexpr (!TRANS) {
        const int row = (q * NW + wave) * 8 + (lane >> 3);
        const int chunk = (lane & 7) ^ ((row >> 1) & 7);
        voff[q] = (uint32_t)((r0 + row) * ld + chunk * 8) * 2u;
      } else {
        constexpr int CPR = R / 8;  // 16-byte chunks per k-row
        const int g = (q * NW + wave) * 64 + lane;  // chunk index within the stage
        const int kr = g / CPR, slot = g % CPR;
        const int chunk = (slot + CPR - 4 * (kr & 3)) % CPR;  // chunk stored in this slot
        voff[q] = (uint32_t)(kr * ld + r0 + chunk * 8) * 2u;
      }
    }
    step = TRANS ? (uint32_t)(kBK * ld * 2) : (uint32_t)(kBK * 2);
  }

  // Issue load q of the current K stage into `lds` (R * 128 bytes); after the
  // last one (q = kInst - 1) the loader moves on to the next stage.
  __device__ __forceinline__ void issue_one(i32x4_t rsrc, char* lds, int wave, int q) {
    const uint32_t addr = __builtin_amdgcn_readfirstlane(lds_address(lds) + (q * NW + wave) * 1024);
    lds_dma16(rsrc, addr, voff[q]);
    voff[q] += step;
  }

  // Issue the loads of the current K stage into `lds` (R * 128 bytes) and move
  // on to the next stage.
  __device__ __forceinline__ void issue(i32x4_t rsrc, char* lds, int wave) {
#pragma unroll
    for (int q = 0; q < kInst; ++q) {
      const uint32_t addr = __builtin_amdgcn_readfirstlane(lds_address(lds) + (q * NW + wave) * 1024);
      lds_dma16(rsrc, addr, voff[q]);
      voff[q] += step;
    }
  }
};

// Fragment reader: the 32 x 16 (rows x k) MFMA operand block starting at tile
// row `row0` (a multiple of 32) and k = 16 * ks of an LDS stage.  Lane l gets
// row row0 + l % 32 and k = 16 ks + 8 (l / 32) + 0..7.
template <bool TRANS, int R>
struct FragReader {
  static constexpr int kInstPerFrag = TRANS ? 2 : 1;  // LDS read instructions per fragment
  int lane_off;  // lane-dependent part of the byte offset
  int key;       // lane-dependent swizzle term

  __device__ __forceinline__ void init(int lane) {
    if constexpr (!TRANS) {
      lane_off = (lane & 31) * 128;
      key = (lane >> 5) ^ (((lane & 31) >> 1) & 7);
    } else {
      const int b = lane >> 4, j = lane & 15;
      lane_off = ((b >> 1) * 8 + (j >> 2)) * (2 * R) + ((b & 1) * 2 + ((j >> 1) & 1)) * 16 + (j & 1) * 8;
      key = (j >> 2) << 2;  // slot rotation of this lane's k-row (k & 3 = j / 4)
    }
  }

  __device__ __forceinline__ bf16x8_t read(const char* lds, int row0, int ks) const {
    if constexpr (!TRANS) {
      const char* p = lds + row0 * 128 + lane_off + (((2 * ks) ^ key) << 4);
      return *reinterpret_cast<const bf16x8_t*>(p);
    } else {
      constexpr int CPR = R / 8;
      const char* p = lds + ks * 16 * (2 * R) + ((((row0 >> 3) + key) % CPR) << 4) + lane_off;
      s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((MERAK_LDS s16x4_t*)(p));
      s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((MERAK_LDS s16x4_t*)(p + 4 * (2 * R)));
      s16x4_t v01 = lo, v23 = hi;
      typedef short s16x8_t __attribute__((ext_vector_type(8)));
      s16x8_t v = {v01[0], v01[1], v01[2], v01[3], v23[0], v23[1], v23[2], v23[3]};
      return __builtin_bit_cast(bf16x8_t, v);
    }
  }
};

// Wait until at most N of this wave's vector-memory loads are outstanding and
// all its LDS reads have completed, then join the workgroup barrier.  (The
// buffer loads that write LDS directly are tracked by vmcnt only.)
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

template <int BM, int BN, int WM, int WN, int NS, bool A_T, bool B_T, int EPI>
__global__ void __launch_bounds__(WM * WN * 64) gemm_mfma_kernel(GemmBatch batch) {
  constexpr int NW = WM * WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;  // wave tile
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int A_BYTES = BM * 128, STAGE = (BM + BN) * 128;
  extern __shared__ __align__(16) char smem[];

  const int tile_id = xcd_remap(blockIdx.x, batch.tile_start[kMaxGroup]);
  int tile0;
  const GemmProblem p = select_problem(batch, tile_id, &tile0);
  const int tile = tile_id - tile0;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  // Groups of 4 tile rows walked column by column, so that neighbouring tiles
  // (same XCD) share operand panels in L2.
  constexpr int GM = 4;
  const int group = tile / (GM * tiles_n);
  const int first_m = group * GM;
  const int gsz = min(tiles_m - first_m, GM);
  const int in_group = tile - group * GM * tiles_n;
  const int m0 = (first_m + in_group % gsz) * BM;
  const int n0 = (in_group / gsz) * BN;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WN, wn = wave % WN;

  const uint32_t a_bytes = A_T ? (uint32_t)(((size_t)(p.K - 1) * p.lda + p.M) * 2)
                               : (uint32_t)(((size_t)(p.M - 1) * p.lda + p.K) * 2);
  const uint32_t b_bytes = B_T ? (uint32_t)(((size_t)(p.K - 1) * p.ldb + p.N) * 2)
                               : (uint32_t)(((size_t)(p.N - 1) * p.ldb + p.K) * 2);
  const i32x4_t ra = operand_rsrc_words(p.a, a_bytes);
  const i32x4_t rb = operand_rsrc_words(p.b, b_bytes);

  TileLoader<A_T, BM, NW> la;
  TileLoader<B_T, BN, NW> lb;
  la.init(m0, p.lda, wave, lane);
  lb.init(n0, p.ldb, wave, lane);
  FragReader<A_T, BM> fa;
  FragReader<B_T, BN> fb;
  fa.init(lane);
  fb.init(lane);

  f32x16_t acc[TN][TM];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[j][i][e] = 0.0f;

  // Software pipeline over an NS-stage LDS ring.  Fragments of K sub-step
  // ks + 1 are read while the MFMAs of sub-step ks run (two register sets).
  // The one barrier per K stage sits before the last sub-step: by then every
  // wave has read all fragments of stage kt, so the loads of stage kt + NS may
  // overwrite it (issued during that last sub-step and the first sub-step of
  // stage kt + 1), and the first fragments of stage kt + 1 are read while the
  // last MFMAs of stage kt run.  Before the barrier each wave waits only for
  // its own loads of stage kt + 1 (later stages stay in flight).
  constexpr int LPT = TileLoader<A_T, BM, NW>::kInst + TileLoader<B_T, BN, NW>::kInst;  // loads per stage
  const int KT = p.K / kBK;
  bf16x8_t a0[TM], a1[TM], b0[TN], b1[TN];  // two fragment register sets
  auto read_frags = [&](const char* st, int ks, bf16x8_t (&a)[TM], bf16x8_t (&b)[TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i) a[i] = fa.read(st, wm * WTM + i * 32, ks);
#pragma unroll
    for (int j = 0; j < TN; ++j) b[j] = fb.read(st + A_BYTES, wn * WTN + j * 32, ks);
  };
  auto mfmas = [&](const bf16x8_t (&a)[TM], const bf16x8_t (&b)[TN]) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int i = 0; i < TM; ++i)
        acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[j], a[i], acc[j][i], 0, 0, 0);
  };
  auto issue = [&](int stage) {
    char* st = smem + stage * STAGE;
    la.issue(ra, st, wave);
    lb.issue(rb, st + A_BYTES, wave);
  };
  // Instruction order within a sub-step.  The fragment reads of the next
  // sub-step do not feed the MFMAs of this one, so they are spread between
  // them (MFMA, read, MFMA, read, ...) rather than issued as one burst ahead
  // of the MFMAs: a burst of LDS reads from every wave of the workgroup at
  // once holds up the waves' MFMA issue.  The same holds for the global ->
  // LDS loads of a later stage, which go out one after each MFMA, split over
  // two sub-steps (step_loads).  Each such placement is pinned with
  // scheduling fences, in one code path for the loop body: a second path (a
  // variant of the sub-step without loads for the last stages) made the
  // compiler rename the accumulators between the paths and spill.
  constexpr int NRD = TM * FragReader<A_T, BM>::kInstPerFrag + TN * FragReader<B_T, BN>::kInstPerFrag;
  constexpr int NMF = TM * TN;
  constexpr int NIL = NRD > NMF ? NRD : NMF;
  constexpr int LA = TileLoader<A_T, BM, NW>::kInst;
  // reads of (st, ks) into set n, interleaved with the MFMAs of set c
  auto step = [&](const char* st, int ks, bf16x8_t (&na)[TM], bf16x8_t (&nb)[TN], const bf16x8_t (&ca)[TM],
                  const bf16x8_t (&cb)[TN]) {
    read_frags(st, ks, na, nb);
    mfmas(ca, cb);
#pragma unroll
    for (int i = 0; i < NIL; ++i) {
      if (i < NMF) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      if (i < NRD) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // The MFMAs of set c, each followed by global -> LDS load q (q in [Q0, Q1)
  // of the stage held in LDS buffer `stage`, if do_loads), then the reads of
  // (st, ks) into set n.
  auto step_loads = [&](const char* st, int ks, bf16x8_t (&na)[TM], bf16x8_t (&nb)[TN], const bf16x8_t (&ca)[TM],
                        const bf16x8_t (&cb)[TN], int stage, bool do_loads, auto q0c, auto q1c) {
    constexpr int Q0 = decltype(q0c)::value, Q1 = decltype(q1c)::value;
    constexpr int NML = NMF > Q1 - Q0 ? NMF : Q1 - Q0;
    char* ld = smem + stage * STAGE;
#pragma unroll
    for (int u = 0; u < NML; ++u) {
      if (u < NMF)
        acc[u / TM][u % TM] =
            __builtin_amdgcn_mfma_f32_32x32x16_bf16(cb[u / TM], ca[u % TM], acc[u / TM][u % TM], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      const int q = Q0 + u;
      if (q < Q1) {
        if (q < LA) {
          if (do_loads) la.issue_one(ra, ld, wave, q);
        } else {
          if (do_loads) lb.issue_one(rb, ld + A_BYTES, wave, q - LA);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    read_frags(st, ks, na, nb);
    __builtin_amdgcn_sched_barrier(0);
  };
  constexpr int LH = (LPT + 1) / 2;  // loads of a stage issued right after the barrier; the rest a sub-step later

#pragma unroll
  for (int s = 0; s < NS; ++s)
    if (s < KT) issue(s);
  if (KT >= NS) wait_vm_barrier<(NS - 1) * LPT>();
  else wait_vm_barrier<0>();
  read_frags(smem, 0, a0, b0);
  __builtin_amdgcn_sched_barrier(0);

  static_assert(kBK / 16 == 4, "the sub-step sequence below assumes four sub-steps per stage");
  for (int kt = 0; kt < KT - 1; ++kt) {
    const int cur = kt % NS;
    const char* st = smem + cur * STAGE;
    // the second part of the loads of stage kt - 1 + NS, into the buffer stage kt - 1 used
    step_loads(st, 1, a1, b1, a0, b0, (kt + NS - 1) % NS, kt >= 1 && kt - 1 + NS < KT,
               std::integral_constant<int, LH>{}, std::integral_constant<int, LPT>{});
    step(st, 2, a0, b0, a1, b1);
    step(st, 3, a1, b1, a0, b0);
    if (kt + NS - 1 < KT) wait_vm_barrier<(NS - 2) * LPT>();
    else wait_vm_barrier<0>();
    step_loads(smem + ((kt + 1) % NS) * STAGE, 0, a0, b0, a1, b1, cur, kt + NS < KT,
               std::integral_constant<int, 0>{}, std::integral_constant<int, LH>{});
  }
  // Epilogues that read a [M, N] operand fetch this lane's chunks of it for
  // the first 32-row slab (in the row-contiguous layout of the staged epilogue
  // below) before the last K stage, so that the loads overlap its MFMAs.
  constexpr int CPR = WTN / 8;          // 8-column chunks per row of a wave tile
  constexpr int CPL = 32 * CPR / 64;    // chunks per lane in a 32-row slab
  static_assert((32 * CPR) % 64 == 0, "whole chunks per lane");
  constexpr bool PRE = (EPI == EPI_BIAS_RESID || EPI == EPI_GELU_BWD) && CPL <= 8;
  u32x4_t pre[PRE ? CPL : 1];
  if constexpr (PRE) {
    const bf16_t* src = reinterpret_cast<const bf16_t*>(EPI == EPI_BIAS_RESID ? p.resid : p.aux);
#pragma unroll
    for (int u = 0; u < CPL; ++u) {
      const int q = lane + 64 * u;
      const int m = m0 + wm * WTM + q / CPR, n = n0 + wn * WTN + (q % CPR) * 8;
      pre[u] = (m < p.M && n < p.N) ? *reinterpret_cast<const u32x4_t*>(src + (size_t)m * p.ldc + n)
                                     : u32x4_t{0u, 0u, 0u, 0u};
    }
  }
  {
    const char* st = smem + ((KT - 1) % NS) * STAGE;
    step(st, 1, a1, b1, a0, b0);
    step(st, 2, a0, b0, a1, b1);
    step(st, 3, a1, b1, a0, b0);
    mfmas(a1, b1);
  }
  // acc[j][i][r]: output row m = m0 + wm*WTM + i*32 + lane%32,
  // column n = n0 + wn*WTN + j*32 + (r/4)*8 + (lane/32)*4 + r%4.
  // Epilogue through LDS, one 32-row slab of the wave tile at a time: the
  // accumulators (row = lane % 32, four columns per register quad) go to a
  // padded fp32 staging tile, and are read back as 8 consecutive columns per
  // lane, so that consecutive lanes cover contiguous row segments of C and of
  // the epilogue's operands (16-byte accesses instead of 8-byte pieces of 32
  // rows).
  constexpr int CLD = WTN + 4;  // staging row, fp32
  static_assert((size_t)NW * 32 * CLD * 4 <= (size_t)NS * STAGE, "epilogue staging fits in the operand ring");
  float* stg = reinterpret_cast<float*>(smem) + wave * 32 * CLD;
  __syncthreads();  // every wave has finished reading operand tiles
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4_t*>(stg + (lane & 31) * CLD + j * 32 + g * 8 + (lane >> 5) * 4) =
            f32x4_t{acc[j][i][4 * g], acc[j][i][4 * g + 1], acc[j][i][4 * g + 2], acc[j][i][4 * g + 3]};
    // The staging tile is this wave's own: its LDS accesses complete in order,
    // so a wait for its own writes (not a workgroup barrier) orders them.
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int u = 0; u < CPL; ++u) {
      const int q = lane + 64 * u;
      const int r = q / CPR, cc = q % CPR;
      const int m = m0 + wm * WTM + i * 32 + r;
      const int n = n0 + wn * WTN + cc * 8;
      if (m < p.M && n < p.N) {
        float v[8];
        const f32x4_t lo = *reinterpret_cast<const f32x4_t*>(stg + r * CLD + cc * 8);
        const f32x4_t hi = *reinterpret_cast<const f32x4_t*>(stg + r * CLD + cc * 8 + 4);
        v[0] = lo[0]; v[1] = lo[1]; v[2] = lo[2]; v[3] = lo[3];
        v[4] = hi[0]; v[5] = hi[1]; v[6] = hi[2]; v[7] = hi[3];
        if constexpr (PRE) epilogue8<bf16_t, EPI>(p, m, n, v, i == 0 ? &pre[u] : nullptr);
        else epilogue8<bf16_t, EPI>(p, m, n, v);
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the slab is read before the next one overwrites it
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
template <int BM, int BN, int WM, int WN, int NS, bool AT, bool BT, int EPI>
static hipError_t run_mfma(GemmBatch& batch, hipStream_t stream) {
  int tiles = 0;
  for (int i = 0; i < batch.n_probs; ++i) {
    batch.tile_start[i] = tiles;
    tiles += ((batch.p[i].M + BM - 1) / BM) * ((batch.p[i].N + BN - 1) / BN);
  }
  for (int i = batch.n_probs; i <= kMaxGroup; ++i) batch.tile_start[i] = tiles;
  if (tiles == 0) return hipSuccess;
  constexpr size_t lds = (size_t)NS * (BM + BN) * 128;
  static_assert(lds <= 160 * 1024, "LDS budget");
  auto kern = gemm_mfma_kernel<BM, BN, WM, WN, NS, AT, BT, EPI>;
  static std::atomic<uint64_t> lds_set{0};  // devices this instantiation's LDS limit is set on
  const hipError_t attr_err = allow_dynamic_lds(reinterpret_cast<const void*>(kern), lds, lds_set);
  if (attr_err != hipSuccess) return attr_err;
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

// Tile shapes of the bf16 kernel: BM x BN with WM x WN waves and NS LDS stages.
enum TileCfg {
  TILE_AUTO = 0,
  TILE_256x256_W4_S2 = 1,  // 2x2 waves of 128x128
  TILE_256x128_W4_S3 = 2,  // 2x2 waves of 128x64
  TILE_128x256_W4_S3 = 3,  // 2x2 waves of 64x128
  TILE_128x128_W4_S2 = 4,  // 2x2 waves of 64x64
  TILE_128x128_W4_S3 = 5,
  TILE_128x128_W4_S4 = 6,
  TILE_256x256_W8_S2 = 7,  // 2x4 waves of 128x64
  TILE_256x128_W8_S3 = 8,  // 4x2 waves of 64x64
  TILE_128x192_W4_S2 = 9,   // 2x2 waves of 64x96
  TILE_256x192_W8_S2 = 10,  // 4x2 waves of 64x96
  TILE_COUNT = 11
};
static std::atomic<int> g_tile_override{TILE_AUTO};

static long long tile_count(const GemmBatch& b, int bm, int bn) {
  long long t = 0;
  for (int i = 0; i < b.n_probs; ++i) t += (long long)((b.p[i].M + bm - 1) / bm) * ((b.p[i].N + bn - 1) / bn);
  return t;
}

// Tile choice (measured on MI355X with random bf16 data, isolated, as two
// concurrent launches, and inside the two-stream stage step).  Large tiles on
// 8 waves (two per SIMD) move the fewest operand bytes per FLOP through L2 and
// LDS: the input- and weight-gradient GEMMs (B read with M/N contiguous) run
// as 256 x 256 tiles, every other GEMM with at least 128 such tiles as
// 256 x 192 tiles.  Narrower problems (most GEMMs of stages with 2048-row
// sub-micro-batches) run as 256 x 128 tiles on 8 waves with a 3-stage ring
// while that still gives at least 100 tiles; the narrowest (the projection's
// input gradient at N = h/t = 768) keep 128 x 192 tiles on 4 waves, whose
// larger grid is faster alone and the same in the stage.  Against 128 x 192
// tiles everywhere the stage step measured +6.3% (819 -> 870 TFLOP/s);
// 256 x 256 tiles everywhere +3.6%, 256 x 192 everywhere +5.3% (before the
// instruction order of the main loop above); with that order, 256 x 256 for
// the weight gradients added 0.6%, while 256 x 192 for the smaller (QKV /
// projection) weight-gradient group lost 0.6%.  The 256 x 128 rule: +2.9% on
// the 1.5B-shaped stage, +1.8% on the 2.5B-shaped shard (their hidden sizes
// 1600 and 1920 make most of their GEMMs narrow), no change elsewhere.
static int choose_tile(const GemmBatch& b, bool a_t, bool b_t) {
  if (g_tile_override != TILE_AUTO) return g_tile_override;
  if (b_t && tile_count(b, 256, 256) >= 128) return TILE_256x256_W8_S2;
  if (tile_count(b, 256, 192) >= 128) return TILE_256x192_W8_S2;
  if (tile_count(b, 256, 128) >= 100) return TILE_256x128_W8_S3;
  return TILE_128x192_W4_S2;
}

template <bool AT, bool BT, int EPI>
static hipError_t run_bf16(GemmBatch& batch, hipStream_t stream) {
  switch (choose_tile(batch, AT, BT)) {
    case TILE_256x256_W4_S2: return run_mfma<256, 256, 2, 2, 2, AT, BT, EPI>(batch, stream);
    case TILE_256x128_W4_S3: return run_mfma<256, 128, 2, 2, 3, AT, BT, EPI>(batch, stream);
    case TILE_128x256_W4_S3: return run_mfma<128, 256, 2, 2, 3, AT, BT, EPI>(batch, stream);
    case TILE_128x128_W4_S3: return run_mfma<128, 128, 2, 2, 3, AT, BT, EPI>(batch, stream);
    case TILE_128x128_W4_S4: return run_mfma<128, 128, 2, 2, 4, AT, BT, EPI>(batch, stream);
    case TILE_256x256_W8_S2: return run_mfma<256, 256, 2, 4, 2, AT, BT, EPI>(batch, stream);
    case TILE_256x128_W8_S3: return run_mfma<256, 128, 4, 2, 3, AT, BT, EPI>(batch, stream);
    case TILE_128x192_W4_S2: return run_mfma<128, 192, 2, 2, 2, AT, BT, EPI>(batch, stream);
    case TILE_256x192_W8_S2: return run_mfma<256, 192, 4, 2, 2, AT, BT, EPI>(batch, stream);
    default: return run_mfma<128, 128, 2, 2, 2, AT, BT, EPI>(batch, stream);
  }
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
  for (int i = 0; i < n_probs; ++i)
    if (dtype == DT_BF16 && !gemm_bf16_offsets_fit(probs[i], a_t, b_t)) return hipErrorInvalidValue;
  GemmBatch batch;
  for (int i = 0; i < n_probs; ++i) batch.p[i] = probs[i];
  batch.n_probs = n_probs;
  if (!a_t && !b_t) return dispatch_epi<false, false>(dtype, epi, batch, stream);
  if (!a_t && b_t) return dispatch_epi<false, true>(dtype, epi, batch, stream);
  if (a_t && !b_t) return dispatch_epi<true, false>(dtype, epi, batch, stream);
  return dispatch_epi<true, true>(dtype, epi, batch, stream);
}

}  // namespace merak

extern "C" int merak_gemm_tile_override(int cfg) {
  if (cfg < merak::TILE_AUTO || cfg >= merak::TILE_COUNT) return -1;
  return merak::g_tile_override.exchange(cfg);
}
