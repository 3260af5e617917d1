// Stage runtime and C ABI (include/merak_stage.h).
//
// Host-side schedule of one GPU's share of a pipeline stage:
//   * forward: for each block, the micro-batch's n sub-micro-batches (even,
//     independent splits along the batch axis, paper Sec. 5.3) are issued on
//     stream (j mod 2), so one slice's GEMMs can run beside another slice's
//     LayerNorm/attention work;
//   * blocks whose recompute bit is set keep only their input (paper Sec. 5.2);
//     merak_stage_recompute rebuilds their activations from it and needs no
//     upstream gradient (early recomputation, Sec. 5.1);
//   * backward: per block, the sub-micro-batches' input-gradient chains run on
//     the two streams; the block's weight, bias and LayerNorm gradients are
//     then formed over the whole micro-batch on an internal third stream
//     (parity-double-buffered scratch lets the next block's chains proceed
//     meanwhile).  No floating-point atomics: results are deterministic.
// The AllReduces of tensor parallelism are the identity on one GPU; their
// inputs (partial sums) go to the caller's hand-off buffers.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <map>
#include <mutex>
#include <new>
#include <vector>

#include "merak_stage.h"
#include "kernels.h"

using namespace merak;

namespace {

constexpr int kMaxBlocks = 64;
constexpr int kMaxTimed = 4096;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Dims {
  int L, h, a, f, s, b, t, n;
  int hl, fl, al, d;
  int T, Ms, bs;  // tokens per micro-batch, tokens and samples per sub-micro-batch
  int dtype;
  size_t esz;
  uint64_t mask;
  float eps;
};

int check_config(const merak_stage_config* c) {
  if (!c) return MERAK_ERR_INVALID_ARG;
  if (c->dtype != MERAK_BF16 && c->dtype != MERAK_FP32) return MERAK_ERR_INVALID_ARG;
  if (c->n_blocks < 1 || c->n_blocks > kMaxBlocks) return MERAK_ERR_SHAPE;
  if (c->hidden <= 0 || c->n_heads <= 0 || c->ffn <= 0 || c->seq_len <= 0 || c->micro_batch <= 0 ||
      c->tp_degree <= 0 || c->n_sub_microbatches <= 0)
    return MERAK_ERR_SHAPE;
  if (c->n_heads % c->tp_degree != 0 || c->hidden % c->n_heads != 0 || c->ffn % c->tp_degree != 0 ||
      c->micro_batch % c->n_sub_microbatches != 0)
    return MERAK_ERR_SHAPE;
  if (c->hidden % 64 != 0 || (c->hidden / c->tp_degree) % 64 != 0 || (c->ffn / c->tp_degree) % 64 != 0 ||
      c->seq_len % 64 != 0)
    return MERAK_ERR_SHAPE;
  if (c->n_blocks < 64 && (c->recompute_mask >> c->n_blocks) != 0) return MERAK_ERR_SHAPE;
  if (!(c->ln_eps > 0.0f)) return MERAK_ERR_SHAPE;
  // Sizes must fit the 32-bit indexing of the launch interface.
  const int64_t T = (int64_t)c->micro_batch * c->seq_len;
  if (T * (int64_t)c->ffn / c->tp_degree >= ((int64_t)1 << 31) || T * (int64_t)c->hidden * 3 >= ((int64_t)1 << 31))
    return MERAK_ERR_SHAPE;
  // The bf16 GEMM addresses each [T, width] activation operand with 32-bit
  // byte offsets, 256 rows of edge-tile padding included (the weight-gradient
  // GEMMs read the whole micro-batch as one operand).
  if (c->dtype == MERAK_BF16) {
    const int64_t hl = c->hidden / c->tp_degree, fl = c->ffn / c->tp_degree;
    const int64_t w = std::max<int64_t>(std::max<int64_t>(c->hidden, fl), 3 * hl);
    if (2 * ((T + 256) * w + w) >= ((int64_t)1 << 31)) return MERAK_ERR_SHAPE;
  }
  const int d = c->hidden / c->n_heads;
  if (d != 64 && d != 96 && d != 128) return MERAK_ERR_UNSUPPORTED;
  return MERAK_OK;
}

Dims make_dims(const merak_stage_config* c) {
  Dims D;
  D.L = c->n_blocks; D.h = c->hidden; D.a = c->n_heads; D.f = c->ffn; D.s = c->seq_len; D.b = c->micro_batch;
  D.t = c->tp_degree; D.n = c->n_sub_microbatches;
  D.hl = D.h / D.t; D.fl = D.f / D.t; D.al = D.a / D.t; D.d = D.h / D.a;
  D.T = D.b * D.s; D.bs = D.b / D.n; D.Ms = D.bs * D.s;
  D.dtype = c->dtype;
  D.esz = c->dtype == MERAK_BF16 ? 2 : 4;
  D.mask = c->recompute_mask;
  D.eps = c->ln_eps;
  return D;
}

// Element offsets of the 12 tensors of one block, and the block stride.
void block_param_offsets(const Dims& D, size_t off[MERAK_PARAMS_PER_BLOCK], size_t* stride) {
  const size_t sizes[MERAK_PARAMS_PER_BLOCK] = {
      (size_t)D.h, (size_t)D.h, (size_t)3 * D.hl * D.h, (size_t)3 * D.hl, (size_t)D.h * D.hl, (size_t)D.h,
      (size_t)D.h, (size_t)D.h, (size_t)D.fl * D.h, (size_t)D.fl, (size_t)D.h * D.fl, (size_t)D.h};
  size_t o = 0;
  for (int i = 0; i < MERAK_PARAMS_PER_BLOCK; ++i) {
    off[i] = o;
    o = align_up(o + sizes[i], 64);
  }
  *stride = o;
}

enum { P_LN1G, P_LN1B, P_WQKV, P_BQKV, P_WO, P_BO, P_LN2G, P_LN2B, P_W1, P_B1, P_W2, P_B2 };

// Byte offsets of one block's saved activations.
struct ActLayout {
  size_t ln1, mu1, rs1, qkv, o, lse, x1, ln2, mu2, rs2, u, g, size;
};

ActLayout act_layout(const Dims& D) {
  ActLayout A;
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
  const size_t T = D.T, e = D.esz;
  A.ln1 = take(T * D.h * e);
  A.mu1 = take(T * 4);
  A.rs1 = take(T * 4);
  A.qkv = take(T * 3 * D.hl * e);
  A.o = take(T * D.hl * e);
  A.lse = take(T * D.al * 4);
  A.x1 = take(T * D.h * e);
  A.ln2 = take(T * D.h * e);
  A.mu2 = take(T * 4);
  A.rs2 = take(T * 4);
  A.u = take(T * D.fl * e);
  A.g = take(T * D.fl * e);
  A.size = o;
  return A;
}

// Backward scratch of one parity.
struct BwdLayout {
  size_t du, dln2, dx1, dO, dqkv, dln1, delta;
  size_t p_bqkv, p_bo, p_b1, p_b2, p_g2, p_be2, p_g1, p_be1;
  size_t size;
};

BwdLayout bwd_layout(const Dims& D) {
  BwdLayout B;
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
  const size_t T = D.T, e = D.esz, G = reduce_groups(D.T);
  B.du = take(T * D.fl * e);
  B.dln2 = take(T * D.h * e);
  B.dx1 = take(T * D.h * e);
  B.dO = take(T * D.hl * e);
  B.dqkv = take(T * 3 * D.hl * e);
  B.dln1 = take(T * D.h * e);
  B.delta = take(T * D.al * 4);
  B.p_bqkv = take(G * 3 * D.hl * 4);
  B.p_bo = take(G * D.h * 4);
  B.p_b1 = take(G * D.fl * 4);
  B.p_b2 = take(G * D.h * 4);
  B.p_g2 = take(G * D.h * 4);
  B.p_be2 = take(G * D.h * 4);
  B.p_g1 = take(G * D.h * 4);
  B.p_be1 = take(G * D.h * 4);
  B.size = o;
  return B;
}

struct WsLayout {
  ActLayout act;
  BwdLayout bwd;
  size_t xs;          // (L-1) block-input checkpoints
  size_t keep_acts;   // activations of non-recomputed blocks
  size_t fwd_tmp;     // activations of recomputed blocks during the forward pass
  size_t chain;       // 3 input-gradient buffers
  size_t par[2];      // backward scratch per parity
  size_t total;
  size_t recompute_total;
  int keep_slot[kMaxBlocks];  // index among kept blocks, or -1
  int rc_slot[kMaxBlocks];    // index among recomputed blocks, or -1
  int n_keep, n_rc;
};

WsLayout ws_layout(const Dims& D) {
  WsLayout W;
  W.act = act_layout(D);
  W.bwd = bwd_layout(D);
  W.n_keep = W.n_rc = 0;
  for (int l = 0; l < D.L; ++l) {
    const bool rc = (D.mask >> l) & 1;
    W.keep_slot[l] = rc ? -1 : W.n_keep++;
    W.rc_slot[l] = rc ? W.n_rc++ : -1;
  }
  const size_t th = align_up((size_t)D.T * D.h * D.esz, 256);
  size_t o = 0;
  W.xs = o; o += (size_t)(D.L - 1) * th;
  W.keep_acts = o; o += (size_t)W.n_keep * W.act.size;
  W.fwd_tmp = o; o += (W.n_rc > 0 ? W.act.size : 0);
  W.chain = o; o += 3 * th;
  W.par[0] = o; o += W.bwd.size;
  W.par[1] = o; o += W.bwd.size;
  W.total = o;
  W.recompute_total = (size_t)W.n_rc * W.act.size;
  return W;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

}  // namespace

// ---------------------------------------------------------------------------
// Handle
// ---------------------------------------------------------------------------
struct merak_stage {
  merak_stage_config cfg;
  Dims D;
  WsLayout W;
  size_t p_off[MERAK_PARAMS_PER_BLOCK];
  size_t p_stride;
  char* ws;
  char* rc;
  hipStream_t aux;
  hipEvent_t ev_fork, ev_s1, ev_j0, ev_j1, ev_aux, ev_dw[2];
  hipEvent_t ev_rc[kMaxBlocks][2];  // recompute of block l done on its two streams
  int state;  // 0 idle, 1 forward pending, 2 recomputed
  const void* x0;
  // optional per-launch event timing of one kernel class
  int timed_class;
  std::vector<hipEvent_t> t_ev;  // 2 * kMaxTimed events, created on first use
  int t_count;
  bool t_overflow;
};

namespace {

enum { ST_IDLE = 0, ST_FWD = 1, ST_RECOMPUTED = 2 };

std::mutex g_mu;
std::map<void*, merak_stage*> g_rc_owner;  // recompute area -> handle that last filled it

char* block_input(merak_stage* S, int l) {
  if (l == 0) return (char*)S->x0;
  return S->ws + S->W.xs + (size_t)(l - 1) * align_up((size_t)S->D.T * S->D.h * S->D.esz, 256);
}

// Saved activations of block l: during the forward pass (phase 0) recomputed
// blocks use the temporary set; after recompute (phase 1) they use their slot
// in the recompute area.
char* block_acts(merak_stage* S, int l, int phase) {
  if (S->W.keep_slot[l] >= 0) return S->ws + S->W.keep_acts + (size_t)S->W.keep_slot[l] * S->W.act.size;
  if (phase == 0) return S->ws + S->W.fwd_tmp;
  return S->rc + (size_t)S->W.rc_slot[l] * S->W.act.size;
}

#define HIP_TRY(expr)                          \
  do {                                         \
    hipError_t e_ = (expr);                    \
    if (e_ != hipSuccess) return MERAK_ERR_HIP; \
  } while (0)

// Run `launch` (returns hipError_t); if its kernel class is being timed, record
// a start/stop event pair around it on `st`.
// Launches left before an injected failure (< 0: none); merak_debug_fail_after.
std::atomic<int> g_fail_countdown{-1};

bool injected_failure() {
  int n = g_fail_countdown.load(std::memory_order_relaxed);
  while (n >= 0) {
    if (g_fail_countdown.compare_exchange_weak(n, n - 1, std::memory_order_relaxed)) return n == 0;
  }
  return false;
}

template <typename F>
int timed(merak_stage* S, int cls, hipStream_t st, F&& launch) {
  if (injected_failure()) return MERAK_ERR_HIP;  // as if the launch had failed
  const bool on = (S->timed_class == cls && cls != MERAK_KC_NONE);
  if (on && S->t_count >= kMaxTimed) S->t_overflow = true;
  const bool rec = on && S->t_count < kMaxTimed;
  if (rec) HIP_TRY(hipEventRecord(S->t_ev[2 * S->t_count], st));
  HIP_TRY(launch());
  if (rec) {
    HIP_TRY(hipEventRecord(S->t_ev[2 * S->t_count + 1], st));
    ++S->t_count;
  }
  return MERAK_OK;
}

#define LAUNCH(cls, st, expr) TRY_INNER(timed(S, (cls), (st), [&]() { return (expr); }))
#define TRY_INNER(expr)            \
  do {                             \
    int r2_ = (expr);              \
    if (r2_ != MERAK_OK) return r2_; \
  } while (0)

inline const char* P(const void* params, const merak_stage* S, int l, int which) {
  return (const char*)params + (S->p_stride * l + S->p_off[which]) * S->D.esz;
}

GemmProblem gp(int M, int N, int K, const void* a, int lda, const void* b, int ldb, void* c, int ldc,
               const void* bias = nullptr, const void* resid = nullptr, void* aux = nullptr, int acc = 0) {
  GemmProblem p;
  p.M = M; p.N = N; p.K = K; p.a = a; p.lda = lda; p.b = b; p.ldb = ldb; p.c = c; p.ldc = ldc;
  p.bias = bias; p.resid = resid; p.aux = aux; p.accumulate = acc;
  return p;
}

// Step k (0..6) of the forward of block l for sub-micro-batch j:
//   0 LN1  1 QKV GEMM  2 attention  3 projection GEMM  4 LN2  5 FC1 GEMM
//   6 FC2 GEMM.
// GEMM steps only describe their problem (*p, *epi) for a grouped launch; the
// other steps are launched on st, each covering `members` sub-micro-batches
// j, j + 2, ... in one launch.
constexpr int kFwdSteps = 7;
inline bool fwd_step_is_gemm(int k) { return k == 1 || k == 3 || k == 5 || k == 6; }
int block_forward_step(merak_stage* S, const void* params, int l, int j, int k, char* A, const char* x, char* y,
                       char* part_o, char* part_f, hipStream_t st, GemmProblem* p, int* epi, int members) {
  const Dims& D = S->D;
  const ActLayout& L = S->W.act;
  const int dt = D.dtype;
  const size_t r0 = (size_t)j * D.Ms;
  const size_t e = D.esz;
  const int M = D.Ms;
  switch (k) {
    case 0:  // LN1
      LAUNCH(MERAK_KC_LN_FWD, st, launch_layernorm_fwd(dt, M, D.h, D.eps, x + r0 * D.h * e, P(params, S, l, P_LN1G),
                                   P(params, S, l, P_LN1B), A + L.ln1 + r0 * D.h * e, (float*)(A + L.mu1) + r0,
                                   (float*)(A + L.rs1) + r0, st, members, 2 * M));
      break;
    case 1:  // QKV (column parallel) + bias
      *p = gp(M, 3 * D.hl, D.h, A + L.ln1 + r0 * D.h * e, D.h, P(params, S, l, P_WQKV), D.h,
              A + L.qkv + r0 * 3 * D.hl * e, 3 * D.hl, P(params, S, l, P_BQKV));
      *epi = EPI_BIAS;
      break;
    case 2:  // causal attention on the local heads
      LAUNCH(MERAK_KC_ATTN_FWD, st, launch_attention_fwd(dt, D.bs, D.s, D.al, D.d, A + L.qkv + r0 * 3 * D.hl * e,
                                     A + L.o + r0 * D.hl * e,
                                     (float*)(A + L.lse) + (size_t)j * D.bs * D.al * D.s, st, members,
                                     2 * D.bs));
      break;
    case 3:  // projection (row parallel): partial sum -> hand-off; x1 = x + partial + b_o
      *p = gp(M, D.h, D.hl, A + L.o + r0 * D.hl * e, D.hl, P(params, S, l, P_WO), D.hl, A + L.x1 + r0 * D.h * e, D.h,
              P(params, S, l, P_BO), x + r0 * D.h * e, part_o ? part_o + r0 * D.h * e : nullptr);
      *epi = EPI_BIAS_RESID;
      break;
    case 4:  // LN2
      LAUNCH(MERAK_KC_LN_FWD, st, launch_layernorm_fwd(dt, M, D.h, D.eps, A + L.x1 + r0 * D.h * e,
                                   P(params, S, l, P_LN2G), P(params, S, l, P_LN2B), A + L.ln2 + r0 * D.h * e,
                                   (float*)(A + L.mu2) + r0, (float*)(A + L.rs2) + r0, st, members, 2 * M));
      break;
    case 5: {  // FC1 (column parallel) + bias + GeLU; keeps the pre-activation u for
               // the GeLU backward, except in the forward of a recomputed block,
               // whose activations (in the shared temporary area) the
               // recomputation rebuilds
      const bool drop_u = ((D.mask >> l) & 1) && A == S->ws + S->W.fwd_tmp;
      *p = gp(M, D.fl, D.h, A + L.ln2 + r0 * D.h * e, D.h, P(params, S, l, P_W1), D.h, A + L.g + r0 * D.fl * e, D.fl,
              P(params, S, l, P_B1), nullptr, drop_u ? nullptr : A + L.u + r0 * D.fl * e);
      *epi = EPI_BIAS_GELU;
      break;
    }
    default:  // FC2 (row parallel): partial sum -> hand-off; y = x1 + partial + b2
      *p = gp(M, D.h, D.fl, A + L.g + r0 * D.fl * e, D.fl, P(params, S, l, P_W2), D.fl, y + r0 * D.h * e, D.h,
              P(params, S, l, P_B2), A + L.x1 + r0 * D.h * e, part_f ? part_f + r0 * D.h * e : nullptr);
      *epi = EPI_BIAS_RESID;
      break;
  }
  return MERAK_OK;
}

// Forward of block l over all sub-micro-batches: sub-micro-batch j runs on
// stream j mod 2, issued step by step; the GEMMs of one step of the
// sub-micro-batches that share a stream go out as one grouped launch (they are
// independent problems of the same shape, so each keeps its own result).
// With y == nullptr (recomputation) the FC2 step is left out: its output is
// the next block's input, which is already checkpointed, and the backward
// needs only FC2's input g.
int block_forward(merak_stage* S, const void* params, int l, char* A, const char* x, char* y, char* part_o,
                  char* part_f, hipStream_t s0, hipStream_t s1) {
  const Dims& D = S->D;
  for (int k = 0; k < (y ? kFwdSteps : kFwdSteps - 1); ++k) {
    for (int par = 0; par < 2; ++par) {
      hipStream_t st = par ? s1 : s0;
      GemmProblem probs[kMaxGroup];
      int np = 0, epi = EPI_STORE;
      const int members = (D.n - par + 1) / 2;  // sub-micro-batches on this stream
      for (int j = par; j < D.n; j += 2) {
        if (!fwd_step_is_gemm(k) && j != par) break;  // one LN / attention launch covers them all
        TRY_INNER(block_forward_step(S, params, l, j, k, A, x, y, part_o, part_f, st, &probs[np], &epi, members));
        if (fwd_step_is_gemm(k) && (++np == kMaxGroup || j + 2 >= D.n)) {
          LAUNCH(MERAK_KC_GEMM_FWD, st, launch_gemm(D.dtype, false, false, epi, probs, np, st));
          np = 0;
        }
      }
    }
  }
  return MERAK_OK;
}

// Step k (0..6) of the input-gradient chain of block l for sub-micro-batch j:
//   0 FC2 dX (+GeLU')  1 FC1 dX  2 LN2 bwd  3 proj dX  4 attention bwd
//   5 QKV dX  6 LN1 bwd.
// GEMM steps only describe their problem for a grouped launch; the LayerNorm
// and attention steps cover `members` sub-micro-batches j, j + 2, ... in one
// launch.
constexpr int kChainSteps = 7;
inline bool bwd_step_is_gemm(int k) { return k == 0 || k == 1 || k == 3 || k == 5; }
int block_backward_step(merak_stage* S, const void* params, int l, int j, int k, const char* A, const char* x,
                        const char* dy, char* dx, char* B, char* d_ln1, char* d_ln2, hipStream_t st, GemmProblem* gpr,
                        int* epi, int members) {
  const Dims& D = S->D;
  const ActLayout& L = S->W.act;
  const BwdLayout& Bl = S->W.bwd;
  const int dt = D.dtype;
  const size_t r0 = (size_t)j * D.Ms;
  const size_t e = D.esz;
  const int M = D.Ms;
  switch (k) {
    case 0:  // FC2 backward: dg = dy W2; du = dg * gelu'(u)
      *gpr = gp(M, D.fl, D.h, dy + r0 * D.h * e, D.h, P(params, S, l, P_W2), D.fl, B + Bl.du + r0 * D.fl * e, D.fl, nullptr,
                nullptr, (void*)(A + L.u + r0 * D.fl * e));
      *epi = EPI_GELU_BWD;
      break;
    case 1:  // FC1 backward: d_ln2 partial = du W1 (hand-off)
      *gpr = gp(M, D.h, D.fl, B + Bl.du + r0 * D.fl * e, D.fl, P(params, S, l, P_W1), D.h, d_ln2 + r0 * D.h * e, D.h);
      *epi = EPI_STORE;
      break;
    case 2:  // LN2 backward + residual gradient: dx1 = dy + LN2'(d_ln2)
      LAUNCH(MERAK_KC_LN_BWD, st, launch_layernorm_bwd(dt, M, D.h, d_ln2 + r0 * D.h * e, A + L.x1 + r0 * D.h * e,
                                 (const float*)(A + L.mu2) + r0, (const float*)(A + L.rs2) + r0,
                                 P(params, S, l, P_LN2G), dy + r0 * D.h * e, B + Bl.dx1 + r0 * D.h * e, st,
                                 members, 2 * M));
      break;
    case 3:  // projection backward: dO = dx1 W_o
      *gpr = gp(M, D.hl, D.h, B + Bl.dx1 + r0 * D.h * e, D.h, P(params, S, l, P_WO), D.hl, B + Bl.dO + r0 * D.hl * e, D.hl);
      *epi = EPI_STORE;
      break;
    case 4: {  // attention backward -> dqkv
      const size_t lse_off = (size_t)j * D.bs * D.al * D.s;
      LAUNCH(MERAK_KC_ATTN_BWD, st, launch_attention_bwd(dt, D.bs, D.s, D.al, D.d, A + L.qkv + r0 * 3 * D.hl * e,
                                   A + L.o + r0 * D.hl * e, (const float*)(A + L.lse) + lse_off,
                                   B + Bl.dO + r0 * D.hl * e, B + Bl.dqkv + r0 * 3 * D.hl * e,
                                   (float*)(B + Bl.delta) + lse_off, st, members, 2 * D.bs));
      break;
    }
    case 5:  // QKV backward: d_ln1 partial = dqkv W_qkv (hand-off)
      *gpr = gp(M, D.h, 3 * D.hl, B + Bl.dqkv + r0 * 3 * D.hl * e, 3 * D.hl, P(params, S, l, P_WQKV), D.h,
                d_ln1 + r0 * D.h * e, D.h);
      *epi = EPI_STORE;
      break;
    default:  // LN1 backward + residual gradient: dx = dx1 + LN1'(d_ln1)
      LAUNCH(MERAK_KC_LN_BWD, st, launch_layernorm_bwd(dt, M, D.h, d_ln1 + r0 * D.h * e, x + r0 * D.h * e,
                                 (const float*)(A + L.mu1) + r0, (const float*)(A + L.rs1) + r0,
                                 P(params, S, l, P_LN1G), B + Bl.dx1 + r0 * D.h * e, dx + r0 * D.h * e, st,
                                 members, 2 * M));
      break;
  }
  return MERAK_OK;
}

// Weight, bias and LayerNorm gradients of block l over the whole micro-batch,
// on stream st, in four parts that can start as soon as the chain has made
// their inputs: part 0 (dW2, dW1, db2, db1) needs dy and du, i.e. the FC2
// backward of every sub-micro-batch; part 1 (dW_o, dW_qkv) and part 2 (b_o,
// b_qkv and LayerNorm 2's sums) need dx1, d_ln2 and dqkv, i.e. the attention
// backward; part 3 (LayerNorm 1's sums) needs d_ln1, made by the QKV
// backward.  Parts 2 and 3 of the first block, the last the backward
// reaches, run on the caller's streams after its chains, beside part 1's
// GEMM on the internal stream.
int block_param_grads(merak_stage* S, int l, int group, const char* A, const char* x, const char* dy, const char* B,
                      const char* d_ln1, const char* d_ln2, float* grads, int acc, hipStream_t st) {
  const Dims& D = S->D;
  const ActLayout& L = S->W.act;
  const BwdLayout& Bl = S->W.bwd;
  const int dt = D.dtype;
  const int T = D.T;
  const int G = (int)reduce_groups(T);
  float* g = grads + S->p_stride * l;
  auto part = [&](size_t off) { return (float*)(B + off); };
  if (group == 0) {
    // dW = dY^T X for FC2 and FC1, one grouped launch
    GemmProblem p[2];
    p[0] = gp(D.h, D.fl, T, dy, D.h, A + L.g, D.fl, g + S->p_off[P_W2], D.fl, nullptr, nullptr, nullptr, acc);
    p[1] = gp(D.fl, D.h, T, B + Bl.du, D.fl, A + L.ln2, D.h, g + S->p_off[P_W1], D.h, nullptr, nullptr, nullptr, acc);
    LAUNCH(MERAK_KC_GEMM_DW, st, launch_gemm(dt, true, true, EPI_F32, p, 2, st));
    // bias gradients: token sums of the layer output gradients (one launch
    // for the partials, one for the final sums)
    const ColPartialJob cj[2] = {{0, T, D.h, dy, nullptr, nullptr, nullptr, part(Bl.p_b2), nullptr},
                                 {0, T, D.fl, B + Bl.du, nullptr, nullptr, nullptr, part(Bl.p_b1), nullptr}};
    LAUNCH(MERAK_KC_REDUCE, st, launch_column_partials_batch(dt, cj, 2, st));
    const ReduceJob rj[2] = {{G, D.h, part(Bl.p_b2), g + S->p_off[P_B2], acc},
                             {G, D.fl, part(Bl.p_b1), g + S->p_off[P_B1], acc}};
    LAUNCH(MERAK_KC_REDUCE, st, launch_reduce_partials_batch(rj, 2, st));
    return MERAK_OK;
  }
  if (group == 1) {
    GemmProblem p[2];
    p[0] = gp(3 * D.hl, D.h, T, B + Bl.dqkv, 3 * D.hl, A + L.ln1, D.h, g + S->p_off[P_WQKV], D.h, nullptr, nullptr,
              nullptr, acc);
    p[1] = gp(D.h, D.hl, T, B + Bl.dx1, D.h, A + L.o, D.hl, g + S->p_off[P_WO], D.hl, nullptr, nullptr, nullptr, acc);
    LAUNCH(MERAK_KC_GEMM_DW_ATTN, st, launch_gemm(dt, true, true, EPI_F32, p, 2, st));
    return MERAK_OK;
  }
  if (group == 2) {  // QKV and projection biases, LayerNorm 2's parameters
    const ColPartialJob cj[3] = {
        {0, T, 3 * D.hl, B + Bl.dqkv, nullptr, nullptr, nullptr, part(Bl.p_bqkv), nullptr},
        {0, T, D.h, B + Bl.dx1, nullptr, nullptr, nullptr, part(Bl.p_bo), nullptr},
        {1, T, D.h, d_ln2, A + L.x1, (const float*)(A + L.mu2), (const float*)(A + L.rs2), part(Bl.p_g2),
         part(Bl.p_be2)}};
    LAUNCH(MERAK_KC_REDUCE, st, launch_column_partials_batch(dt, cj, 3, st));
    const ReduceJob rj[4] = {{G, 3 * D.hl, part(Bl.p_bqkv), g + S->p_off[P_BQKV], acc},
                             {G, D.h, part(Bl.p_bo), g + S->p_off[P_BO], acc},
                             {G, D.h, part(Bl.p_g2), g + S->p_off[P_LN2G], acc},
                             {G, D.h, part(Bl.p_be2), g + S->p_off[P_LN2B], acc}};
    LAUNCH(MERAK_KC_REDUCE, st, launch_reduce_partials_batch(rj, 4, st));
    return MERAK_OK;
  }
  // LayerNorm 1's parameters
  const ColPartialJob cj[1] = {
      {1, T, D.h, d_ln1, x, (const float*)(A + L.mu1), (const float*)(A + L.rs1), part(Bl.p_g1), part(Bl.p_be1)}};
  LAUNCH(MERAK_KC_REDUCE, st, launch_column_partials_batch(dt, cj, 1, st));
  const ReduceJob rj[2] = {{G, D.h, part(Bl.p_g1), g + S->p_off[P_LN1G], acc},
                           {G, D.h, part(Bl.p_be1), g + S->p_off[P_LN1B], acc}};
  LAUNCH(MERAK_KC_REDUCE, st, launch_reduce_partials_batch(rj, 2, st));
  return MERAK_OK;
}

int fork(merak_stage* S, hipStream_t s0, hipStream_t s1) {
  HIP_TRY(hipEventRecord(S->ev_fork, s0));
  HIP_TRY(hipStreamWaitEvent(s1, S->ev_fork, 0));
  return MERAK_OK;
}

int join(merak_stage* S, hipStream_t s0, hipStream_t s1) {
  HIP_TRY(hipEventRecord(S->ev_s1, s1));
  HIP_TRY(hipStreamWaitEvent(s0, S->ev_s1, 0));
  return MERAK_OK;
}

int check_ptr(const void* p) {
  if (!p) return MERAK_ERR_INVALID_ARG;
  if (!aligned(p, 16)) return MERAK_ERR_ALIGN;
  return MERAK_OK;
}

#define TRY(expr)               \
  do {                          \
    int r_ = (expr);            \
    if (r_ != MERAK_OK) return r_; \
  } while (0)

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

const char* merak_status_str(int status) {
  switch (status) {
    case MERAK_OK: return "ok";
    case MERAK_ERR_INVALID_ARG: return "invalid argument";
    case MERAK_ERR_SHAPE: return "unsupported or inconsistent shape";
    case MERAK_ERR_ORDER: return "call-order violation";
    case MERAK_ERR_ALIGN: return "misaligned pointer";
    case MERAK_ERR_WORKSPACE: return "workspace too small";
    case MERAK_ERR_HIP: return "HIP runtime error";
    case MERAK_ERR_UNSUPPORTED: return "unsupported configuration";
    default: return "unknown status";
  }
}

int merak_stage_validate(const merak_stage_config* cfg) { return check_config(cfg); }

int merak_stage_param_layout(const merak_stage_config* cfg, size_t* total_elems, size_t* offsets) {
  TRY(check_config(cfg));
  if (!total_elems) return MERAK_ERR_INVALID_ARG;
  const Dims D = make_dims(cfg);
  size_t off[MERAK_PARAMS_PER_BLOCK], stride;
  block_param_offsets(D, off, &stride);
  *total_elems = stride * D.L;
  if (offsets)
    for (int l = 0; l < D.L; ++l)
      for (int i = 0; i < MERAK_PARAMS_PER_BLOCK; ++i) offsets[l * MERAK_PARAMS_PER_BLOCK + i] = stride * l + off[i];
  return MERAK_OK;
}

int merak_stage_workspace_bytes(const merak_stage_config* cfg, size_t* workspace_bytes, size_t* recompute_bytes) {
  TRY(check_config(cfg));
  const WsLayout W = ws_layout(make_dims(cfg));
  if (workspace_bytes) *workspace_bytes = W.total;
  if (recompute_bytes) *recompute_bytes = W.recompute_total;
  return MERAK_OK;
}

int merak_stage_create(const merak_stage_config* cfg, void* workspace, size_t workspace_bytes, void* recompute_area,
                       size_t recompute_bytes, merak_stage_t* out) {
  if (!out) return MERAK_ERR_INVALID_ARG;
  *out = nullptr;
  TRY(check_config(cfg));
  const Dims D = make_dims(cfg);
  const WsLayout W = ws_layout(D);
  if (!workspace) return MERAK_ERR_INVALID_ARG;
  if (!aligned(workspace, 256)) return MERAK_ERR_ALIGN;
  if (workspace_bytes < W.total) return MERAK_ERR_WORKSPACE;
  if (W.recompute_total > 0) {
    if (!recompute_area) return MERAK_ERR_INVALID_ARG;
    if (!aligned(recompute_area, 256)) return MERAK_ERR_ALIGN;
    if (recompute_bytes < W.recompute_total) return MERAK_ERR_WORKSPACE;
  }
  merak_stage* S = new (std::nothrow) merak_stage();
  if (!S) return MERAK_ERR_INVALID_ARG;
  S->cfg = *cfg;
  S->D = D;
  S->W = W;
  block_param_offsets(D, S->p_off, &S->p_stride);
  S->ws = (char*)workspace;
  S->rc = (char*)recompute_area;
  S->state = ST_IDLE;
  S->x0 = nullptr;
  S->timed_class = MERAK_KC_NONE;
  S->t_count = 0;
  S->t_overflow = false;
  hipError_t e = hipStreamCreateWithFlags(&S->aux, hipStreamNonBlocking);
  const bool have_stream = (e == hipSuccess);
  hipEvent_t* evs[] = {&S->ev_fork, &S->ev_s1, &S->ev_j0, &S->ev_j1, &S->ev_aux, &S->ev_dw[0], &S->ev_dw[1]};
  int made = 0;
  for (hipEvent_t* ev : evs) {
    if (e != hipSuccess) break;
    e = hipEventCreateWithFlags(ev, hipEventDisableTiming);
    if (e == hipSuccess) ++made;
  }
  int made_rc = 0;
  for (int l = 0; l < D.L && e == hipSuccess; ++l) {
    e = hipEventCreateWithFlags(&S->ev_rc[l][0], hipEventDisableTiming);
    if (e != hipSuccess) break;
    e = hipEventCreateWithFlags(&S->ev_rc[l][1], hipEventDisableTiming);
    if (e != hipSuccess) {
      (void)hipEventDestroy(S->ev_rc[l][0]);
      break;
    }
    ++made_rc;
  }
  if (e != hipSuccess) {
    for (int i = 0; i < made; ++i) (void)hipEventDestroy(*evs[i]);
    for (int l = 0; l < made_rc; ++l) {
      (void)hipEventDestroy(S->ev_rc[l][0]);
      (void)hipEventDestroy(S->ev_rc[l][1]);
    }
    if (have_stream) (void)hipStreamDestroy(S->aux);
    delete S;
    return MERAK_ERR_HIP;
  }
  *out = S;
  return MERAK_OK;
}

int merak_stage_destroy(merak_stage_t S) {
  if (!S) return MERAK_ERR_INVALID_ARG;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    for (auto it = g_rc_owner.begin(); it != g_rc_owner.end();)
      it = (it->second == S) ? g_rc_owner.erase(it) : std::next(it);
  }
  hipEvent_t evs[] = {S->ev_fork, S->ev_s1, S->ev_j0, S->ev_j1, S->ev_aux, S->ev_dw[0], S->ev_dw[1]};
  for (hipEvent_t ev : evs) (void)hipEventDestroy(ev);
  for (int l = 0; l < S->D.L; ++l) {
    (void)hipEventDestroy(S->ev_rc[l][0]);
    (void)hipEventDestroy(S->ev_rc[l][1]);
  }
  for (hipEvent_t ev : S->t_ev) (void)hipEventDestroy(ev);
  (void)hipStreamDestroy(S->aux);
  delete S;
  return MERAK_OK;
}

int merak_debug_fail_after(int launches) {
  return g_fail_countdown.exchange(launches < 0 ? -1 : launches);
}

int merak_stage_set_timing(merak_stage_t S, int kernel_class) {
  if (!S) return MERAK_ERR_INVALID_ARG;
  if (kernel_class < MERAK_KC_NONE || kernel_class >= MERAK_KC_COUNT) return MERAK_ERR_INVALID_ARG;
  if (kernel_class != MERAK_KC_NONE && S->t_ev.empty()) {
    S->t_ev.resize(2 * kMaxTimed);
    for (size_t i = 0; i < S->t_ev.size(); ++i) {
      if (hipEventCreate(&S->t_ev[i]) != hipSuccess) {
        for (size_t k = 0; k < i; ++k) (void)hipEventDestroy(S->t_ev[k]);
        S->t_ev.clear();
        return MERAK_ERR_HIP;
      }
    }
  }
  S->timed_class = kernel_class;
  S->t_count = 0;
  S->t_overflow = false;
  return MERAK_OK;
}

int merak_stage_read_timing(merak_stage_t S, double* total_ms, int64_t* launches) {
  if (!S || !total_ms || !launches) return MERAK_ERR_INVALID_ARG;
  if (S->t_overflow) return MERAK_ERR_ORDER;
  double sum = 0.0;
  for (int i = 0; i < S->t_count; ++i) {
    float ms = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, S->t_ev[2 * i], S->t_ev[2 * i + 1]));
    sum += ms;
  }
  *total_ms = sum;
  *launches = S->t_count;
  S->t_count = 0;
  return MERAK_OK;
}

int merak_stage_fwd(merak_stage_t S, const void* params, const void* x, void* y, void* fwd_partials, void* stream0,
                    void* stream1) {
  if (!S) return MERAK_ERR_INVALID_ARG;
  TRY(check_ptr(params));
  TRY(check_ptr(x));
  TRY(check_ptr(y));
  if (fwd_partials && !aligned(fwd_partials, 16)) return MERAK_ERR_ALIGN;
  hipStream_t s0 = (hipStream_t)stream0, s1 = (hipStream_t)stream1;
  const Dims& D = S->D;
  // Idle until every launch of the pass has been enqueued: a failure part-way
  // leaves a handle that refuses recompute and bwd.
  S->state = ST_IDLE;
  S->x0 = x;
  TRY(fork(S, s0, s1));
  const size_t th = (size_t)D.T * D.h * D.esz;
  for (int l = 0; l < D.L; ++l) {
    char* A = block_acts(S, l, 0);
    const char* xin = block_input(S, l);
    char* yout = (l == D.L - 1) ? (char*)y : block_input(S, l + 1);
    char* po = fwd_partials ? (char*)fwd_partials + (size_t)(2 * l) * th : nullptr;
    char* pf = fwd_partials ? (char*)fwd_partials + (size_t)(2 * l + 1) * th : nullptr;
    TRY(block_forward(S, params, l, A, xin, yout, po, pf, s0, s1));
  }
  TRY(join(S, s0, s1));
  S->state = ST_FWD;
  return MERAK_OK;
}

int merak_stage_recompute(merak_stage_t S, const void* params, void* stream0, void* stream1) {
  if (!S) return MERAK_ERR_INVALID_ARG;
  TRY(check_ptr(params));
  if (S->state == ST_IDLE) return MERAK_ERR_ORDER;
  if (S->D.mask == 0) return MERAK_OK;
  hipStream_t s0 = (hipStream_t)stream0, s1 = (hipStream_t)stream1;
  const Dims& D = S->D;
  // The area is this handle's from the first launch on: a handle that filled
  // it before can no longer run its backward on it, and if a launch fails
  // part-way neither can this one (its state stays short of RECOMPUTED).
  {
    std::lock_guard<std::mutex> lk(g_mu);
    g_rc_owner[S->rc] = S;
  }
  S->state = ST_FWD;
  TRY(fork(S, s0, s1));
  for (int l = 0; l < D.L; ++l) {
    if (!((D.mask >> l) & 1)) continue;
    char* A = block_acts(S, l, 1);
    const char* xin = block_input(S, l);
    TRY(block_forward(S, params, l, A, xin, nullptr, nullptr, nullptr, s0, s1));  // everything but FC2
    // the backward of block l waits for these (it may run on other streams)
    HIP_TRY(hipEventRecord(S->ev_rc[l][0], s0));
    HIP_TRY(hipEventRecord(S->ev_rc[l][1], s1));
  }
  TRY(join(S, s0, s1));
  S->state = ST_RECOMPUTED;
  return MERAK_OK;
}

int merak_stage_bwd(merak_stage_t S, const void* params, const void* dy, void* dx, float* grads, int accumulate,
                    void* bwd_partials, void* stream0, void* stream1) {
  if (!S) return MERAK_ERR_INVALID_ARG;
  TRY(check_ptr(params));
  TRY(check_ptr(dy));
  TRY(check_ptr(dx));
  TRY(check_ptr(grads));
  if (accumulate != 0 && accumulate != 1) return MERAK_ERR_INVALID_ARG;
  if (bwd_partials && !aligned(bwd_partials, 16)) return MERAK_ERR_ALIGN;
  if (S->state == ST_IDLE) return MERAK_ERR_ORDER;
  if (S->D.mask != 0) {
    if (S->state != ST_RECOMPUTED) return MERAK_ERR_ORDER;
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_rc_owner.find(S->rc);
    if (it == g_rc_owner.end() || it->second != S) return MERAK_ERR_ORDER;
  }
  hipStream_t s0 = (hipStream_t)stream0, s1 = (hipStream_t)stream1;
  const Dims& D = S->D;
  const size_t th = (size_t)D.T * D.h * D.esz;
  const size_t th_al = align_up(th, 256);
  S->state = ST_IDLE;  // consumed, also if a launch fails part-way
  TRY(fork(S, s0, s1));
  HIP_TRY(hipStreamWaitEvent(S->aux, S->ev_fork, 0));
  for (int l = D.L - 1; l >= 0; --l) {
    const int par = l & 1;
    char* A = block_acts(S, l, 1);
    const char* xin = block_input(S, l);
    const char* dyl = (l == D.L - 1) ? (const char*)dy : S->ws + S->W.chain + (size_t)((l + 1) % 3) * th_al;
    char* dxl = (l == 0) ? (char*)dx : S->ws + S->W.chain + (size_t)(l % 3) * th_al;
    char* B = S->ws + S->W.par[par];
    char* d1 = bwd_partials ? (char*)bwd_partials + (size_t)(2 * l) * th : B + S->W.bwd.dln1;
    char* d2 = bwd_partials ? (char*)bwd_partials + (size_t)(2 * l + 1) * th : B + S->W.bwd.dln2;
    if (l <= D.L - 3) {  // parity scratch was last read by the gradients of block l+2
      HIP_TRY(hipStreamWaitEvent(s0, S->ev_dw[par], 0));
      HIP_TRY(hipStreamWaitEvent(s1, S->ev_dw[par], 0));
    }
    if ((D.mask >> l) & 1) {  // the activations recomputed for this block
      for (int q = 0; q < 2; ++q) {
        HIP_TRY(hipStreamWaitEvent(s0, S->ev_rc[l][q], 0));
        HIP_TRY(hipStreamWaitEvent(s1, S->ev_rc[l][q], 0));
        HIP_TRY(hipStreamWaitEvent(S->aux, S->ev_rc[l][q], 0));
      }
    }
    // Chains issued step by step over the sub-micro-batches (sub-micro-batch j
    // on stream j mod 2), so that the FFN weight gradients can start on the
    // internal stream once every FC2 backward is done.  The GEMMs of one step
    // of the sub-micro-batches that share a stream form one grouped launch.
    for (int k = 0; k < kChainSteps; ++k) {
      for (int sp = 0; sp < 2; ++sp) {
        hipStream_t st = sp ? s1 : s0;
        GemmProblem probs[kMaxGroup];
        int np = 0, epi = EPI_STORE;
        const int members = (D.n - sp + 1) / 2;  // sub-micro-batches on this stream
        for (int j = sp; j < D.n; j += 2) {
          if (!bwd_step_is_gemm(k) && j != sp) break;  // one LN / attention launch covers them all
          TRY(block_backward_step(S, params, l, j, k, A, xin, dyl, dxl, B, d1, d2, st, &probs[np], &epi, members));
          if (bwd_step_is_gemm(k) && (++np == kMaxGroup || j + 2 >= D.n)) {
            LAUNCH(MERAK_KC_GEMM_DX, st, launch_gemm(D.dtype, false, true, epi, probs, np, st));
            np = 0;
          }
        }
      }
      // Parameter gradients on the internal stream once every sub-micro-
      // batch has passed the step that makes their inputs.  The first block
      // (the last one here) leaves its sums (parts 2 and 3) to the caller's
      // streams after its chain, where they run beside the internal stream's
      // last weight-gradient GEMM instead of after it.
      const int part = k == 0 ? 0 : k == 4 ? 1 : (k == 5 && l > 0) ? 3 : -1;
      if (part >= 0) {
        HIP_TRY(hipEventRecord(S->ev_j0, s0));
        HIP_TRY(hipEventRecord(S->ev_j1, s1));
        HIP_TRY(hipStreamWaitEvent(S->aux, S->ev_j0, 0));
        HIP_TRY(hipStreamWaitEvent(S->aux, S->ev_j1, 0));
        TRY(block_param_grads(S, l, part, A, xin, dyl, B, d1, d2, grads, accumulate, S->aux));
        if (part == 1 && l > 0) TRY(block_param_grads(S, l, 2, A, xin, dyl, B, d1, d2, grads, accumulate, S->aux));
      }
    }
    if (l == 0) {
      HIP_TRY(hipEventRecord(S->ev_j0, s0));
      HIP_TRY(hipEventRecord(S->ev_j1, s1));
      HIP_TRY(hipStreamWaitEvent(s0, S->ev_j1, 0));
      HIP_TRY(hipStreamWaitEvent(s1, S->ev_j0, 0));
      TRY(block_param_grads(S, l, 2, A, xin, dyl, B, d1, d2, grads, accumulate, s1));
      TRY(block_param_grads(S, l, 3, A, xin, dyl, B, d1, d2, grads, accumulate, s0));
    }
    HIP_TRY(hipEventRecord(S->ev_dw[par], S->aux));
  }
  HIP_TRY(hipEventRecord(S->ev_aux, S->aux));
  TRY(join(S, s0, s1));
  HIP_TRY(hipStreamWaitEvent(s0, S->ev_aux, 0));
  return MERAK_OK;
}

// ---------------------------------------------------------------------------
// Stage-aware recomputation planner (host only)
// ---------------------------------------------------------------------------
namespace {

// Share of kept blocks of stage i (1-based) of s; `prev` is the share of stage
// i - 1 (used by the penultimate stage).
double plan_share(int s, int i, double alpha1, double prev) {
  if (i == s) return 1.0;
  if (i == 1) return alpha1;
  if (i == s - 1) return prev;
  const double a = (double)(s - 1) * alpha1 / (double)(s - i);
  return a < 1.0 ? a : 1.0;
}

bool plan_fits(int s, double a1, double mr, double ma, double cap) {
  double prev = 0.0;
  for (int i = 1; i <= s; ++i) {
    const double a = plan_share(s, i, a1, prev);
    if (mr + (double)(s - i) * a * ma > cap) return false;
    prev = a;
  }
  return true;
}

}  // namespace

int merak_plan_recompute(int n_stages, double alpha1, int blocks_per_stage, double* alpha, uint64_t* masks) {
  if (n_stages < 1 || n_stages > 4096 || !(alpha1 >= 0.0 && alpha1 <= 1.0) || !alpha || !masks)
    return MERAK_ERR_INVALID_ARG;
  if (blocks_per_stage < 1 || blocks_per_stage > 64) return MERAK_ERR_SHAPE;
  double prev = 0.0;
  for (int i = 1; i <= n_stages; ++i) {
    const double a = plan_share(n_stages, i, alpha1, prev);
    int keep = (int)std::floor(a * blocks_per_stage + 1e-12);
    keep = keep < 0 ? 0 : (keep > blocks_per_stage ? blocks_per_stage : keep);
    const int n_rc = blocks_per_stage - keep;
    alpha[i - 1] = a;
    masks[i - 1] = n_rc >= 64 ? ~(uint64_t)0 : (((uint64_t)1 << n_rc) - 1);
    prev = a;
  }
  return MERAK_OK;
}

int merak_plan_alpha1(int n_stages, double mem_runtime, double mem_activation, double capacity, double step,
                      double* alpha1) {
  if (n_stages < 1 || n_stages > 4096 || !alpha1 || !(step > 0.0) || !(mem_activation >= 0.0))
    return MERAK_ERR_INVALID_ARG;
  if (!plan_fits(n_stages, 0.0, mem_runtime, mem_activation, capacity)) return MERAK_ERR_UNSUPPORTED;
  double best = 0.0;
  for (long k = 1; (double)k * step <= 1.0 + 1e-12; ++k) {
    const double a1 = (double)k * step < 1.0 ? (double)k * step : 1.0;
    if (!plan_fits(n_stages, a1, mem_runtime, mem_activation, capacity)) break;
    best = a1;
  }
  *alpha1 = best;
  return MERAK_OK;
}

// ---------------------------------------------------------------------------
// Pipeline schedules (host only)
// ---------------------------------------------------------------------------
namespace {

inline int32_t sched_op(int type, int mb) { return (int32_t)(((uint32_t)type << 24) | (uint32_t)mb); }

// Op list of one stage (see the header for the three orders).
void build_stage_ops(int kind, int s, int m, int i, std::vector<int32_t>& ops) {
  ops.clear();
  if (kind == MERAK_SCHED_SCP && i == s - 1) {  // the last stage keeps its activation
    for (int j = 0; j < m; ++j) {
      ops.push_back(sched_op(MERAK_OP_FWD, j));
      ops.push_back(sched_op(MERAK_OP_BWD, j));
    }
    return;
  }
  if (kind == MERAK_SCHED_SCP && i == s - 2 && m >= 2) {  // one forward brought ahead
    ops.push_back(sched_op(MERAK_OP_FWD, 0));
    ops.push_back(sched_op(MERAK_OP_FWD, 1));
    ops.push_back(sched_op(MERAK_OP_RECOMPUTE, 0));
    int nf = 2;
    if (nf < m) ops.push_back(sched_op(MERAK_OP_FWD, nf++));
    ops.push_back(sched_op(MERAK_OP_BWD, 0));
    for (int j = 1; j < m; ++j) {
      ops.push_back(sched_op(MERAK_OP_RECOMPUTE, j));
      ops.push_back(sched_op(MERAK_OP_BWD, j));
      if (nf < m) ops.push_back(sched_op(MERAK_OP_FWD, nf++));
    }
    return;
  }
  const int warm = std::min(s - 1 - i, m);
  int nf = 0;
  for (; nf < warm; ++nf) ops.push_back(sched_op(MERAK_OP_FWD, nf));
  for (int j = 0; j < m; ++j) {
    if (nf < m) ops.push_back(sched_op(MERAK_OP_FWD, nf++));
    if (kind == MERAK_SCHED_1F1B) {
      ops.push_back(sched_op(MERAK_OP_RECOMPUTE_BWD, j));
    } else {
      ops.push_back(sched_op(MERAK_OP_RECOMPUTE, j));
      ops.push_back(sched_op(MERAK_OP_BWD, j));
    }
  }
}

int check_sched(int kind, int s, int m) {
  if (kind < MERAK_SCHED_1F1B || kind > MERAK_SCHED_SCP) return MERAK_ERR_INVALID_ARG;
  if (s < 1 || s > 1024 || m < 1 || m >= (1 << 24)) return MERAK_ERR_SHAPE;
  return MERAK_OK;
}

}  // namespace

int merak_schedule_stage(int kind, int n_stages, int n_micro, int stage, int32_t* ops, int capacity, int* n_ops) {
  TRY(check_sched(kind, n_stages, n_micro));
  if (stage < 0 || stage >= n_stages || !n_ops || capacity < 0 || (capacity > 0 && !ops)) return MERAK_ERR_INVALID_ARG;
  std::vector<int32_t> v;
  build_stage_ops(kind, n_stages, n_micro, stage, v);
  *n_ops = (int)v.size();
  if ((int)v.size() > capacity) return MERAK_ERR_WORKSPACE;
  std::copy(v.begin(), v.end(), ops);
  return MERAK_OK;
}

int merak_schedule_simulate(int kind, int n_stages, int n_micro, double cost_fwd, double cost_rc, double cost_bwd,
                            double* makespan, double* busy) {
  TRY(check_sched(kind, n_stages, n_micro));
  const int s = n_stages, m = n_micro;
  if ((int64_t)s * m > ((int64_t)1 << 22)) return MERAK_ERR_SHAPE;
  if (!makespan || !busy || !(cost_fwd >= 0.0) || !(cost_rc >= 0.0) || !(cost_bwd >= 0.0)) return MERAK_ERR_INVALID_ARG;
  std::vector<std::vector<int32_t>> plan(s);
  for (int i = 0; i < s; ++i) build_stage_ops(kind, s, m, i, plan[i]);
  // finish times per (stage, micro-batch); < 0 = not yet run
  std::vector<double> fF((size_t)s * m, -1.0), fR((size_t)s * m, -1.0), fB((size_t)s * m, -1.0);
  std::vector<char> hasR((size_t)s * m, 0);
  for (int i = 0; i < s; ++i)
    for (int32_t op : plan[i])
      if ((op >> 24) == MERAK_OP_RECOMPUTE) hasR[(size_t)i * m + (op & 0xffffff)] = 1;
  std::vector<double> free_at(s, 0.0), work(s, 0.0);
  std::vector<size_t> pos(s, 0);
  size_t left = 0;
  for (auto& p : plan) left += p.size();
  while (left) {
    bool moved = false;
    for (int i = 0; i < s; ++i) {
      if (pos[i] == plan[i].size()) continue;
      const int type = plan[i][pos[i]] >> 24, j = plan[i][pos[i]] & 0xffffff;
      const size_t at = (size_t)i * m + j;
      double ready = free_at[i];
      bool ok = true;
      if (type == MERAK_OP_FWD && i > 0) {
        const double f = fF[(size_t)(i - 1) * m + j];
        ok = ok && f >= 0.0;
        ready = std::max(ready, f);
      }
      if (type == MERAK_OP_BWD || type == MERAK_OP_RECOMPUTE_BWD) {
        if (i < s - 1) {
          const double f = fB[(size_t)(i + 1) * m + j];
          ok = ok && f >= 0.0;
          ready = std::max(ready, f);
        }
        if (type == MERAK_OP_BWD && hasR[at]) {
          ok = ok && fR[at] >= 0.0;
          ready = std::max(ready, fR[at]);
        }
      }
      if (!ok) continue;
      const double cost = type == MERAK_OP_FWD ? cost_fwd
                          : type == MERAK_OP_RECOMPUTE ? cost_rc
                          : type == MERAK_OP_BWD ? cost_bwd : cost_rc + cost_bwd;
      free_at[i] = ready + cost;
      work[i] += cost;
      (type == MERAK_OP_FWD ? fF : type == MERAK_OP_RECOMPUTE ? fR : fB)[at] = free_at[i];
      ++pos[i];
      --left;
      moved = true;
    }
    if (!moved) return MERAK_ERR_ORDER;  // cannot happen for the built-in orders
  }
  *makespan = *std::max_element(free_at.begin(), free_at.end());
  for (int i = 0; i < s; ++i) busy[i] = work[i];
  return MERAK_OK;
}

// ---------------------------------------------------------------------------
// Running one stage's schedule on this GPU
// ---------------------------------------------------------------------------
int merak_schedule_inflight(int kind, int n_stages, int n_micro, int stage, int* max_inflight) {
  TRY(check_sched(kind, n_stages, n_micro));
  if (stage < 0 || stage >= n_stages || !max_inflight) return MERAK_ERR_INVALID_ARG;
  std::vector<int32_t> v;
  build_stage_ops(kind, n_stages, n_micro, stage, v);
  int live = 0, most = 0;
  for (int32_t op : v) {
    const int type = op >> 24;
    if (type == MERAK_OP_FWD) most = std::max(most, ++live);
    if (type == MERAK_OP_BWD || type == MERAK_OP_RECOMPUTE_BWD) --live;
  }
  *max_inflight = most;
  return MERAK_OK;
}

int merak_schedule_run(int kind, int n_stages, int n_micro, int stage, merak_stage_t* handles, int n_handles,
                       const void* params, const void* const* x, void* const* y, const void* const* dy,
                       void* const* dx, float* grads, int accumulate, void* stream0, void* stream1) {
  TRY(check_sched(kind, n_stages, n_micro));
  if (stage < 0 || stage >= n_stages || !handles || n_handles < 1 || !x || !y || !dy || !dx)
    return MERAK_ERR_INVALID_ARG;
  if (accumulate != 0 && accumulate != 1) return MERAK_ERR_INVALID_ARG;
  TRY(check_ptr(params));
  TRY(check_ptr(grads));
  for (int i = 0; i < n_handles; ++i) {
    if (!handles[i]) return MERAK_ERR_INVALID_ARG;
    for (int k = 0; k < i; ++k)
      if (handles[k] == handles[i]) return MERAK_ERR_INVALID_ARG;
    if (memcmp(&handles[i]->cfg, &handles[0]->cfg, sizeof(merak_stage_config)) != 0) return MERAK_ERR_SHAPE;
  }
  for (int j = 0; j < n_micro; ++j) {
    TRY(check_ptr(x[j]));
    TRY(check_ptr(y[j]));
    TRY(check_ptr(dy[j]));
    TRY(check_ptr(dx[j]));
  }
  int need = 0;
  TRY(merak_schedule_inflight(kind, n_stages, n_micro, stage, &need));
  if (n_handles < need) return MERAK_ERR_WORKSPACE;
  std::vector<int32_t> ops;
  build_stage_ops(kind, n_stages, n_micro, stage, ops);
  // One handle per micro-batch in flight: taken at its forward, returned after
  // its backward.  Every call goes to the same two streams in op order, so the
  // gradients accumulate in backward order (micro-batch 0 first).
  std::vector<int> free_list, owner(n_micro, -1);
  for (int i = n_handles - 1; i >= 0; --i) free_list.push_back(i);
  int acc = accumulate;
  for (int32_t op : ops) {
    const int type = op >> 24, j = op & 0xffffff;
    if (type == MERAK_OP_FWD) {
      if (free_list.empty()) return MERAK_ERR_WORKSPACE;  // cannot happen after the count above
      owner[j] = free_list.back();
      free_list.pop_back();
      TRY(merak_stage_fwd(handles[owner[j]], params, x[j], y[j], nullptr, stream0, stream1));
      continue;
    }
    if (owner[j] < 0) return MERAK_ERR_ORDER;
    merak_stage_t h = handles[owner[j]];
    if (type == MERAK_OP_RECOMPUTE || type == MERAK_OP_RECOMPUTE_BWD) TRY(merak_stage_recompute(h, params, stream0, stream1));
    if (type == MERAK_OP_BWD || type == MERAK_OP_RECOMPUTE_BWD) {
      TRY(merak_stage_bwd(h, params, dy[j], dx[j], grads, acc, nullptr, stream0, stream1));
      acc = 1;
      free_list.push_back(owner[j]);
      owner[j] = -1;
    }
  }
  return MERAK_OK;
}

// ---------------------------------------------------------------------------
// Per-kernel entry points
// ---------------------------------------------------------------------------
int merak_gemm(int dtype, int a_trans, int b_trans, int epilogue, int M, int N, int K, const void* a, int lda,
               const void* b, int ldb, void* c, const void* bias, const void* resid, void* aux, int accumulate,
               void* stream) {
  if (dtype != MERAK_BF16 && dtype != MERAK_FP32) return MERAK_ERR_INVALID_ARG;
  if ((a_trans != 0 && a_trans != 1) || (b_trans != 0 && b_trans != 1)) return MERAK_ERR_INVALID_ARG;
  if (epilogue < 0 || epilogue >= EPI_COUNT) return MERAK_ERR_INVALID_ARG;
  if (M <= 0 || N <= 0 || K <= 0 || M % 64 || N % 64 || K % 64) return MERAK_ERR_SHAPE;
  if (lda < (a_trans ? M : K) || ldb < (b_trans ? N : K) || lda % 8 || ldb % 8) return MERAK_ERR_SHAPE;
  TRY(check_ptr(a));
  TRY(check_ptr(b));
  TRY(check_ptr(c));
  const bool need_bias = epilogue == EPI_BIAS || epilogue == EPI_BIAS_GELU || epilogue == EPI_BIAS_RESID;
  if (need_bias) TRY(check_ptr(bias));
  if (epilogue == EPI_BIAS_RESID) TRY(check_ptr(resid));
  if (epilogue == EPI_BIAS_GELU || epilogue == EPI_GELU_BWD) TRY(check_ptr(aux));
  if (aux && !aligned(aux, 16)) return MERAK_ERR_ALIGN;
  if (accumulate != 0 && accumulate != 1) return MERAK_ERR_INVALID_ARG;
  GemmProblem p = gp(M, N, K, a, lda, b, ldb, c, N, bias, resid, aux, accumulate);
  if (dtype == MERAK_BF16 && !gemm_bf16_offsets_fit(p, a_trans, b_trans)) return MERAK_ERR_SHAPE;
  HIP_TRY(launch_gemm(dtype, a_trans, b_trans, epilogue, &p, 1, (hipStream_t)stream));
  return MERAK_OK;
}

int merak_layernorm_fwd(int dtype, int rows, int h, float eps, const void* x, const void* gamma, const void* beta,
                        void* y, float* mean, float* rstd, void* stream) {
  if (dtype != MERAK_BF16 && dtype != MERAK_FP32) return MERAK_ERR_INVALID_ARG;
  if (rows <= 0 || h <= 0 || h % 8 || h > 8192 || !(eps > 0.0f)) return MERAK_ERR_SHAPE;
  TRY(check_ptr(x)); TRY(check_ptr(gamma)); TRY(check_ptr(beta)); TRY(check_ptr(y));
  TRY(check_ptr(mean)); TRY(check_ptr(rstd));
  HIP_TRY(launch_layernorm_fwd(dtype, rows, h, eps, x, gamma, beta, y, mean, rstd, (hipStream_t)stream));
  return MERAK_OK;
}

size_t merak_reduce_scratch_elems(int rows, int cols) {
  if (rows <= 0 || cols <= 0) return 0;
  return reduce_groups(rows) * (size_t)cols;
}

int merak_layernorm_bwd(int dtype, int rows, int h, const void* dout, const void* x, const float* mean,
                        const float* rstd, const void* gamma, const void* dres, void* dx, float* dgamma,
                        float* dbeta, int accumulate, float* scratch, void* stream) {
  if (dtype != MERAK_BF16 && dtype != MERAK_FP32) return MERAK_ERR_INVALID_ARG;
  if (rows <= 0 || h <= 0 || h % 8 || h > 8192) return MERAK_ERR_SHAPE;
  if (accumulate != 0 && accumulate != 1) return MERAK_ERR_INVALID_ARG;
  TRY(check_ptr(dout)); TRY(check_ptr(x)); TRY(check_ptr(mean)); TRY(check_ptr(rstd)); TRY(check_ptr(gamma));
  TRY(check_ptr(dres)); TRY(check_ptr(dx)); TRY(check_ptr(dgamma)); TRY(check_ptr(dbeta)); TRY(check_ptr(scratch));
  hipStream_t st = (hipStream_t)stream;
  const size_t n = merak_reduce_scratch_elems(rows, h);
  const int G = (int)reduce_groups(rows);
  HIP_TRY(launch_layernorm_bwd(dtype, rows, h, dout, x, mean, rstd, gamma, dres, dx, st));
  HIP_TRY(launch_layernorm_param_partials(dtype, rows, h, dout, x, mean, rstd, scratch, scratch + n, st));
  HIP_TRY(launch_reduce_partials(G, h, scratch, dgamma, accumulate, st));
  HIP_TRY(launch_reduce_partials(G, h, scratch + n, dbeta, accumulate, st));
  return MERAK_OK;
}

int merak_layernorm_bwd_noalloc(int dtype, int rows, int h, const void* dout, const void* x, const float* mean,
                                const float* rstd, const void* gamma, const void* dres, void* dx, float* dgamma,
                                float* dbeta, int accumulate, void* stream) {
  if (dtype != MERAK_BF16 && dtype != MERAK_FP32) return MERAK_ERR_INVALID_ARG;
  if (rows <= 0 || h <= 0 || h % 8 || h > 8192) return MERAK_ERR_SHAPE;
  if (accumulate != 0 && accumulate != 1) return MERAK_ERR_INVALID_ARG;
  TRY(check_ptr(dout)); TRY(check_ptr(x)); TRY(check_ptr(mean)); TRY(check_ptr(rstd)); TRY(check_ptr(gamma));
  TRY(check_ptr(dres)); TRY(check_ptr(dx)); TRY(check_ptr(dgamma)); TRY(check_ptr(dbeta));
  const size_t n = merak_reduce_scratch_elems(rows, h);
  if (2 * n > kNoAllocScratchFloats) return MERAK_ERR_WORKSPACE;
  float* scratch = nullptr;  // the library's array on the current device
  HIP_TRY(noalloc_scratch(&scratch));
  hipStream_t st = (hipStream_t)stream;
  const int G = (int)reduce_groups(rows);
  // Same kernels and order as merak_layernorm_bwd; the partial-sum kernel
  // writes every scratch element the reduction then reads.
  HIP_TRY(launch_layernorm_bwd(dtype, rows, h, dout, x, mean, rstd, gamma, dres, dx, st));
  HIP_TRY(launch_layernorm_param_partials(dtype, rows, h, dout, x, mean, rstd, scratch, scratch + n, st));
  HIP_TRY(launch_reduce_partials(G, h, scratch, dgamma, accumulate, st));
  HIP_TRY(launch_reduce_partials(G, h, scratch + n, dbeta, accumulate, st));
  return MERAK_OK;
}

size_t merak_noalloc_scratch_elems(void) { return kNoAllocScratchFloats; }

int merak_column_sum(int dtype, int rows, int cols, const void* x, float* out, int accumulate, float* scratch,
                     void* stream) {
  if (dtype != MERAK_BF16 && dtype != MERAK_FP32) return MERAK_ERR_INVALID_ARG;
  if (rows <= 0 || cols <= 0 || cols % 8) return MERAK_ERR_SHAPE;
  if (accumulate != 0 && accumulate != 1) return MERAK_ERR_INVALID_ARG;
  TRY(check_ptr(x)); TRY(check_ptr(out)); TRY(check_ptr(scratch));
  hipStream_t st = (hipStream_t)stream;
  HIP_TRY(launch_column_partials(dtype, rows, cols, x, scratch, st));
  HIP_TRY(launch_reduce_partials((int)reduce_groups(rows), cols, scratch, out, accumulate, st));
  return MERAK_OK;
}

int merak_count_nonfinite(int dtype, const void* x, int64_t n, uint64_t* count, void* stream) {
  if (dtype != MERAK_BF16 && dtype != MERAK_FP32) return MERAK_ERR_INVALID_ARG;
  if (n < 0) return MERAK_ERR_SHAPE;
  TRY(check_ptr(count));
  if (n > 0) TRY(check_ptr(x));
  HIP_TRY(launch_count_nonfinite(dtype, x, (long long)n, (unsigned long long*)count, (hipStream_t)stream));
  return MERAK_OK;
}

int merak_attention_fwd(int dtype, int batch, int seq, int heads, int head_dim, const void* qkv, void* o, float* lse,
                        void* stream) {
  if (dtype != MERAK_BF16 && dtype != MERAK_FP32) return MERAK_ERR_INVALID_ARG;
  if (batch <= 0 || heads <= 0 || seq <= 0 || seq % 64) return MERAK_ERR_SHAPE;
  if (head_dim != 64 && head_dim != 96 && head_dim != 128) return MERAK_ERR_UNSUPPORTED;
  TRY(check_ptr(qkv)); TRY(check_ptr(o)); TRY(check_ptr(lse));
  HIP_TRY(launch_attention_fwd(dtype, batch, seq, heads, head_dim, qkv, o, lse, (hipStream_t)stream));
  return MERAK_OK;
}

int merak_attention_bwd(int dtype, int batch, int seq, int heads, int head_dim, const void* qkv, const void* o,
                        const float* lse, const void* dout, void* dqkv, float* delta, void* stream) {
  if (dtype != MERAK_BF16 && dtype != MERAK_FP32) return MERAK_ERR_INVALID_ARG;
  if (batch <= 0 || heads <= 0 || seq <= 0 || seq % 64) return MERAK_ERR_SHAPE;
  if (head_dim != 64 && head_dim != 96 && head_dim != 128) return MERAK_ERR_UNSUPPORTED;
  TRY(check_ptr(qkv)); TRY(check_ptr(o)); TRY(check_ptr(lse)); TRY(check_ptr(dout)); TRY(check_ptr(dqkv));
  TRY(check_ptr(delta));
  HIP_TRY(launch_attention_bwd(dtype, batch, seq, heads, head_dim, qkv, o, lse, dout, dqkv, delta,
                               (hipStream_t)stream));
  return MERAK_OK;
}

}  // extern "C"
