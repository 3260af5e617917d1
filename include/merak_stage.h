/*
 * merak_stage.h: C ABI of the MI355X (gfx950) stage-shard library.
 *
 * One GPU's share of a GPT pipeline stage: L consecutive transformer blocks
 * (a pipeline stage is a contiguous run of blocks, paper Sec. 2 "Pipeline
 * model parallelism" and Sec. 4.2), each cut Megatron-style into a
 * tensor-model-parallel shard (Sec. 2 "Tensor model parallelism"; Sec. 4.1):
 * column-parallel QKV and FC1, causal attention on the shard's heads,
 * row-parallel projection and FC2.  A block has two AllReduces in the forward
 * pass and two in the backward pass (Sec. 5.3).  On one GPU each AllReduce is
 * the identity; the value this shard would contribute to it (its partial sum)
 * is written to a caller-supplied hand-off buffer.
 *
 * The method's two schedule features are carried by the kernels' schedule:
 *   - sub-pipelined TMP (Sec. 5.3): each micro-batch is split evenly along the
 *     batch axis into n independent sub-micro-batches that run on two HIP
 *     streams, so one slice's GEMMs overlap another slice's other work;
 *   - stage-aware recomputation (Sec. 5.2): a per-block mask selects blocks
 *     that keep only their input; their activations are rebuilt by
 *     merak_stage_recompute, which needs no upstream gradient and may run
 *     early, before the gradient arrives (Sec. 5.1, early recomputation).
 *
 * Block math (pre-LN GPT block; internals are not fixed by the paper):
 *   ln1 = LN1(x);  qkv = ln1 W_qkv^T + b_qkv  ([q|k|v] x local heads x d)
 *   O   = softmax(q k^T / sqrt(d), causal) v;  p_o = O W_o^T   (partial)
 *   x1  = x + R(p_o) + b_o;  ln2 = LN2(x1);  u = ln2 W1^T + b1;  g = GeLU_tanh(u)
 *   p_f = g W2^T (partial);  y = x1 + R(p_f) + b2;  R = identity on one GPU.
 * LayerNorm: biased variance, eps inside the square root, fp32 statistics.
 *
 * Conventions for every entry point
 *   - Return value: MERAK_OK (0) or a negative merak_status.  Argument, shape,
 *     alignment, workspace and call-order errors are detected on the host
 *     before anything is enqueued; such a call has no side effects.
 *   - Device pointers are caller-owned (allocated by the caller, for example
 *     as torch tensors); the library never allocates device memory.  Every
 *     device pointer must be 16-byte aligned; workspaces 256-byte aligned.
 *   - Streams are hipStream_t values passed as void* (NULL = the null
 *     stream); stream0 and stream1 may be equal.  Calls enqueue work and
 *     return; all work of a call is ordered after prior work on stream0 and
 *     stream1, and its completion is recorded on stream0 (stream0 waits for
 *     stream1 before the call returns).  Kernel faults surface at the
 *     caller's next synchronisation, as usual in HIP.
 *   - Element types: MERAK_BF16 = bf16 activations/weights with fp32
 *     accumulation; MERAK_FP32 = the fp32 check mode (every tensor fp32).
 *     Weight gradients are always fp32.
 *   - Layouts are row-major.  Activations are [micro_batch, seq_len, features].
 *     Weights are stored [out, in]: a linear layer computes X W^T + b.
 */
#ifndef MERAK_STAGE_H
#define MERAK_STAGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MERAK_OK = 0,
  MERAK_ERR_INVALID_ARG = -1, /* NULL handle/pointer, bad enum, bad flag        */
  MERAK_ERR_SHAPE = -2,       /* dimensions violate the constraints below       */
  MERAK_ERR_ORDER = -3,       /* call-order violation (see merak_stage_bwd)     */
  MERAK_ERR_ALIGN = -4,       /* device pointer not 16-byte (256 for workspaces)*/
  MERAK_ERR_WORKSPACE = -5,   /* workspace smaller than the size query returned */
  MERAK_ERR_HIP = -6,         /* a HIP runtime call failed                      */
  MERAK_ERR_UNSUPPORTED = -7  /* valid but not implemented (e.g. head_dim)     */
} merak_status;

typedef enum { MERAK_BF16 = 0, MERAK_FP32 = 1 } merak_dtype;

/* Number of parameter tensors per block, in flat-buffer order:
 *   0 ln1_g[h]   1 ln1_b[h]   2 w_qkv[3h/t, h]   3 b_qkv[3h/t]
 *   4 w_o[h, h/t]             5 b_o[h]
 *   6 ln2_g[h]   7 ln2_b[h]   8 w1[f/t, h]       9 b1[f/t]
 *  10 w2[h, f/t]             11 b2[h]
 * The shard map (which rows/columns of the full model a rank owns) is
 * Megatron's: rank r owns heads [r a/t, (r+1) a/t) -- its w_qkv rows are its
 * q rows, then its k rows, then its v rows -- and FFN units [r f/t, (r+1) f/t).
 * LayerNorm parameters, b_o and b2 are replicated; a row-parallel bias is
 * added once, after the reduction. */
#define MERAK_PARAMS_PER_BLOCK 12

/* Stage configuration.  Dimensions are those of the full (t = 1) model.
 * Constraints (else MERAK_ERR_SHAPE): 1 <= n_blocks <= 64; n_heads % tp_degree
 * == 0; hidden % n_heads == 0; ffn % tp_degree == 0; micro_batch %
 * n_sub_microbatches == 0; hidden, hidden/tp_degree, ffn/tp_degree and
 * seq_len multiples of 64; recompute_mask has no bit >= n_blocks; ln_eps > 0;
 * micro_batch*seq_len times ffn/tp_degree and times 3*hidden below 2^31; in
 * MERAK_BF16, (micro_batch*seq_len + 256) * max(hidden, 3*hidden/tp_degree,
 * ffn/tp_degree) * 2 bytes below 2^31 (the GEMM's 32-bit operand offsets).
 * head_dim = hidden/n_heads must be 64, 96 or 128 (else MERAK_ERR_UNSUPPORTED). */
typedef struct {
  int32_t n_blocks;           /* L: blocks in the stage                               */
  int32_t hidden;             /* h                                                    */
  int32_t n_heads;            /* a (global)                                           */
  int32_t ffn;                /* f (global)                                           */
  int32_t seq_len;            /* s                                                    */
  int32_t micro_batch;        /* b                                                    */
  int32_t tp_degree;          /* t: local heads a/t, local FFN width f/t              */
  int32_t n_sub_microbatches; /* n: even split of the micro-batch (Sec. 5.3)          */
  uint64_t recompute_mask;    /* bit l: block l keeps only its input (Sec. 5.2)       */
  int32_t dtype;              /* merak_dtype                                          */
  float ln_eps;               /* LayerNorm epsilon (1e-5)                             */
} merak_stage_config;

typedef struct merak_stage* merak_stage_t;

/* Human-readable name of a status code (static string). */
const char* merak_status_str(int status);

/* Host-only check of a configuration; no GPU needed. */
int merak_stage_validate(const merak_stage_config* cfg);

/* Parameter layout of one rank's stage shard.  *total_elems receives the element
 * count of the flat parameter buffer (elements of the config's dtype) and of the
 * fp32 gradient buffer (same layout).  If offsets is not NULL it receives
 * n_blocks * MERAK_PARAMS_PER_BLOCK element offsets, block-major, in the order
 * listed above.  Every offset is a multiple of 64 elements.  Host-only. */
int merak_stage_param_layout(const merak_stage_config* cfg, size_t* total_elems, size_t* offsets);

/* Device memory a handle needs (host-only query).
 *   *workspace_bytes: per-handle memory (activations kept for the backward pass
 *      of the blocks that are not recomputed, inputs of recomputed blocks, and
 *      backward scratch);
 *   *recompute_bytes: activations of the recomputed blocks (0 when the mask is
 *      0).  Handles that never have a recompute->bwd window open at the same
 *      time may share one recompute area.
 * Either output pointer may be NULL. */
int merak_stage_workspace_bytes(const merak_stage_config* cfg, size_t* workspace_bytes,
                                size_t* recompute_bytes);

/* Create a handle bound to a configuration and caller-owned device memory.
 * The workspace must hold at least *workspace_bytes and stays owned by the
 * caller; it must not be freed before merak_stage_destroy.  recompute_area may
 * be NULL when recompute_bytes is 0.  Needs the GPU (creates HIP events on the
 * current device).  On success *out receives the handle. */
int merak_stage_create(const merak_stage_config* cfg, void* workspace, size_t workspace_bytes,
                       void* recompute_area, size_t recompute_bytes, merak_stage_t* out);

/* Destroy a handle (waits for nothing; the caller synchronises first). */
int merak_stage_destroy(merak_stage_t stage);

/* Forward pass of the stage for one micro-batch.
 *   params        [total_elems] (dtype): the shard's parameters, layout above.
 *   x             [b, s, h] (dtype): stage input.  It is read again by
 *                 merak_stage_recompute and merak_stage_bwd, so it must stay
 *                 unchanged until that backward work has completed.
 *   y             [b, s, h] (dtype): stage output.
 *   fwd_partials  NULL or [L][2][b, s, h] (dtype): hand-off buffers; [l][0] is
 *                 block l's projection partial p_o, [l][1] its FC2 partial p_f
 *                 (the inputs the two forward AllReduces would reduce).
 * Sub-micro-batch j (samples [j b/n, (j+1) b/n)) runs on stream (j mod 2).
 * Starts a new micro-batch: earlier activations of this handle are dropped. */
int merak_stage_fwd(merak_stage_t stage, const void* params, const void* x, void* y,
                    void* fwd_partials, void* stream0, void* stream1);

/* Rebuild the activations of every block whose recompute bit is set, from the
 * block inputs kept by merak_stage_fwd, into the recompute area: the block's
 * forward up to FC2's input (FC2's output is the next block's kept input, and
 * its backward needs only the input).  Results are bit-identical to what the
 * forward pass computed.  Needs no upstream gradient
 * (early recomputation).  MERAK_ERR_ORDER if no forward pass is pending.  A
 * no-op (MERAK_OK) when the mask is 0.  params must hold the same values as in
 * the forward call.
 * The streams may differ from the ones the backward will use: the backward of
 * each recomputed block waits for that block's recomputation only, so the
 * recomputation of the first blocks can overlap the backward of the later
 * ones (which the backward reaches first).  The caller orders these streams
 * after the forward pass (the block inputs are its results). */
int merak_stage_recompute(merak_stage_t stage, const void* params, void* stream0, void* stream1);

/* Backward pass of the stage for the pending micro-batch.
 *   dy            [b, s, h] (dtype): gradient of the stage output.
 *   dx            [b, s, h] (dtype): gradient of the stage input.
 *   grads         [total_elems] fp32: parameter gradients, same layout as params;
 *                 overwritten when accumulate = 0, added to when accumulate = 1.
 *   bwd_partials  NULL or [L][2][b, s, h] (dtype): [l][0] = block l's partial of
 *                 the LN1-output gradient (dqkv W_qkv), [l][1] = the partial of
 *                 the LN2-output gradient (du W1): the inputs of the two backward
 *                 AllReduces.
 * Weight gradients are computed per block over the whole micro-batch once all
 * its sub-micro-batches are done (deterministic; no floating-point atomics).
 * MERAK_ERR_ORDER if no forward pass is pending, if the mask is nonzero and
 * merak_stage_recompute has not run since the forward pass, or if another
 * handle has recomputed into a shared recompute area since.  Consumes the
 * pending micro-batch. */
int merak_stage_bwd(merak_stage_t stage, const void* params, const void* dy, void* dx,
                    float* grads, int accumulate, void* bwd_partials, void* stream0,
                    void* stream1);

/* Kernel classes the stage launches (for merak_stage_set_timing). */
typedef enum {
  MERAK_KC_NONE = 0,
  MERAK_KC_GEMM_FWD = 1,   /* QKV, projection, FC1, FC2 GEMMs (forward and recompute)    */
  MERAK_KC_GEMM_DX = 2,    /* input-gradient GEMMs of the backward pass                  */
  MERAK_KC_GEMM_DW = 3,    /* weight-gradient GEMMs of FC1 and FC2, one launch per block */
  MERAK_KC_ATTN_FWD = 4,   /* attention forward                                          */
  MERAK_KC_ATTN_BWD = 5,   /* attention backward (dQ with delta, then dK/dV kernels)     */
  MERAK_KC_LN_FWD = 6,     /* LayerNorm forward                                          */
  MERAK_KC_LN_BWD = 7,     /* LayerNorm backward (input gradient)                        */
  MERAK_KC_REDUCE = 8,     /* bias / LayerNorm parameter gradient reductions             */
  MERAK_KC_GEMM_DW_ATTN = 9, /* weight-gradient GEMMs of QKV and projection, one per block */
  MERAK_KC_COUNT = 10
} merak_kernel_class;

/* Measurement aid: from now on, bracket every launch of `kernel_class` made by
 * this handle with a pair of HIP events recorded on the stream the launch goes
 * to (MERAK_KC_NONE turns it off).  At most 4096 launches are recorded between
 * two reads.  Host-side bookkeeping only; results do not change. */
int merak_stage_set_timing(merak_stage_t stage, int kernel_class);

/* Failure injection for tests of the error paths: after `launches` more kernel
 * launches by the stage calls (any handle), the next one is not made and its
 * call returns MERAK_ERR_HIP, as if the launch had failed; -1 turns it off.
 * Returns the previous setting.  A stage call that fails part-way leaves its
 * handle refusing the calls that depend on it: a failed fwd leaves the handle
 * idle, a failed recompute leaves it (and any handle that filled the same
 * recompute area before) unable to run bwd, a failed bwd leaves it idle. */
int merak_debug_fail_after(int launches);

/* After the caller has synchronised: total milliseconds of the recorded launches
 * (sum of per-launch event intervals) and their count; then clears the record.
 * MERAK_ERR_ORDER if more than 4096 launches were made since the last read. */
int merak_stage_read_timing(merak_stage_t stage, double* total_ms, int64_t* launches);

/* ------------------------------------------------------------------------
 * Stage-aware recomputation planner (paper Sec. 5.2).  Host-only, no GPU.
 *
 * Stage i of s (numbered from 1) keeps the activations of a share alpha_i of
 * its blocks and recomputes the rest.  Keeping them costs (s - i) * alpha_i *
 * M_a on top of the runtime memory M_r (stage i holds s - i micro-batches in
 * flight); all stages are given the same memory, which fixes
 *   alpha_i = min(1, (s - 1) alpha_1 / (s - i))   for 2 <= i < s - 1,
 *   alpha_{s-1} = alpha_{s-2},  alpha_s = 1  (shifted critical path schedule).
 * A stage with L blocks keeps floor(alpha_i * L) of them; the recompute mask
 * (MERAK config field recompute_mask) has bits 0 .. L - keep - 1 set.
 * ---------------------------------------------------------------------- */

/* alpha[0..s-1] and masks[0..s-1] for s stages (1 <= s <= 4096), 0 <= alpha1
 * <= 1, blocks_per_stage in 1..64.  MERAK_ERR_INVALID_ARG / MERAK_ERR_SHAPE on
 * bad arguments (nothing written). */
int merak_plan_recompute(int n_stages, double alpha1, int blocks_per_stage, double* alpha, uint64_t* masks);

/* The largest alpha_1 on the grid 0, step, 2 step, ... (capped at 1) for which
 * every stage fits: M_r + (s - i) alpha_i M_a <= capacity (the paper raises
 * alpha_1 until an out-of-memory error; this memory model stands in for it).
 * MERAK_ERR_UNSUPPORTED if even alpha_1 = 0 does not fit. */
int merak_plan_alpha1(int n_stages, double mem_runtime, double mem_activation, double capacity, double step,
                      double* alpha1);

/* ------------------------------------------------------------------------
 * Pipeline schedules (paper Sec. 5.1).  Host-only, no GPU.
 *
 * Per stage, the order of its forward (F), recomputation (R) and backward (B)
 * calls over m micro-batches; a stage runs them with merak_stage_fwd,
 * merak_stage_recompute and merak_stage_bwd (one handle per micro-batch in
 * flight).  Dependencies: F of stage i needs F of stage i-1, B needs B of
 * stage i+1 and the stage's own R of that micro-batch; R needs nothing from
 * other stages.
 *   MERAK_SCHED_1F1B:  s-1-i warm-up forwards, then one forward / one backward,
 *     the backward recomputing first (op MERAK_OP_RECOMPUTE_BWD);
 *   MERAK_SCHED_EARLY_RECOMPUTE: the same with R split off, run as soon as the
 *     stage is free;
 *   MERAK_SCHED_SCP (shifted critical path): the last stage skips R; the
 *     penultimate stage runs F0 F1 R0 F2 B0 and then R_j B_j F_{j+2}; the other
 *     stages as in early recomputation.
 * With costs F = R = T_m, B = 2 T_m the bubble ratios (makespan - 4 m T_m) /
 * (4 m T_m) are (s-1)/m, 3(s-1)/(4m) and 3(s-2)/(4m) for m >= s.
 * ---------------------------------------------------------------------- */
typedef enum { MERAK_SCHED_1F1B = 0, MERAK_SCHED_EARLY_RECOMPUTE = 1, MERAK_SCHED_SCP = 2 } merak_schedule_kind;
typedef enum { MERAK_OP_FWD = 0, MERAK_OP_RECOMPUTE = 1, MERAK_OP_BWD = 2, MERAK_OP_RECOMPUTE_BWD = 3 } merak_op_type;

/* Op list of one stage: ops[k] = (type << 24) | micro_batch, k < *n_ops
 * (at most 3 m).  1 <= n_stages <= 1024, 1 <= n_micro < 2^24, 0 <= stage <
 * n_stages.  MERAK_ERR_WORKSPACE if capacity is too small (*n_ops = needed). */
int merak_schedule_stage(int kind, int n_stages, int n_micro, int stage, int32_t* ops, int capacity, int* n_ops);

/* Largest number of this stage's micro-batches between their forward and their
 * backward at any point of its op list (the handles merak_schedule_run needs). */
int merak_schedule_inflight(int kind, int n_stages, int n_micro, int stage, int* max_inflight);

/* Run stage `stage`'s op list on this GPU: each F, R and B becomes a
 * merak_stage_fwd, merak_stage_recompute or merak_stage_bwd call (an R+B op
 * both), on stream0/stream1, in list order.  Micro-batch j reads x[j] and dy[j]
 * and writes y[j] and dx[j] ([micro_batch, seq_len, hidden] each, as for the
 * stage calls); the inputs of other stages are the caller's (on one GPU they
 * are already resident).  A micro-batch takes one of the n_handles handles at
 * its forward and returns it after its backward, so n_handles must be at least
 * merak_schedule_inflight(...) (else MERAK_ERR_WORKSPACE); the handles must be
 * distinct, share one configuration (else MERAK_ERR_SHAPE) and may share one
 * recompute area when at most one micro-batch is between R and B at a time, as
 * in these schedules (a taken-over area gives MERAK_ERR_ORDER).  The backwards
 * add into grads in micro-batch order; the first one overwrites it when
 * accumulate = 0.  Under MERAK_SCHED_SCP the last stage runs no R, so its
 * handles need recompute_mask = 0 (else its first backward returns
 * MERAK_ERR_ORDER).  Arguments are checked before anything is enqueued; an
 * error returned by a stage call leaves the calls before it enqueued. */
int merak_schedule_run(int kind, int n_stages, int n_micro, int stage, merak_stage_t* handles, int n_handles,
                       const void* params, const void* const* x, void* const* y, const void* const* dy,
                       void* const* dx, float* grads, int accumulate, void* stream0, void* stream1);

/* Greedy in-order execution of all stages' op lists with the given costs
 * (a recompute-in-backward op costs cost_rc + cost_bwd): the makespan and each
 * stage's busy time (busy[0..n_stages-1]).  n_stages * n_micro <= 2^22. */
int merak_schedule_simulate(int kind, int n_stages, int n_micro, double cost_fwd, double cost_rc, double cost_bwd,
                            double* makespan, double* busy);

/* ------------------------------------------------------------------------
 * Graph sharding (paper Sec. 4.2, Alg. 1 "Search Node Dependency" and Alg. 2
 * "Graph-Sharding").  Host-only, no GPU.
 *
 * Splits a model's dataflow graph into a sequence of subgraphs that run one
 * after the other, so that consecutive runs of the sequence can be assigned to
 * pipeline stages.  Nodes are visited in topological order; a node joins the
 * subgraph of its farthest dependency (a graph input's first user, the
 * subgraph after the one whose output it reads, or the subgraph of any other
 * earlier node except the last visited one), pulling the nodes visited since
 * that dependency along; common nodes (cheap values used all over the graph,
 * such as a causal mask) are no dependency.  A subgraph closes once its
 * parameters exceed sum(params) / k; its outputs are the closing node plus the
 * visited common nodes that still have uses left.
 *
 * Readings where the paper is silent: a node reading a graph input twice is
 * no dependency of itself; the dependency node itself keeps its
 * subgraph when later nodes join it; reopening a subgraph drops the outputs
 * recorded for it and for every later subgraph; the last subgraph is emitted
 * even if it never closed, with the graph outputs as its outputs; a
 * subgraph's inputs are the previous subgraph's outputs plus the graph inputs
 * whose first user it holds.
 *
 * Graph (n_nodes nodes in topological order, graph inputs included):
 *   kind[i]         MERAK_NODE_COMPUTE, MERAK_NODE_INPUT (a graph input: no
 *                   arguments, not assigned to a subgraph) or MERAK_NODE_COMMON;
 *   params[i]       parameters the node holds (>= 0);
 *   arg_ptr[0..n_nodes], arg_idx[]: node i's arguments are
 *                   arg_idx[arg_ptr[i] .. arg_ptr[i+1]), one entry per use,
 *                   each an index < i;
 *   common_uses[i]  for common nodes, how many argument entries name it;
 *   graph_outputs[0..n_outputs-1]: node indices the graph returns;
 *   k               requested number of subgraphs (>= 1).
 * Result:
 *   subgraph_of[i]  subgraph id of node i (-1 for graph inputs);
 *   *n_subgraphs;
 *   io_ptr[0..2 * n_nodes], io_idx[0..io_capacity-1]: subgraph j's inputs are
 *   io_idx[io_ptr[2j] .. io_ptr[2j+1]) and its outputs io_idx[io_ptr[2j+1] ..
 *   io_ptr[2j+2]) (node indices).
 * Errors: MERAK_ERR_INVALID_ARG (null pointers, n_nodes < 1, k < 1, an
 * argument index not smaller than its node's, a graph input with arguments,
 * an unknown kind, negative params or uses), MERAK_ERR_WORKSPACE if io_idx
 * is too small (*n_subgraphs is still set; io_ptr[2 * *n_subgraphs] then
 * holds the capacity needed).  Nothing else is written on an argument error.
 * ---------------------------------------------------------------------- */
typedef enum { MERAK_NODE_COMPUTE = 0, MERAK_NODE_INPUT = 1, MERAK_NODE_COMMON = 2 } merak_node_kind;

int merak_graph_shard(int n_nodes, const int32_t* kind, const int64_t* params, const int32_t* arg_ptr,
                      const int32_t* arg_idx, const int32_t* common_uses, int n_outputs,
                      const int32_t* graph_outputs, int k, int32_t* subgraph_of, int32_t* n_subgraphs,
                      int32_t* io_ptr, int32_t* io_idx, int io_capacity);

/* ------------------------------------------------------------------------
 * Per-kernel entry points (each launches one hot-path kernel on `stream`).
 * They exist so each kernel can be checked and timed on its own; the stage
 * calls above use the same kernels.  dtype is merak_dtype; pointers follow the
 * conventions above (16-byte aligned).  No entry point allocates memory.
 * Every size argument must be positive: an empty input (rows, M, N, K, seq,
 * batch or heads of 0) returns MERAK_ERR_SHAPE with nothing enqueued.
 * ---------------------------------------------------------------------- */

/* GEMM epilogues. */
typedef enum {
  MERAK_EPI_STORE = 0,      /* C = acc                                               (dtype) */
  MERAK_EPI_BIAS = 1,       /* C = acc + bias[n]                                     (dtype) */
  MERAK_EPI_BIAS_GELU = 2,  /* aux = u = acc + bias[n];  C = GeLU_tanh(u)            (dtype) */
  MERAK_EPI_BIAS_RESID = 3, /* aux = acc (skipped if aux is NULL); C = resid + acc + bias[n] */
  MERAK_EPI_GELU_BWD = 4,   /* C = acc * GeLU_tanh'(aux), aux holding the stored u   (dtype) */
  MERAK_EPI_F32 = 5         /* fp32 C = acc, or C += acc when accumulate = 1                 */
} merak_epilogue;

/* GEMM of the shard's linear layers: C[M,N] = op(A)[M,K] * op(B)[K,N], fp32
 * accumulation (bf16 MFMA in MERAK_BF16 mode).
 *   a_trans = 0: A[m,k] at a[m*lda + k];  1: A[m,k] at a[k*lda + m].
 *   b_trans = 0: B[k,n] at b[n*ldb + k] (a weight [N,K]: "X W^T");
 *             1: B[k,n] at b[k*ldb + n].
 * M, N, K must be positive multiples of 64 and lda, ldb multiples of 8, and in
 * MERAK_BF16 each operand, counted with 256 rows of edge-tile padding past M
 * (or N), must span fewer than 2^31 bytes (else MERAK_ERR_SHAPE).  C, resid and aux are [M, N] row-major (ld = N); bias is
 * [N].  Elements are of `dtype` except C for MERAK_EPI_F32 (always fp32). */
int merak_gemm(int dtype, int a_trans, int b_trans, int epilogue, int M, int N, int K,
               const void* a, int lda, const void* b, int ldb, void* c, const void* bias,
               const void* resid, void* aux, int accumulate, void* stream);

/* Tile-shape override of the bf16 GEMM kernel, for tests and tuning:
 * 0 restores the built-in choice, 1..10 force one shape (256x256/4 waves/2
 * stages, 256x128/4/3, 128x256/4/3, 128x128/4/2, 128x128/4/3, 128x128/4/4,
 * 256x256/8/2, 256x128/8/3, 128x192/4/2, 256x192/8/2).  Process-wide; returns the previous value, or -1
 * for an out-of-range cfg (nothing changed).  Host-only, not thread-safe. */
int merak_gemm_tile_override(int cfg);

/* LayerNorm forward over `rows` rows of width h (h % 8 == 0, h <= 8192):
 * y = gamma * (x - mean) * rstd + beta; mean and rstd fp32 [rows]. */
int merak_layernorm_fwd(int dtype, int rows, int h, float eps, const void* x, const void* gamma,
                        const void* beta, void* y, float* mean, float* rstd, void* stream);

/* fp32 scratch elements needed by the column reductions below for a
 * [rows, cols] input (0 for empty input). */
size_t merak_reduce_scratch_elems(int rows, int cols);

/* LayerNorm backward fused with the residual-gradient add:
 * dx = dres + LN'(dout).  dgamma = sum over rows of dout * xhat, dbeta = sum of
 * dout, both written (accumulate = 0) or added (accumulate = 1), summed in a
 * fixed order (deterministic).  scratch: fp32, 2 * merak_reduce_scratch_elems(rows, h). */
int merak_layernorm_bwd(int dtype, int rows, int h, const void* dout, const void* x,
                        const float* mean, const float* rstd, const void* gamma,
                        const void* dres, void* dx, float* dgamma, float* dbeta,
                        int accumulate, float* scratch, void* stream);

/* merak_layernorm_bwd without the scratch argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, kernels and results as
 * merak_layernorm_bwd (bit for bit).  The partial sums go to a scratch array the
 * library holds in its own device memory: merak_noalloc_scratch_elems() fp32
 * elements (16 MiB) per GPU, kept until the process ends; the call allocates
 * nothing.  Requires 2 * merak_reduce_scratch_elems(rows, h) <=
 * merak_noalloc_scratch_elems(), else MERAK_ERR_WORKSPACE with nothing
 * enqueued.  The first call on a device looks up the array's address there
 * (MERAK_ERR_HIP if that fails).  Every call on one GPU shares that GPU's
 * array: calls that may overlap on one GPU (other streams, other host threads)
 * race and must be ordered by the caller. */
int merak_layernorm_bwd_noalloc(int dtype, int rows, int h, const void* dout, const void* x,
                                const float* mean, const float* rstd, const void* gamma,
                                const void* dres, void* dx, float* dgamma, float* dbeta,
                                int accumulate, void* stream);
size_t merak_noalloc_scratch_elems(void);

/* out[c] (= or +=) sum over rows r of x[r, c] (fp32 out; cols % 8 == 0), fixed
 * summation order.  scratch: fp32, merak_reduce_scratch_elems(rows, cols). */
int merak_column_sum(int dtype, int rows, int cols, const void* x, float* out, int accumulate,
                     float* scratch, void* stream);

/* Failure detection: the number of NaN and +-Inf elements among the n elements
 * of x (dtype; 16-byte aligned unless n = 0) is written to *count, a device
 * uint64 (16-byte aligned) that the call overwrites; read it after the stream
 * has reached the call.  n = 0 writes 0.  An integer count, so it does not
 * depend on timing.  Enqueues two kernels and allocates nothing. */
int merak_count_nonfinite(int dtype, const void* x, int64_t n, uint64_t* count, void* stream);

/* Causal attention forward on a packed qkv buffer [batch, seq, 3, heads, d]
 * (row stride 3*heads*d, the QKV GEMM's output layout): o [batch, seq, heads, d]
 * and lse fp32 [batch, heads, seq] = natural log of sum_j exp(q_i k_j / sqrt(d))
 * over j <= i.  seq % 64 == 0; d in {64, 96, 128}. */
int merak_attention_fwd(int dtype, int batch, int seq, int heads, int head_dim,
                        const void* qkv, void* o, float* lse, void* stream);

/* Causal attention backward: dqkv [batch, seq, 3, heads, d] from qkv, o, lse and
 * dout [batch, seq, heads, d].  delta: fp32 scratch of batch*heads*seq elements.
 * Deterministic (no atomics). */
int merak_attention_bwd(int dtype, int batch, int seq, int heads, int head_dim,
                        const void* qkv, const void* o, const float* lse, const void* dout,
                        void* dqkv, float* delta, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* MERAK_STAGE_H */
