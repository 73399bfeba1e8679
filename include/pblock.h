/*
 * pblock.h — C ABI of the MI355X (gfx950) parallel transformer block library.
 *
 * The block is Eq. 2 of MegaScale (Section 3.1):
 *
 *     y = x + MLP(LN(x)) + Attention(LN(x))
 *
 * with ONE LayerNorm whose output h feeds both branches, a fused in-projection
 * Z = h W_in^T + b_in whose columns are [Q | K | V | U], causal sliding-window
 * attention (Section 3.1, "Sliding window attention") on Q, K, V, the GeLU MLP
 * activation G = gelu(U), and one fused out-projection over C = [O | G]:
 *
 *     y = x + C W_out^T + b_out.
 *
 * Window rule: query i attends to key j of the same batch row iff
 * 0 <= i - j < window (window keys, the query's own position included);
 * window >= seq is ordinary causal attention.  Scores are scaled by
 * 1/sqrt(head_dim).  LayerNorm uses the biased variance with eps inside the
 * square root.  GeLU is the tanh form when gelu_tanh != 0, else the erf form.
 *
 * Section 3.3 replaces attention with FlashAttention-2 and LN/GeLU with fused
 * kernels; this library does the same on gfx950 (banded flash-style attention
 * that skips key tiles outside the window, MFMA GEMMs with fused bias / GeLU /
 * residual epilogues).  None of that changes the result beyond rounding.
 *
 * ---------------------------------------------------------------- layouts
 * All tensors are dense, row-major, in device memory (HBM), 16-byte aligned.
 * Let T = batch*seq, H = hidden, A = heads*head_dim, F = ffn,
 *     N_in = 3A + F, K_out = A + F.
 *   x, y, dy, dx  [T, H]          activation dtype (bf16 or fp32), token-major
 *   ln_gamma/beta [H]             activation dtype
 *   w_in          [N_in, H]       activation dtype; rows Q | K | V | MLP-up;
 *                                 head h owns rows h*d .. h*d+d-1 of each of
 *                                 Q, K and V (d = head_dim)
 *   b_in          [N_in]          activation dtype
 *   w_out         [H, K_out]      activation dtype; columns attention-out |
 *                                 MLP-down (the two output projections of
 *                                 Eq. 2, side by side)
 *   b_out         [H]             activation dtype: the sum of the attention
 *                                 and MLP output biases (only their sum enters
 *                                 Eq. 2)
 *   dgamma, dbeta [H], dw_in [N_in, H], db_in [N_in], dw_out [H, K_out],
 *   db_out [H]                    fp32, always
 *
 * Saved stash (forward -> backward), regions in this order, each starting at
 * a 256-byte boundary (see pblock_saved_offsets):
 *   h     [T, H]      act   LN output
 *   z     [T, N_in]   act   Q | K | V | U  (U before GeLU)
 *   c     [T, K_out]  act   O | G          (attention output, GeLU output)
 *   mean  [T]         fp32  LN row mean
 *   rstd  [T]         fp32  LN row 1/sqrt(var + eps)
 *   lse   [batch, heads, seq] fp32  log of each softmax denominator, in the
 *                     scaled-score domain
 *
 * ---------------------------------------------------------------- ownership
 * The caller allocates every buffer (inputs, outputs, the stash, the
 * workspace).  The library allocates no device memory and keeps no state
 * between calls: the HIP events that the pipelined all-gather and
 * reduce-scatter order their streams with live in a pb_tp_context that the
 * caller creates and destroys, and the step events of the *_timed calls are
 * passed with each call.  (pblock_swattn_forward_noalloc alone uses a
 * library-owned device array; see there.)  Every call is
 * asynchronous on the given HIP stream; buffers must stay valid until the
 * stream has passed the call.  Other calls on disjoint buffers may run
 * concurrently.  Parameter gradients are overwritten, not accumulated.
 * The block's forward and backward calls (parallel and serial) only launch
 * kernels on the given stream (no allocation, memset, copy or
 * synchronisation), so a caller may capture them into a HIP graph and
 * replay it.
 *
 * ---------------------------------------------------------------- errors
 * Functions return a pb_status.  Arguments are checked on the host before any
 * HIP call is made; on a failed check nothing is launched and
 * pblock_last_error() describes the problem.  PB_ERR_HIP reports a launch
 * failure (hipGetLastError after the launches).  Nothing throws, aborts or
 * exits across this interface.
 */
#ifndef PBLOCK_H
#define PBLOCK_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { PB_BF16 = 0, PB_F32 = 1 } pb_dtype;

typedef enum {
  PB_OK = 0,
  PB_ERR_INVALID_ARG = 1, /* null/misaligned pointer, non-positive size ... */
  PB_ERR_UNSUPPORTED = 2, /* a shape this build has no kernel for          */
  PB_ERR_WORKSPACE = 3,   /* workspace smaller than pblock_workspace_bytes */
  PB_ERR_HIP = 4          /* a kernel launch failed                        */
} pb_status;

typedef struct {
  int batch;     /* >= 1                                                    */
  int seq;       /* >= 1                                                    */
  int hidden;    /* H >= 8, multiple of 8, <= 32768                         */
  int heads;     /* >= 1                                                    */
  int head_dim;  /* 64, 96 or 128                                           */
  int ffn;       /* F >= 8, multiple of 8                                   */
  int window;    /* >= 1; keys seen per query, itself included              */
  float ln_eps;  /* > 0, e.g. 1e-5                                          */
  int gelu_tanh; /* 1: tanh form of GeLU, 0: erf form                      */
  pb_dtype dtype;/* storage type of activations and parameters              */
} pb_config;

/* Checks a configuration on the host.  Makes no HIP call. */
pb_status pblock_validate(const pb_config* cfg);

/* Bytes of the forward -> backward stash described above (0 on a bad cfg). */
size_t pblock_saved_bytes(const pb_config* cfg);

/* Byte offsets of the stash regions, in the order h, z, c, mean, rstd, lse.
 * offsets must hold 6 entries.  Host only. */
pb_status pblock_saved_offsets(const pb_config* cfg, size_t* offsets);

/* Workspace sizes.  mode:
 *   PB_WS_FORWARD             pblock_forward with a caller stash (saved != NULL)
 *   PB_WS_FORWARD_WITH_STASH  pblock_forward with saved == NULL: the stash is
 *                             kept at the start of ws
 *   PB_WS_BACKWARD            pblock_backward
 * The sizes include a region for tail-split GEMM partial tiles (the last,
 * partial wave of output tiles is split along K so the chip stays full).
 * That region is optional: a smaller ws (down to 0 bytes for PB_WS_FORWARD,
 * the stash for PB_WS_FORWARD_WITH_STASH, and the size without the region
 * for PB_WS_BACKWARD) also works, unsplit (results then differ only in
 * rounding order).  0 on a bad cfg. */
enum { PB_WS_FORWARD_WITH_STASH = 0, PB_WS_BACKWARD = 1, PB_WS_FORWARD = 2 };
size_t pblock_workspace_bytes(const pb_config* cfg, int mode);

/* Steps of the forward and backward passes, for the *_timed calls. */
typedef enum {
  PB_STEP_LN_FWD = 0, /* LayerNorm of x                                     */
  PB_STEP_IN_PROJ,    /* Z = h W_in^T + b_in, G = gelu(U)                   */
  PB_STEP_ATTN_FWD,   /* sliding-window attention, O and lse                */
  PB_STEP_OUT_PROJ,   /* y = x + C W_out^T + b_out                          */
  PB_STEP_DC,         /* dC = dy W_out; dU = dC_mlp * gelu'(U)              */
  PB_STEP_DW_OUT,     /* dW_out = dy^T C                                    */
  PB_STEP_DB_OUT,     /* empty: db_out is summed with dgamma and dbeta in
                         the LN backward step's column sums              */
  PB_STEP_ATTN_BWD,   /* dQ, dK, dV                                         */
  PB_STEP_DH,         /* dh = dZ W_in                                       */
  PB_STEP_DW_IN,      /* dW_in = dZ^T h                                     */
  PB_STEP_DB_IN,      /* db_in = sum over tokens of dZ; empty when formed
                         in dW_in's launch shared with dh                 */
  PB_STEP_LN_BWD,     /* dx = dy + LN backward; dgamma, dbeta, db_out       */
  PB_STEP_COUNT
} pb_step;

/* Per-call step events (benchmarking).  pblock_forward_timed and
 * pblock_backward_timed record begin[i] on their stream just before the
 * launches of step i and end[i] just after them; NULL entries, and a NULL
 * pb_step_events, are skipped.  The events belong to the caller and are
 * only recorded, never waited on.  A step whose work shares a launch with
 * another step records nothing between its events (PB_STEP_DW_OUT, and
 * PB_STEP_DW_IN and PB_STEP_DB_IN, when pblock_backward_pairs reports the
 * pair; PB_STEP_DB_OUT always). */
typedef struct {
  hipEvent_t begin[PB_STEP_COUNT];
  hipEvent_t end[PB_STEP_COUNT];
} pb_step_events;

/* Forward pass of the block (Eq. 2).  Writes y [T, H].  When saved is not
 * NULL it also fills the stash that pblock_backward reads, and ws (NULL or
 * up to pblock_workspace_bytes(cfg, PB_WS_FORWARD) bytes) only holds GEMM
 * partial tiles.  When saved is NULL (inference) the stash goes to the start
 * of ws, which must then hold at least the stash
 * (pblock_workspace_bytes(cfg, PB_WS_FORWARD_WITH_STASH) for full speed). */
pb_status pblock_forward(const pb_config* cfg, const void* x,
                         const void* ln_gamma, const void* ln_beta,
                         const void* w_in, const void* b_in,
                         const void* w_out, const void* b_out,
                         void* y, void* saved, void* ws, size_t ws_bytes,
                         hipStream_t stream);
/* pblock_forward, recording step_ev (NULL: none) around each step. */
pb_status pblock_forward_timed(const pb_config* cfg, const void* x,
                               const void* ln_gamma, const void* ln_beta,
                               const void* w_in, const void* b_in,
                               const void* w_out, const void* b_out,
                               void* y, void* saved, void* ws,
                               size_t ws_bytes, hipStream_t stream,
                               const pb_step_events* step_ev);

/* Byte offsets, within the backward workspace, of the intermediates that
 * pblock_backward leaves there, in the order:
 *   d_o [T, A]     act  the attention output's gradient (dC[:, :A])
 *   dz  [T, N_in]  act  dQ | dK | dV | dU, the in-projection's output
 *                       gradient (dQ, dK, dV from the attention backward)
 *   dh  [T, H]     act  the LayerNorm output's gradient
 *   delta [batch, heads, seq] fp32  the attention backward's row terms
 *                       rowsum(dO O) per head
 * They hold these values once the backward call has passed on its stream,
 * until the workspace is used again.  offsets must hold 4 entries.  Host
 * only; for inspection and tests. */
pb_status pblock_workspace_offsets(const pb_config* cfg, size_t* offsets);

/* Backward pass: the gradients of sum(y * dy) with respect to x and every
 * parameter, given the stash of the matching forward call.  dx is in the
 * activation dtype; the six parameter gradients are fp32 and overwritten.
 * ws should hold pblock_workspace_bytes(cfg, PB_WS_BACKWARD) bytes (fewer,
 * down to the size without the GEMM partial-tile region, also works).
 * Where dC and dW_out (dh and dW_in) share a launch, that launch is
 * persistent: one workgroup per CU takes tiles from per-XCD queues whose
 * heads live in ws and are zeroed by the call itself, so ws needs no
 * initialisation and two calls in flight at once need separate workspaces
 * (as for every other region of ws). */
pb_status pblock_backward(const pb_config* cfg, const void* x,
                          const void* ln_gamma, const void* ln_beta,
                          const void* w_in, const void* b_in,
                          const void* w_out, const void* b_out,
                          const void* saved, const void* dy, void* dx,
                          float* dgamma, float* dbeta, float* dw_in,
                          float* db_in, float* dw_out, float* db_out,
                          void* ws, size_t ws_bytes, hipStream_t stream);
/* pblock_backward, recording step_ev (NULL: none) around each step. */
pb_status pblock_backward_timed(const pb_config* cfg, const void* x,
                                const void* ln_gamma, const void* ln_beta,
                                const void* w_in, const void* b_in,
                                const void* w_out, const void* b_out,
                                const void* saved, const void* dy, void* dx,
                                float* dgamma, float* dbeta, float* dw_in,
                                float* db_in, float* dw_out, float* db_out,
                                void* ws, size_t ws_bytes, hipStream_t stream,
                                const pb_step_events* step_ev);

/* ------------------------------------------------------- launch planning
 * Host-only queries of how the calls above launch their GEMMs (for
 * benchmarks and profilers that attribute kernel time to steps).  They make
 * no HIP call.
 *
 * pblock_gemm_plan: the launch of one GEMM C[M, N] = A[M, K] B[K, N] in
 * dtype, given a full GEMM workspace (as the block's calls have).  256 x 256
 * output tiles; when the last wave of tiles is partial (or the whole grid is
 * smaller than the 256 compute units), each of its `tail` tiles is split
 * into `splits` K-slices whose fp32 partial tiles a second kernel sums.
 * Fills tiles, n_full (tiles computed whole), tail, splits (1: no split),
 * workgroups (of the GEMM kernel: n_full + tail * splits) and threads (per
 * workgroup).  bf16 with K % 64 == 0 takes the matrix-core path that splits;
 * anything else launches unsplit (the fp32 path's tiles are 64 x 64).
 *
 * pblock_backward_pairs: which backward GEMMs share one launch with the
 * weight-gradient GEMM after them (1) or launch alone (0).  block 0, the
 * parallel block: paired[0] = dC with dW_out, paired[1] = dh with dW_in.
 * block 1, the serial block: paired[0..3] = dG with dW_down, dh2 with
 * dW_up, dO with dW_o, dh1 with dW_qkv.  A shared launch has
 * tiles(first) + tiles(second) workgroups. */
typedef struct {
  int tiles, n_full, tail, splits, workgroups, threads;
} pb_gemm_plan;
pb_status pblock_gemm_plan(pb_dtype dtype, int M, int N, int K,
                           pb_gemm_plan* plan);
pb_status pblock_backward_pairs(const pb_config* cfg, int block, int* paired);

/* ---------------------------------------------------------- serial block
 * The standard pre-LN block that Eq. 2 replaces (Section 3.1, Eq. 1), for
 * comparison and for models that keep it:
 *
 *     x1 = x + Attention(LN1(x)) W_o^T + b_o
 *     y  = x1 + gelu(LN2(x1) W_up^T + b_up) W_down^T + b_down
 *
 * The second residual adds x1 (the paper's printed Eq. 1 writes x there; the
 * block it describes, and the one this computes, carries x1).  Weights use
 * the parallel block's packed layouts as slices: W_qkv = w_in rows 0..3A-1,
 * W_up = rows 3A..N_in-1 (b_in likewise); W_o = w_out columns 0..A-1, W_down
 * = columns A..K_out-1.  Two LayerNorms (ln1_*, ln2_*, activation dtype [H])
 * and two output biases (b_o, b_down, activation dtype [H]); the same window
 * rule, scaling, LayerNorm and GeLU as above.
 *
 * Stash regions, in this order, each at a 256-byte boundary
 * (pblock_serial_saved_offsets, 10 entries):
 *   h1 [T, H] act, z [T, N_in] act (Q | K | V | U), c [T, K_out] act (O | G),
 *   mean1 [T] fp32, rstd1 [T] fp32, lse [batch, heads, seq] fp32,
 *   x1 [T, H] act, h2 [T, H] act, mean2 [T] fp32, rstd2 [T] fp32.
 *
 * Workspace modes, ownership, asynchrony and errors are those of the
 * parallel block's calls (pblock_serial_workspace_bytes takes the same
 * PB_WS_* modes).  Gradients dln1_*, dln2_*, dw_in, db_in, dw_out, db_o,
 * db_down are fp32, in the layouts of their parameters, and overwritten. */
size_t pblock_serial_saved_bytes(const pb_config* cfg);
pb_status pblock_serial_saved_offsets(const pb_config* cfg, size_t* offsets);
size_t pblock_serial_workspace_bytes(const pb_config* cfg, int mode);
pb_status pblock_serial_forward(const pb_config* cfg, const void* x,
                                const void* ln1_gamma, const void* ln1_beta,
                                const void* ln2_gamma, const void* ln2_beta,
                                const void* w_in, const void* b_in,
                                const void* w_out, const void* b_o,
                                const void* b_down, void* y, void* saved,
                                void* ws, size_t ws_bytes, hipStream_t stream);
pb_status pblock_serial_backward(const pb_config* cfg, const void* x,
                                 const void* ln1_gamma, const void* ln1_beta,
                                 const void* ln2_gamma, const void* ln2_beta,
                                 const void* w_in, const void* b_in,
                                 const void* w_out, const void* b_o,
                                 const void* b_down, const void* saved,
                                 const void* dy, void* dx, float* dln1_gamma,
                                 float* dln1_beta, float* dln2_gamma,
                                 float* dln2_beta, float* dw_in, float* db_in,
                                 float* dw_out, float* db_o, float* db_down,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

/* Causal sliding-window attention alone (Section 3.1 SWA; the exact
 * FlashAttention-2 result of Section 3.3), for all heads of all batch rows.
 * q, k, v: element (b, s, head, e) at ptr[(b*seq + s)*ld + head*head_dim + e],
 * ld in elements (>= heads*head_dim, multiple of 8).  o uses ld_o the same
 * way.  lse [batch, heads, seq] fp32 as in the stash.  Reads cfg->batch, seq,
 * heads, head_dim, window and dtype only.
 *
 * Workspace (pblock_swattn_workspace_bytes, by mode):
 *   PB_ATTN_WS_FORWARD      optional space for the forward: when batch*heads
 *                           is too small to fill the GPU, the key range of
 *                           each query block is split over several
 *                           workgroups whose fp32 partial results are merged
 *                           afterwards.  ws may be NULL (or smaller), which
 *                           runs unsplit; 0 means no split is planned.
 *   PB_ATTN_WS_BACKWARD_MIN bytes the backward requires (one fp32 softmax row
 *                           term per query).
 *   PB_ATTN_WS_BACKWARD     the same plus the split backward's partials; any
 *                           size from _MIN up works, below this one unsplit.
 * Results of the split and unsplit runs agree to fp32 rounding; each is
 * deterministic (fixed merge order, no atomics). */
enum { PB_ATTN_WS_FORWARD = 0, PB_ATTN_WS_BACKWARD_MIN = 1, PB_ATTN_WS_BACKWARD = 2 };
size_t pblock_swattn_workspace_bytes(const pb_config* cfg, int mode);
pb_status pblock_swattn_forward(const pb_config* cfg, const void* q,
                                const void* k, const void* v, int ld_qkv,
                                void* o, int ld_o, float* lse, void* ws,
                                size_t ws_bytes, hipStream_t stream);

/* pblock_swattn_forward without a workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, layouts and results as
 * pblock_swattn_forward with a full PB_ATTN_WS_FORWARD workspace (the same
 * kernels and split plan; bitwise the same output).  The split partials
 * live in a device array inside the library, PB_NOALLOC_SCRATCH_BYTES per
 * GPU, held from the first call on that GPU (made with it current) until the
 * process ends.  Nothing is allocated per call and nothing in it needs
 * clearing.  A shape whose split plan needs more scratch than that is
 * rejected with PB_ERR_UNSUPPORTED before any HIP call.  Every call on one
 * GPU shares that GPU's scratch: calls that overlap on one GPU (on
 * different streams, or from several host threads) race and must be
 * ordered by the caller. */
#define PB_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
pb_status pblock_swattn_forward_noalloc(const pb_config* cfg, const void* q,
                                        const void* k, const void* v,
                                        int ld_qkv, void* o, int ld_o,
                                        float* lse, hipStream_t stream);

/* Gradient of pblock_swattn_forward: given q, k, v, o (ld_o), lse and the
 * output gradient d_o (ld_do), writes dq, dk, dv (ld_dqkv).  ws: see above
 * (at least PB_ATTN_WS_BACKWARD_MIN bytes, else PB_ERR_WORKSPACE). */
pb_status pblock_swattn_backward(const pb_config* cfg, const void* q,
                                 const void* k, const void* v, int ld_qkv,
                                 const void* o, int ld_o, const void* d_o,
                                 int ld_do, const float* lse, void* dq,
                                 void* dk, void* dv, int ld_dqkv, void* ws,
                                 size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------ tensor-parallel context
 * The HIP events with which pblock_ag_in_proj and pblock_rs_out_proj order
 * their copy streams against the GEMM stream: 3 tp + 1 events, created by
 * pblock_tp_context_create on the device current at that call, with timing
 * disabled.  A context serves calls with the same tp on that device, one
 * after another (re-recording an event between calls is safe: a stream
 * that waits on it has already taken the earlier state); calls from several
 * host threads need one context each.  pblock_tp_context_destroy may be
 * called once the calls that used it have been issued (HIP keeps a recorded
 * event alive until its work has passed); NULL is ignored.
 * Errors: PB_ERR_INVALID_ARG for tp outside 1..64 or ctx NULL, PB_ERR_HIP
 * when an event cannot be created (nothing is left allocated). */
typedef struct pb_tp_context pb_tp_context;
pb_status pblock_tp_context_create(int tp, pb_tp_context** ctx);
void pblock_tp_context_destroy(pb_tp_context* ctx);

/* ------------------------------------------- in-projection + all-gather
 * Section 3.2 ("Overlapping in tensor/sequence parallelism", Fig. 3):
 * under sequence parallelism the LayerNorm output h is sharded along the
 * tokens over tp ranks and all-gathered before the column-parallel
 * in-projection; the paper breaks that GEMM into chunks and pipelines them
 * with the communication.  Here the shards are copied into h on the comm
 * streams in ring order from `rank` (rank, rank + 1, ...; the k-th on
 * comm_streams[k % n_comm]), and the in-projection runs on `stream` in
 * launches of shards_per_launch shards each, every launch waiting (by
 * event) only for its own shards.  Shards already in place at the head of
 * that order (this rank's own LayerNorm output, say) need no copy and form
 * a first launch of their own, which runs while the first copies land.
 * shards_per_launch = tp is the unpipelined order: all copies, then one
 * GEMM.
 *
 * shards[j]: rank j's rows of h, [T / tp, H] in the activation dtype (on
 *   one GPU, buffers in local memory; across GPUs, peer memory opened by IPC
 *   handles).  A shard already in place (shards[j] == h + j (T / tp) H) is
 *   not copied.  h: [T, H], the gathered LN output.
 * z [T, N_in], c [T, K_out]: written as pblock_forward writes the stash's
 *   Z and the G half of C (bias, and GeLU of the MLP-up columns); the
 *   result does not depend on tp, rank or the launch grouping beyond the
 *   rounding of K-split tiles.
 * Requirements: T % tp == 0, 1 <= tp <= 64, 0 <= rank < tp,
 *   1 <= shards_per_launch <= tp, 1 <= n_comm <= 8, comm streams distinct
 *   from each other and from `stream`.
 * ws: optional GEMM split region of pblock_ag_in_proj_workspace_bytes(cfg,
 *   tp, shards_per_launch) bytes (NULL/0 runs every launch unsplit).
 * ctx: a pb_tp_context made for this tp on the current device.
 * The copies start after the work already on `stream`; later work on
 *   `stream` follows every copy and GEMM. */
size_t pblock_ag_in_proj_workspace_bytes(const pb_config* cfg, int tp,
                                         int shards_per_launch);
pb_status pblock_ag_in_proj(const pb_config* cfg, int tp, int rank,
                            const void* const* shards, void* h,
                            const void* w_in, const void* b_in, void* z,
                            void* c, int shards_per_launch, void* ws,
                            size_t ws_bytes, hipStream_t stream, int n_comm,
                            const hipStream_t* comm_streams,
                            pb_tp_context* ctx);

/* The same overlap in the backward pass (the mirror of the forward's
 * reduce-scatter): the output gradient dy arrives sharded along the tokens
 * and is all-gathered before dC = dy W_out, the first GEMM of the backward.
 * pblock_ag_dc copies dy_shards[j] ([T / tp, H], rank j's rows) into dy
 * [T, H] exactly as pblock_ag_in_proj copies the LayerNorm shards, and runs
 * dC over groups of shards_per_launch landed shards, writing d_o [T, A]
 * (= dC[:, :A]) and the MLP part of dz [T, N_in] (dz[:, 3A:] = dC[:, A:] *
 * gelu'(U), U read from z [T, N_in], the stash's Z) as pblock_backward
 * writes them.  w_out [H, K_out] as in pblock_forward.  Requirements, ws
 * (pblock_ag_dc_workspace_bytes) and ctx as for pblock_ag_in_proj.  The
 * weight gradient dW_out = dy^T C needs every shard and is left to the
 * caller (after the call, dy holds them all). */
size_t pblock_ag_dc_workspace_bytes(const pb_config* cfg, int tp,
                                    int shards_per_launch);
pb_status pblock_ag_dc(const pb_config* cfg, int tp, int rank,
                       const void* const* dy_shards, void* dy,
                       const void* w_out, const void* z, void* d_o, void* dz,
                       int shards_per_launch, void* ws, size_t ws_bytes,
                       hipStream_t stream, int n_comm,
                       const hipStream_t* comm_streams, pb_tp_context* ctx);

/* --------------------------------------- out-projection + reduce-scatter
 * Section 3.2 ("Overlapping in tensor/sequence parallelism", Fig. 3), the
 * other half of the pattern above: after the row-parallel out-projection
 * every rank holds a partial sum P_r = C_r W_out,r^T of every token row
 * (C_r, W_out,r: its own columns of the out-projection input and weight),
 * and a reduce-scatter leaves rank j with the sum over ranks of its own
 * rows.  The paper pipelines that GEMM in chunks with the communication.
 *
 * pblock_rs_out_proj (the sending side of rank `rank`) computes P_r on
 * `stream` in row chunks of T / tp rows, in ring order from rank + 1 (this
 * rank's own chunk last), shards_per_launch chunks per launch; each chunk
 * j is copied to dst[j] on comm_streams[k % n_comm] (k its position in that
 * order) as soon as its launch has finished.  shards_per_launch = tp is the
 * unpipelined order: one GEMM, then all copies.
 *   c [T, K_out], w_out [H, K_out]: as in pblock_forward, in the activation
 *     dtype; cfg describes this rank's share (A, F its own widths).
 *   partial [T, H]: P_r in the activation dtype (rounded from the fp32
 *     accumulation).  dst[j]: [T / tp, H], where rank j receives this
 *     rank's chunk (on one GPU, local buffers; across GPUs, peer memory
 *     opened by IPC handles).  A chunk already in place (dst[j] == partial
 *     + j (T / tp) H) is not copied.
 *   Requirements as for pblock_ag_in_proj; ws: optional GEMM split region
 *   of pblock_rs_out_proj_workspace_bytes(cfg, tp, shards_per_launch)
 *   bytes (NULL/0 runs every launch unsplit); ctx as for pblock_ag_in_proj.
 *   Later work on `stream` follows every GEMM and copy.
 *
 * pblock_rs_reduce (the receiving side of one rank): y_shard = x_shard +
 * b_out + sum over q = 0 .. tp-1 of parts[q], summed in fp32 in the order
 * of q and rounded once; parts[q], x_shard, y_shard: [T / tp, H] in the
 * activation dtype, 16-byte aligned; b_out: [H].  x_shard and b_out may
 * each be NULL (left out of the sum).  With parts[q] the chunk
 * rank q sent here, y_shard is this rank's rows of the block output of
 * Eq. 2 (the out-projection of all ranks, the bias and the residual). */
size_t pblock_rs_out_proj_workspace_bytes(const pb_config* cfg, int tp,
                                          int shards_per_launch);
pb_status pblock_rs_out_proj(const pb_config* cfg, int tp, int rank,
                             const void* c, const void* w_out, void* partial,
                             void* const* dst, int shards_per_launch, void* ws,
                             size_t ws_bytes, hipStream_t stream, int n_comm,
                             const hipStream_t* comm_streams,
                             pb_tp_context* ctx);

/* The backward's mirror of the forward's all-gather: the column-parallel
 * in-projection leaves every rank a partial sum of the LayerNorm output's
 * gradient, dh_r = dZ_r W_in,r (dZ_r, W_in,r: its own columns of dZ and
 * rows of W_in), and a reduce-scatter leaves rank j the sum of its own rows
 * (the sequence-parallel dh that the LayerNorm backward of its shard needs).
 * pblock_rs_dh computes dh_r = dz [T, N_in] w_in [N_in, H] into partial
 * [T, H] (activation dtype) in row chunks and sends them to dst exactly as
 * pblock_rs_out_proj does; the receiving side is pblock_rs_reduce with
 * x_shard = b_out = NULL.  Requirements, ws (pblock_rs_dh_workspace_bytes)
 * and ctx as for pblock_rs_out_proj. */
size_t pblock_rs_dh_workspace_bytes(const pb_config* cfg, int tp,
                                    int shards_per_launch);
pb_status pblock_rs_dh(const pb_config* cfg, int tp, int rank, const void* dz,
                       const void* w_in, void* partial, void* const* dst,
                       int shards_per_launch, void* ws, size_t ws_bytes,
                       hipStream_t stream, int n_comm,
                       const hipStream_t* comm_streams, pb_tp_context* ctx);
pb_status pblock_rs_reduce(const pb_config* cfg, int tp,
                           const void* const* parts, const void* x_shard,
                           const void* b_out, void* y_shard,
                           hipStream_t stream);

/* ------------------------------------------------------------- LAMB step
 * One step of the LAMB optimizer the paper trains with (Section 3.1, "LAMB
 * optimizer"; the layer-wise method of You et al., 2020) over up to
 * PB_LAMB_MAX_TENSORS tensors, each its own trust-ratio "layer".  For each
 * tensor, with t = cfg->step:
 *
 *   g  = grad_scale * grad
 *   m  = beta1 m + (1 - beta1) g,   v = beta2 v + (1 - beta2) g^2
 *   u  = (m / c1) / (sqrt(v / c2) + eps) + weight_decay * w
 *        c1 = 1 - beta1^t, c2 = 1 - beta2^t (1 and 1 when bias_correction = 0)
 *   r  = ||w|| / ||u|| over the whole tensor (1 if either norm is 0)
 *   w  = w - lr * r * u
 *
 * param, exp_avg (m) and exp_avg_sq (v) are fp32 and updated in place; grad
 * is fp32 (as pblock_backward writes it).  param_copy, when not NULL,
 * receives the updated weights in copy_dtype (bf16: round to nearest even),
 * e.g. the block's bf16 parameters.  Every pointer is device memory, 16-byte
 * aligned; the five arrays of a tensor must not overlap.  trust_ratio, when
 * not NULL, is a device array of n_tensors floats that receives r.
 * Tensors with numel = 0 are allowed (nothing is touched).  More tensors:
 * call again; tensors are independent, so the result is the same.
 *
 * ws must hold pblock_lamb_workspace_bytes(n_tensors, tensors) bytes (per-
 * chunk partial norms and the ratios).  Asynchronous on the stream; the
 * result does not depend on timing (fixed reduction order, no atomics).
 * Errors: PB_ERR_INVALID_ARG for a bad config (lr or grad_scale not finite,
 * beta outside [0, 1), eps <= 0, step < 1, negative or non-finite decay,
 * n_tensors outside 1..16), a NULL or misaligned pointer, or too many
 * elements; PB_ERR_WORKSPACE for a small ws. */
#define PB_LAMB_MAX_TENSORS 16
typedef struct {
  float lr;
  float beta1, beta2;
  float eps;
  float grad_scale;
  int step;            /* t >= 1 */
  int bias_correction; /* 0 or 1 */
} pb_lamb_config;
typedef struct {
  float* param;        /* [numel] fp32 master weights */
  const float* grad;   /* [numel] fp32 */
  float* exp_avg;      /* [numel] fp32 */
  float* exp_avg_sq;   /* [numel] fp32 */
  void* param_copy;    /* NULL or [numel] in copy_dtype */
  size_t numel;
  float weight_decay;  /* lambda of this tensor (0 for biases and norms, say) */
} pb_lamb_tensor;
size_t pblock_lamb_workspace_bytes(int n_tensors, const pb_lamb_tensor* tensors);
pb_status pblock_lamb_step(const pb_lamb_config* cfg, int n_tensors,
                           const pb_lamb_tensor* tensors, pb_dtype copy_dtype,
                           float* trust_ratio, void* ws, size_t ws_bytes,
                           hipStream_t stream);


/* Human-readable name of a status, and a description of the most recent
 * failed check on the calling thread ("" if none). */
const char* pblock_status_string(pb_status status);
const char* pblock_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PBLOCK_H */
