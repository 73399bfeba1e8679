// Host-side launchers of the block's kernels.  Each returns nothing; the
// caller checks hipGetLastError() after its launch sequence.  Shapes are
// validated by the C-ABI layer before any launcher runs.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

namespace pb {

enum class Dt { BF16, F32 };

// ---------------------------------------------------------------- LayerNorm
// h = gamma * (x - mean) * rstd + beta per row of x [rows, H].
void launch_ln_forward(Dt dt, const void* x, const void* gamma, const void* beta, void* h,
                       float* mean, float* rstd, int rows, int H, float eps, hipStream_t s);
// dx = dy + rstd * (g - mean(g) - xhat * mean(g * xhat)), g = gamma * dh, per
// row, given the row terms sum g and sum g xhat as 64-column group partials
// rowpart [rows, ln_row_groups(H)] (written by the dh GEMM's LnGrad
// epilogue).  Column-parallel: workgroups of 16 rows x 2048 columns; partial
// column sums of dh * xhat, dh and dy per 16-row chunk go to part_dgamma,
// part_dbeta and part_dy [ln_backward_chunks(rows), H].
int ln_backward_chunks(int rows);
void launch_ln_backward(Dt dt, const void* x, const float* mean, const float* rstd,
                        const void* gamma, const void* dh, const float2* rowpart,
                        const void* dy, void* dx, float* part_dgamma, float* part_dbeta,
                        float* part_dy, int rows, int H, hipStream_t s);

// ------------------------------------------------------------ column sums
// out[c] = sum over r of src[r * ld + c] for a [rows, cols] matrix (cols a
// multiple of 8).  Deterministic two-stage reduction through part, which holds
// colsum_partial_floats(rows, cols) floats.
size_t colsum_partial_floats(int rows, int cols);
void launch_colsum(Dt dt, const void* src, int ld, int rows, int cols, float* part, float* out,
                   hipStream_t s);
void launch_colsum_f32(const float* src, int ld, int rows, int cols, float* part, float* out,
                       hipStream_t s);
// Three fp32 [rows, cols] arrays at once (same ld; cols a multiple of 4), in
// one launch and without a partial buffer: for the few hundred rows of the
// LayerNorm backward's per-chunk partial sums.
void launch_colsum3_f32(const float* a, const float* b, const float* c, int ld, int rows,
                        int cols, float* out_a, float* out_b, float* out_c, hipStream_t s);

// -------------------------------------------------------------- LAMB step
// One LAMB step over up to kLambMaxTensors fp32 tensors, each with its own
// trust ratio.  Elements are processed in chunks of kLambChunk per
// workgroup.  Tensor i owns chunks [chunk0[i], chunk_end[i]); chunk0[i] is a
// multiple of kLambGroup (chunks up to the next boundary are padding) and
// chunk0[n] is the padded total.
constexpr int kLambMaxTensors = 16;
constexpr int kLambChunk = 1024;
constexpr int kLambGroup = 256;
struct LambTable {
  float* w[kLambMaxTensors];
  const float* g[kLambMaxTensors];
  float* m[kLambMaxTensors];
  float* v[kLambMaxTensors];
  void* copy[kLambMaxTensors];  // nullptr: no copy of this tensor
  long long numel[kLambMaxTensors];
  float wd[kLambMaxTensors];
  int chunk0[kLambMaxTensors + 1];
  int chunk_end[kLambMaxTensors];
  int n;
};
struct LambScalars {
  float lr, beta1, beta2, eps, grad_scale;
  float c1, c2;  // 1 / (1 - beta^t), or 1 without bias correction
};
int lamb_chunks(long long numel);
int lamb_padded_chunks(long long numel);  // rounded up to a multiple of kLambGroup
// partial: chunk0[n] float2; group: chunk0[n] / kLambGroup double2; ratio:
// n floats (all workspace); ratio_out: n floats or nullptr.
void launch_lamb(const LambTable& t, const LambScalars& sc, Dt copy_dt, float2* partial,
                 double2* group, float* ratio, float* ratio_out, hipStream_t s);

// ------------------------------------------------------ reduce-scatter sum
// y = x + bias + sum over q < n of parts[q], row-major [rows, H] (H a
// multiple of 8), summed in fp32 in the order of q.
constexpr int kRsMaxParts = 64;
struct RsParts {
  const void* p[kRsMaxParts];
  int n;
};
void launch_rs_reduce(Dt dt, const RsParts& parts, const void* x, const void* bias, void* y,
                      int rows, int H, hipStream_t s);

// ------------------------------------------------------------------ GEMMs
// C[m, n] = sum_k A(m, k) B(k, n), fp32 accumulation.
// A(m, k) is A[m * lda + k] when a_kcontig, else A[k * lda + m]; B(k, n) is
// B[n * ldb + k] when b_kcontig, else B[k * ldb + n].
enum class Epi {
  StoreF32,    // out_f32[m * ld_out + n] = acc
  BiasGelu,    // z = acc + bias[n] -> out[m * ld_out + n]; for n >= split also
               // gelu(z) -> out2[m * ld_out2 + (n - split) + col2]
  BiasResid,   // out[m * ld_out + n] = acc + bias[n] + resid[m * ld_out + n]
  DgeluSplit,  // n < split: out[m * ld_out + n] = acc;
               // n >= split: with c = n - split + col2,
               //   out2[m * ld_out2 + c] = acc * gelu'(aux[m * ld_out2 + c])
  LnGrad,      // out[m * ld_out + n] = acc (= dh, activation type), and the LayerNorm
               // backward's row terms per 64-column group g = n / 64:
               //   rowpart[m * rowpart_ld + g] = (sum gamma dh, sum gamma dh xhat)
               // with gamma = bias[n], xhat = (aux[m * ld_out + n] - mean[m]) rstd[m]
};
struct EpiArgs {
  void* out = nullptr;
  int ld_out = 0;
  void* out2 = nullptr;
  int ld_out2 = 0;
  const void* bias = nullptr;
  const void* resid = nullptr;
  const void* aux = nullptr;
  int split = 0;
  int col2 = 0;
  int gelu_tanh = 1;
  const float* mean = nullptr;  // LnGrad only
  const float* rstd = nullptr;
  float2* rowpart = nullptr;
  int rowpart_ld = 0;
  // DgeluSplit, LDS-staged path only (launch_gemm_pair): when delta is set,
  // also delta[(b heads + h) seq + t] = sum over head h's columns of
  // out[m, n] o_rows[m * ld_o_rows + n] for m = b seq + t, n < split, with
  // out rounded to the activation type first; head_dim 64 or 128, split and
  // the tile's column blocks aligned to heads.
  const void* o_rows = nullptr;
  int ld_o_rows = 0;
  float* delta = nullptr;
  int delta_seq = 0, delta_heads = 0, delta_hd = 0;
  // StoreF32 as the second GEMM of launch_gemm_pair only: when set, also
  // rowsum[m] = sum over k of A(m, k) (fp32), for every row m < M.
  float* rowsum = nullptr;
};
// 64-column groups of the LnGrad row terms for a row of n columns.
inline int ln_row_groups(int n) { return (n + 63) / 64; }
// Tail split: the first n_full tiles (a whole number of 256-tile waves) are
// computed whole; each of the last `tail` tiles is split into `splits`
// K-slices whose fp32 partial tiles go to a workspace and are summed in slice
// order by a second kernel that applies the epilogue.  Only for the bf16
// LDS-DMA path (K a multiple of 64); {tiles, 0, 1} means no split.
struct SplitPlan {
  int n_full, tail, splits;
};
SplitPlan gemm_split_plan(Dt dt, int M, int N, int K);
size_t gemm_split_floats(const SplitPlan& p);
// The launch of one GEMM given a full split workspace, as launch_gemm makes
// it for operands whose LDS-DMA offsets fit 32 bits: output tiles, the tail
// split, and the main kernel's grid.
struct GemmLaunch {
  int tiles;
  SplitPlan plan;
  int workgroups, threads;
};
GemmLaunch gemm_launch_of(Dt dt, int M, int N, int K);
// split_ws may be NULL (or too small): the GEMM then runs unsplit.
void launch_gemm(Dt dt, Epi epi, bool a_kcontig, bool b_kcontig, const void* A, int lda,
                 const void* B, int ldb, int M, int N, int K, const EpiArgs& ep, float* split_ws,
                 size_t split_ws_floats, hipStream_t s);

// Two independent GEMMs in one launch, neither split along K: the first
// one's tiles are started first (give it the longer K), and the second one's
// tiles fill the CUs the first leaves idle.  Supported: bf16, K multiples of
// 64 and operands the LDS-DMA path takes, with the first GEMM A K-contiguous,
// B MN-contiguous and a DgeluSplit or LnGrad epilogue, the second both
// MN-contiguous with StoreF32 (the backward pass's dC + dW_out and
// dh + dW_in).  launch_gemm_pair launches nothing and returns false for any
// other pair.
struct GemmSpec {
  Epi epi;
  bool a_kcontig, b_kcontig;
  const void* A;
  int lda;
  const void* B;
  int ldb;
  int M, N, K;
  EpiArgs ep;
};
//
// With queue non-NULL the launch is persistent: one workgroup per CU takes
// tiles from per-XCD queues until none is left, so XCDs that run slower hand
// their last tiles to the others.  queue points to kQueueInts ints (device
// memory) that must be zero when the launch runs, e.g. from
// launch_queue_reset earlier on the same stream; the launch leaves them
// non-zero, and two launches in flight at once need separate queues.  The
// results are the same bits either way.
constexpr int kQueueInts = 8;
void launch_queue_reset(int* queue, int n, hipStream_t s);  // n ints = 0 (a kernel)
bool gemm_pair_supported(Dt dt, const GemmSpec& g1, const GemmSpec& g2);
bool launch_gemm_pair(Dt dt, const GemmSpec& g1, const GemmSpec& g2, int* queue, hipStream_t s);

// -------------------------------------------------------------- attention
// Causal sliding-window attention over [batch, seq] rows; q/k/v/o/do/dq/dk/dv
// element (b, t, head, e) at ptr[(b * seq + t) * ld + head * head_dim + e].
struct AttnShape {
  int batch, seq, heads, head_dim, window;
};

// Work split of the bf16 attention kernels.  Each workgroup owns a block of 64
// queries (forward, dQ) or 64 keys (dK/dV) and walks tiles of the other axis.
// When there are too few blocks to fill the chip, a block's tile range is cut
// into chunks of at most *_chunk tiles handled by separate workgroups; those
// write fp32 partial results that a combine kernel merges in chunk order, so
// results stay deterministic.  *_n is the chunk count of the longest block
// (1: unsplit).
struct AttnSplit {
  int fwd_chunk, fwd_n;  // forward and dQ: key tiles of 64
  int kv_chunk, kv_n;    // dK/dV: query tiles of 32
};
AttnSplit attn_split_plan(Dt dt, const AttnShape& a);
// The backward's plan: both backward roles run in one launch, so it splits
// only when their blocks together are too few for the chip.
AttnSplit attn_bwd_split_plan(Dt dt, const AttnShape& a);
// Bytes of partial results the split forward / backward needs (0: unsplit).
size_t attn_fwd_partial_bytes(const AttnShape& a, const AttnSplit& p);
size_t attn_bwd_partial_bytes(const AttnShape& a, const AttnSplit& p);

// O = softmax(Q K^T / sqrt(d), sliding-window causal mask) V per head; lse
// [batch, heads, seq] is the natural-log row log-sum-exp.  part may be NULL;
// the split plan is used only when part_bytes >= attn_fwd_partial_bytes.
void launch_attn_forward(Dt dt, const AttnShape& a, const void* q, const void* k, const void* v,
                         int ld_qkv, void* o, int ld_o, float* lse, void* part,
                         size_t part_bytes, hipStream_t s);
// delta[b, head, t] = sum_e do * o (softmax row term of the backward pass),
// formed here unless delta_ready (the caller has already written it).
// o uses ld_o, d_o uses ld_do; delta holds batch*heads*seq floats.  part as
// for the forward, against attn_bwd_partial_bytes.
void launch_attn_backward(Dt dt, const AttnShape& a, const void* q, const void* k, const void* v,
                          int ld_qkv, const void* o, int ld_o, const void* d_o, int ld_do,
                          const float* lse, float* delta, bool delta_ready, void* dq, void* dk,
                          void* dv, int ld_d, void* part, size_t part_bytes, hipStream_t s);

}  // namespace pb
