// C ABI of the parallel transformer block library: argument checks (host
// only, before any HIP call), stash / workspace layout, and the kernel
// sequence of the forward and backward passes on the caller's stream.
#include "pblock.h"

#include <math.h>

#include <cmath>

#include <algorithm>
#include <array>
#include <atomic>
#include <initializer_list>
#include <mutex>
#include <new>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "kernels.h"

namespace {

thread_local char g_err[512] = "";

pb_status fail(pb_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return st;
}

// Records the caller's step events (the *_timed entry points) around the
// launches of one step; ev may be NULL.
struct StepScope {
  const pb_step_events* ev;
  int step;
  hipStream_t s;
  StepScope(const pb_step_events* e, pb_step st, hipStream_t stream) : ev(e), step(st), s(stream) {
    if (ev && ev->begin[step]) (void)hipEventRecord(ev->begin[step], s);
  }
  ~StepScope() {
    if (ev && ev->end[step]) (void)hipEventRecord(ev->end[step], s);
  }
};

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

struct Dims {
  long long T, H, A, F, N_in, K_out, heads, d, B, S, W;
  size_t esz;  // bytes per activation element
};

Dims dims_of(const pb_config* c) {
  Dims d;
  d.B = c->batch;
  d.S = c->seq;
  d.T = (long long)c->batch * c->seq;
  d.H = c->hidden;
  d.heads = c->heads;
  d.d = c->head_dim;
  d.A = (long long)c->heads * c->head_dim;
  d.F = c->ffn;
  d.N_in = 3 * d.A + d.F;
  d.K_out = d.A + d.F;
  d.W = c->window;
  d.esz = c->dtype == PB_BF16 ? 2 : 4;
  return d;
}

constexpr long long kMaxInt = 2147483647LL;

pb_status check_config(const pb_config* c) {
  if (!c) return fail(PB_ERR_INVALID_ARG, "cfg is NULL");
  if (c->dtype != PB_BF16 && c->dtype != PB_F32)
    return fail(PB_ERR_INVALID_ARG, "dtype %d is neither PB_BF16 nor PB_F32", (int)c->dtype);
  if (c->batch < 1 || c->seq < 1 || c->heads < 1 || c->window < 1)
    return fail(PB_ERR_INVALID_ARG, "batch, seq, heads and window must be >= 1");
  if (c->hidden < 8 || c->hidden % 8)
    return fail(PB_ERR_INVALID_ARG, "hidden=%d must be a positive multiple of 8", c->hidden);
  if (c->hidden > 32768)
    return fail(PB_ERR_UNSUPPORTED, "hidden=%d > 32768 (LayerNorm keeps a row in registers)",
                c->hidden);
  if (c->ffn < 8 || c->ffn % 8)
    return fail(PB_ERR_INVALID_ARG, "ffn=%d must be a positive multiple of 8", c->ffn);
  if (c->head_dim != 64 && c->head_dim != 96 && c->head_dim != 128)
    return fail(PB_ERR_UNSUPPORTED, "head_dim=%d: kernels exist for 64, 96 and 128", c->head_dim);
  if (!(c->ln_eps > 0.f) || !isfinite(c->ln_eps))
    return fail(PB_ERR_INVALID_ARG, "ln_eps must be finite and > 0");
  if (c->gelu_tanh != 0 && c->gelu_tanh != 1)
    return fail(PB_ERR_INVALID_ARG, "gelu_tanh must be 0 or 1");
  if (c->heads > 65535 || c->batch > 65535)
    return fail(PB_ERR_UNSUPPORTED, "heads and batch must be <= 65535 (grid limits)");
  const Dims d = dims_of(c);
  if (d.T * d.heads > kMaxInt || d.N_in > kMaxInt / 4 || d.T > kMaxInt / 4)
    return fail(PB_ERR_UNSUPPORTED, "problem too large for 32-bit row/column indices");
  return PB_OK;
}

pb::AttnShape attn_shape(const Dims& d) {
  pb::AttnShape a;
  a.batch = (int)d.B;
  a.seq = (int)d.S;
  a.heads = (int)d.heads;
  a.head_dim = (int)d.d;
  // a window of at least seq keys is full causal attention; clamping keeps
  // the kernels' index arithmetic within int range
  a.window = (int)(d.W < d.S ? d.W : d.S);
  return a;
}

struct SavedLayout {
  size_t off[6];  // h, z, c, mean, rstd, lse
  size_t total;
};
SavedLayout saved_layout(const Dims& d) {
  SavedLayout L;
  size_t o = 0;
  const size_t sizes[6] = {(size_t)(d.T * d.H) * d.esz, (size_t)(d.T * d.N_in) * d.esz,
                           (size_t)(d.T * d.K_out) * d.esz, (size_t)d.T * 4, (size_t)d.T * 4,
                           (size_t)(d.B * d.heads * d.S) * 4};
  for (int i = 0; i < 6; ++i) {
    L.off[i] = o;
    o = align256(o + sizes[i]);
  }
  L.total = o;
  return L;
}

// Optional space for split work: the GEMMs' tail-split partial tiles and the
// attention kernels' chunk partials.  They are never live at the same time,
// so one region serves both.
size_t split_bytes_fwd(const Dims& d, pb::Dt dt) {
  const int T = (int)d.T, H = (int)d.H, N_in = (int)d.N_in, K_out = (int)d.K_out;
  size_t m = std::max(pb::gemm_split_floats(pb::gemm_split_plan(dt, T, N_in, H)),
                      pb::gemm_split_floats(pb::gemm_split_plan(dt, T, H, K_out))) * 4;
  const pb::AttnShape a = attn_shape(d);
  return std::max(m, pb::attn_fwd_partial_bytes(a, pb::attn_split_plan(dt, a)));
}
size_t split_bytes_bwd(const Dims& d, pb::Dt dt) {
  const int T = (int)d.T, H = (int)d.H, N_in = (int)d.N_in, K_out = (int)d.K_out;
  size_t m = pb::gemm_split_floats(pb::gemm_split_plan(dt, T, K_out, H));
  m = std::max(m, pb::gemm_split_floats(pb::gemm_split_plan(dt, H, K_out, T)));
  m = std::max(m, pb::gemm_split_floats(pb::gemm_split_plan(dt, T, H, N_in)));
  m = std::max(m, pb::gemm_split_floats(pb::gemm_split_plan(dt, N_in, H, T)));
  const pb::AttnShape a = attn_shape(d);
  return std::max(m * 4, pb::attn_bwd_partial_bytes(a, pb::attn_bwd_split_plan(dt, a)));
}

// Queue heads of the backward's persistent GEMM launches: kQueueInts ints per
// launch, zeroed at the start of each call.
constexpr int kBwdQueueSets = 4;
constexpr size_t kBwdQueueBytes = kBwdQueueSets * pb::kQueueInts * sizeof(int);

struct BwdLayout {
  size_t d_o, dz, dh, delta, rowpart, pdg, pdb, pdy, part, queue, split, base, total;
};
BwdLayout bwd_layout(const Dims& d) {
  BwdLayout L;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align256(o + bytes);
    return at;
  };
  const int nblk = pb::ln_backward_chunks((int)d.T);
  L.d_o = take((size_t)(d.T * d.A) * d.esz);
  L.dz = take((size_t)(d.T * d.N_in) * d.esz);
  L.dh = take((size_t)(d.T * d.H) * d.esz);
  L.delta = take((size_t)(d.B * d.heads * d.S) * 4);
  L.rowpart = take((size_t)d.T * pb::ln_row_groups((int)d.H) * sizeof(float2));
  L.pdg = take((size_t)nblk * d.H * 4);
  L.pdb = take((size_t)nblk * d.H * 4);
  L.pdy = take((size_t)nblk * d.H * 4);
  size_t part = pb::colsum_partial_floats((int)d.T, (int)d.H);
  size_t p2 = pb::colsum_partial_floats((int)d.T, (int)d.N_in);
  size_t p3 = pb::colsum_partial_floats(nblk, (int)d.H);
  if (p2 > part) part = p2;
  if (p3 > part) part = p3;
  L.part = take(part * 4);
  L.queue = take(kBwdQueueBytes);
  L.base = o;  // required; the tail-split region after it is optional
  L.split = take(split_bytes_bwd(d, d.esz == 2 ? pb::Dt::BF16 : pb::Dt::F32));
  L.total = o;
  return L;
}

// ------------------------------------------------------------ serial block
// Stash of the serial block: h1, Z (Q|K|V|U), C (O|G), mean1, rstd1, lse,
// x1, h2, mean2, rstd2.
struct SerialLayout {
  size_t off[10];
  size_t total;
};
SerialLayout serial_layout(const Dims& d) {
  SerialLayout L;
  size_t o = 0;
  const size_t th = (size_t)(d.T * d.H) * d.esz;
  const size_t sizes[10] = {th, (size_t)(d.T * d.N_in) * d.esz, (size_t)(d.T * d.K_out) * d.esz,
                            (size_t)d.T * 4, (size_t)d.T * 4, (size_t)(d.B * d.heads * d.S) * 4,
                            th, th, (size_t)d.T * 4, (size_t)d.T * 4};
  for (int i = 0; i < 10; ++i) {
    L.off[i] = o;
    o = align256(o + sizes[i]);
  }
  L.total = o;
  return L;
}

// Largest tail-split space among a list of GEMM shapes (M, N, K).
size_t max_split_bytes(pb::Dt dt, std::initializer_list<std::array<int, 3>> shapes) {
  size_t m = 0;
  for (const auto& s : shapes)
    m = std::max(m, pb::gemm_split_floats(pb::gemm_split_plan(dt, s[0], s[1], s[2])) * 4);
  return m;
}
size_t serial_split_fwd(const Dims& d, pb::Dt dt) {
  const int T = (int)d.T, H = (int)d.H, A = (int)d.A, F = (int)d.F;
  size_t m = max_split_bytes(dt, {{T, 3 * A, H}, {T, H, A}, {T, F, H}, {T, H, F}});
  const pb::AttnShape a = attn_shape(d);
  return std::max(m, pb::attn_fwd_partial_bytes(a, pb::attn_split_plan(dt, a)));
}
size_t serial_split_bwd(const Dims& d, pb::Dt dt) {
  const int T = (int)d.T, H = (int)d.H, A = (int)d.A, F = (int)d.F;
  size_t m = max_split_bytes(dt, {{T, F, H}, {H, F, T}, {T, H, F}, {F, H, T}, {T, A, H},
                                  {H, A, T}, {T, H, 3 * A}, {3 * A, H, T}});
  const pb::AttnShape a = attn_shape(d);
  return std::max(m, pb::attn_bwd_partial_bytes(a, pb::attn_bwd_split_plan(dt, a)));
}

// Backward workspace of the serial block: dO, dZ, dh (activation type, shared by both
// LayerNorms), dx1, softmax row terms, LN row terms, LN partial column sums,
// column-sum scratch, then the optional split region.
struct SerialBwdLayout {
  size_t d_o, dz, dh, dx1, delta, rowpart, pdg, pdb, pdy, part, queue, split, base, total;
};
SerialBwdLayout serial_bwd_layout(const Dims& d) {
  SerialBwdLayout L;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align256(o + bytes);
    return at;
  };
  const int nblk = pb::ln_backward_chunks((int)d.T);
  L.d_o = take((size_t)(d.T * d.A) * d.esz);
  L.dz = take((size_t)(d.T * d.N_in) * d.esz);
  L.dh = take((size_t)(d.T * d.H) * d.esz);
  L.dx1 = take((size_t)(d.T * d.H) * d.esz);
  L.delta = take((size_t)(d.B * d.heads * d.S) * 4);
  L.rowpart = take((size_t)d.T * pb::ln_row_groups((int)d.H) * sizeof(float2));
  L.pdg = take((size_t)nblk * d.H * 4);
  L.pdb = take((size_t)nblk * d.H * 4);
  L.pdy = take((size_t)nblk * d.H * 4);
  size_t part = pb::colsum_partial_floats((int)d.T, (int)d.N_in);
  part = std::max(part, pb::colsum_partial_floats(nblk, (int)d.H));
  L.part = take(part * 4);
  L.queue = take(kBwdQueueBytes);
  L.base = o;
  L.split = take(serial_split_bwd(d, d.esz == 2 ? pb::Dt::BF16 : pb::Dt::F32));
  L.total = o;
  return L;
}

pb_status check_ptr(const void* p, const char* name) {
  if (!p) return fail(PB_ERR_INVALID_ARG, "%s is NULL", name);
  if ((uintptr_t)p % 16) return fail(PB_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return PB_OK;
}

#define PB_CHECK(expr)             \
  do {                             \
    pb_status _st = (expr);        \
    if (_st != PB_OK) return _st;  \
  } while (0)

pb_status finish_launches() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(PB_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  g_err[0] = '\0';
  return PB_OK;
}

pb::Dt dt_of(const pb_config* c) { return c->dtype == PB_BF16 ? pb::Dt::BF16 : pb::Dt::F32; }

// Element offset helper for activation buffers.
const void* at(const void* base, long long elems, size_t esz) {
  return (const char*)base + (size_t)elems * esz;
}
void* at(void* base, long long elems, size_t esz) { return (char*)base + (size_t)elems * esz; }

pb_status check_attn_config(const pb_config* c) {
  if (!c) return fail(PB_ERR_INVALID_ARG, "cfg is NULL");
  if (c->dtype != PB_BF16 && c->dtype != PB_F32)
    return fail(PB_ERR_INVALID_ARG, "dtype %d is neither PB_BF16 nor PB_F32", (int)c->dtype);
  if (c->batch < 1 || c->seq < 1 || c->heads < 1 || c->window < 1)
    return fail(PB_ERR_INVALID_ARG, "batch, seq, heads and window must be >= 1");
  if (c->head_dim != 64 && c->head_dim != 96 && c->head_dim != 128)
    return fail(PB_ERR_UNSUPPORTED, "head_dim=%d: kernels exist for 64, 96 and 128", c->head_dim);
  if (c->heads > 65535 || c->batch > 65535)
    return fail(PB_ERR_UNSUPPORTED, "heads and batch must be <= 65535 (grid limits)");
  if ((long long)c->batch * c->seq * c->heads > kMaxInt)
    return fail(PB_ERR_UNSUPPORTED, "batch*seq*heads exceeds 32-bit indexing");
  return PB_OK;
}

size_t swattn_delta_bytes(const pb_config* c) {
  return align256((size_t)c->batch * c->heads * c->seq * 4);
}

pb_status check_ld(int ld, const pb_config* c, const char* name) {
  if (ld < (long long)c->heads * c->head_dim || ld % 8)
    return fail(PB_ERR_INVALID_ARG, "%s=%d must be >= heads*head_dim and a multiple of 8", name,
                ld);
  return PB_OK;
}

}  // namespace

extern "C" {

pb_status pblock_validate(const pb_config* cfg) {
  pb_status st = check_config(cfg);
  if (st == PB_OK) g_err[0] = '\0';
  return st;
}

size_t pblock_saved_bytes(const pb_config* cfg) {
  if (check_config(cfg) != PB_OK) return 0;
  return saved_layout(dims_of(cfg)).total;
}

pb_status pblock_saved_offsets(const pb_config* cfg, size_t* offsets) {
  PB_CHECK(check_config(cfg));
  if (!offsets) return fail(PB_ERR_INVALID_ARG, "offsets is NULL");
  const SavedLayout L = saved_layout(dims_of(cfg));
  for (int i = 0; i < 6; ++i) offsets[i] = L.off[i];
  return PB_OK;
}

size_t pblock_workspace_bytes(const pb_config* cfg, int mode) {
  if (check_config(cfg) != PB_OK) return 0;
  const Dims d = dims_of(cfg);
  const size_t split = align256(split_bytes_fwd(d, dt_of(cfg)));
  switch (mode) {
    case PB_WS_FORWARD_WITH_STASH: return saved_layout(d).total + split;
    case PB_WS_BACKWARD: return bwd_layout(d).total;
    case PB_WS_FORWARD: return split;
    default: return 0;
  }
}

pb_status pblock_workspace_offsets(const pb_config* cfg, size_t* offsets) {
  PB_CHECK(check_config(cfg));
  if (!offsets) return fail(PB_ERR_INVALID_ARG, "offsets is NULL");
  const BwdLayout W = bwd_layout(dims_of(cfg));
  offsets[0] = W.d_o;
  offsets[1] = W.dz;
  offsets[2] = W.dh;
  offsets[3] = W.delta;
  return PB_OK;
}

pb_status pblock_forward(const pb_config* cfg, const void* x, const void* ln_gamma,
                         const void* ln_beta, const void* w_in, const void* b_in,
                         const void* w_out, const void* b_out, void* y, void* saved, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  return pblock_forward_timed(cfg, x, ln_gamma, ln_beta, w_in, b_in, w_out, b_out, y, saved, ws,
                              ws_bytes, stream, nullptr);
}

pb_status pblock_forward_timed(const pb_config* cfg, const void* x, const void* ln_gamma,
                               const void* ln_beta, const void* w_in, const void* b_in,
                               const void* w_out, const void* b_out, void* y, void* saved,
                               void* ws, size_t ws_bytes, hipStream_t stream,
                               const pb_step_events* step_ev) {
  PB_CHECK(check_config(cfg));
  PB_CHECK(check_ptr(x, "x"));
  PB_CHECK(check_ptr(ln_gamma, "ln_gamma"));
  PB_CHECK(check_ptr(ln_beta, "ln_beta"));
  PB_CHECK(check_ptr(w_in, "w_in"));
  PB_CHECK(check_ptr(b_in, "b_in"));
  PB_CHECK(check_ptr(w_out, "w_out"));
  PB_CHECK(check_ptr(b_out, "b_out"));
  PB_CHECK(check_ptr(y, "y"));
  const Dims d = dims_of(cfg);
  const SavedLayout L = saved_layout(d);
  const pb::Dt dt = dt_of(cfg);
  void* stash = saved;
  char* split_base = (char*)ws;
  size_t split_bytes = ws ? ws_bytes : 0;
  if (stash) {
    PB_CHECK(check_ptr(stash, "saved"));
    if (ws) PB_CHECK(check_ptr(ws, "ws"));
  } else {
    PB_CHECK(check_ptr(ws, "ws (needed when saved is NULL)"));
    if (ws_bytes < L.total)
      return fail(PB_ERR_WORKSPACE, "ws_bytes=%zu < %zu needed to hold the stash", ws_bytes,
                  L.total);
    stash = ws;
    split_base = (char*)ws + L.total;
    split_bytes = ws_bytes - L.total;
  }
  float* split_ws = (float*)split_base;
  const size_t split_f = split_bytes / 4;
  const size_t e = d.esz;
  char* sb = (char*)stash;
  void* h = sb + L.off[0];
  void* z = sb + L.off[1];
  void* c = sb + L.off[2];
  float* mean = (float*)(sb + L.off[3]);
  float* rstd = (float*)(sb + L.off[4]);
  float* lse = (float*)(sb + L.off[5]);
  const int T = (int)d.T, H = (int)d.H, A = (int)d.A, N_in = (int)d.N_in, K_out = (int)d.K_out;

  // F1: shared LayerNorm
  {
    StepScope sc(step_ev, PB_STEP_LN_FWD, stream);
    pb::launch_ln_forward(dt, x, ln_gamma, ln_beta, h, mean, rstd, T, H, cfg->ln_eps, stream);
  }
  // F2: Z = h W_in^T + b_in (Q | K | V | U); G = gelu(U) -> C[:, A:]
  pb::EpiArgs e1;
  e1.out = z;
  e1.ld_out = N_in;
  e1.out2 = c;
  e1.ld_out2 = K_out;
  e1.bias = b_in;
  e1.split = 3 * A;
  e1.col2 = A;
  e1.gelu_tanh = cfg->gelu_tanh;
  {
    StepScope sc(step_ev, PB_STEP_IN_PROJ, stream);
    pb::launch_gemm(dt, pb::Epi::BiasGelu, true, true, h, H, w_in, H, T, N_in, H, e1, split_ws,
                    split_f, stream);
  }
  // F3: sliding-window attention, O -> C[:, :A]
  {
    StepScope sc(step_ev, PB_STEP_ATTN_FWD, stream);
    pb::launch_attn_forward(dt, attn_shape(d), z, at(z, A, e), at(z, 2LL * A, e), N_in, c, K_out,
                            lse, split_base, split_bytes, stream);
  }
  // F5: y = x + C W_out^T + b_out (both branches and the residual of Eq. 2)
  pb::EpiArgs e2;
  e2.out = y;
  e2.ld_out = H;
  e2.bias = b_out;
  e2.resid = x;
  {
    StepScope sc(step_ev, PB_STEP_OUT_PROJ, stream);
    pb::launch_gemm(dt, pb::Epi::BiasResid, true, true, c, K_out, w_out, K_out, T, H, K_out, e2,
                    split_ws, split_f, stream);
  }
  return finish_launches();
}

namespace {
// The GEMMs of the backward passes that may share a launch, built in one
// place for the launches and for pblock_backward_pairs, so that the query
// reports the pairing the launches make.  Null operands and default epilogue
// arguments describe the shapes alone.
struct ParallelBwdGemms {
  pb::GemmSpec dc, dw_out, dh, dw_in;
};
ParallelBwdGemms parallel_bwd_gemms(const Dims& d, const void* dy, const void* w_out,
                                    const void* c, const void* dz, const void* w_in,
                                    const void* h, const pb::EpiArgs& e_dc,
                                    const pb::EpiArgs& e_dwo, const pb::EpiArgs& e_dh,
                                    const pb::EpiArgs& e_dwi) {
  const int T = (int)d.T, H = (int)d.H, N_in = (int)d.N_in, K_out = (int)d.K_out;
  return {
      // dC = dy W_out (B MN-contiguous)
      {pb::Epi::DgeluSplit, true, false, dy, H, w_out, K_out, T, K_out, H, e_dc},
      // dW_out = dy^T C (contraction over tokens)
      {pb::Epi::StoreF32, false, false, dy, H, c, K_out, H, K_out, T, e_dwo},
      // dh = dZ W_in
      {pb::Epi::LnGrad, true, false, dz, N_in, w_in, H, T, H, N_in, e_dh},
      // dW_in = dZ^T h
      {pb::Epi::StoreF32, false, false, dz, N_in, h, H, N_in, H, T, e_dwi}};
}

struct SerialBwdGemms {
  pb::GemmSpec dg, dw_down, dh2, dw_up, d_o, dw_o, dh1, dw_qkv;
};
struct SerialBwdOperands {
  const void *dy, *dx1, *c, *dz, *h1, *h2, *w_in, *w_out;
};
SerialBwdGemms serial_bwd_gemms(const Dims& d, const SerialBwdOperands& o,
                                const pb::EpiArgs& e_dg, const pb::EpiArgs& e_wd,
                                const pb::EpiArgs& e_dh2, const pb::EpiArgs& e_wu,
                                const pb::EpiArgs& e_do, const pb::EpiArgs& e_wo,
                                const pb::EpiArgs& e_dh1, const pb::EpiArgs& e_wq) {
  const int T = (int)d.T, H = (int)d.H, A = (int)d.A, F = (int)d.F, N_in = (int)d.N_in,
            K_out = (int)d.K_out;
  const size_t e = d.esz;
  auto off = [&](const void* p, long long n) { return p ? at(p, n, e) : nullptr; };
  return {
      // dG = dy W_down
      {pb::Epi::DgeluSplit, true, false, o.dy, H, off(o.w_out, A), K_out, T, F, H, e_dg},
      // dW_down = dy^T G
      {pb::Epi::StoreF32, false, false, o.dy, H, off(o.c, A), K_out, H, F, T, e_wd},
      // dh2 = dU W_up
      {pb::Epi::LnGrad, true, false, off(o.dz, 3LL * A), N_in, off(o.w_in, 3LL * A * H), H, T, H,
       F, e_dh2},
      // dW_up = dU^T h2
      {pb::Epi::StoreF32, false, false, off(o.dz, 3LL * A), N_in, o.h2, H, F, H, T, e_wu},
      // dO = dx1 W_o
      {pb::Epi::DgeluSplit, true, false, o.dx1, H, o.w_out, K_out, T, A, H, e_do},
      // dW_o = dx1^T O
      {pb::Epi::StoreF32, false, false, o.dx1, H, o.c, K_out, H, A, T, e_wo},
      // dh1 = dQKV W_qkv
      {pb::Epi::LnGrad, true, false, o.dz, N_in, o.w_in, H, T, H, 3 * A, e_dh1},
      // dW_qkv = dQKV^T h1
      {pb::Epi::StoreF32, false, false, o.dz, N_in, o.h1, H, 3 * A, H, T, e_wq}};
}
}  // namespace

pb_status pblock_gemm_plan(pb_dtype dtype, int M, int N, int K, pb_gemm_plan* plan) {
  if (!plan) return fail(PB_ERR_INVALID_ARG, "plan is NULL");
  if (dtype != PB_BF16 && dtype != PB_F32) return fail(PB_ERR_INVALID_ARG, "unknown dtype");
  if (M < 1 || N < 1 || K < 1) return fail(PB_ERR_INVALID_ARG, "M, N, K must be >= 1");
  const pb::Dt dt = dtype == PB_BF16 ? pb::Dt::BF16 : pb::Dt::F32;
  const pb::GemmLaunch g = pb::gemm_launch_of(dt, M, N, K);
  plan->tiles = g.tiles;
  plan->n_full = g.plan.n_full;
  plan->tail = g.plan.tail;
  plan->splits = g.plan.splits;
  plan->workgroups = g.workgroups;
  plan->threads = g.threads;
  return PB_OK;
}

pb_status pblock_backward_pairs(const pb_config* cfg, int block, int* paired) {
  PB_CHECK(check_config(cfg));
  if (!paired) return fail(PB_ERR_INVALID_ARG, "paired is NULL");
  if (block != 0 && block != 1) return fail(PB_ERR_INVALID_ARG, "block=%d must be 0 or 1", block);
  const Dims d = dims_of(cfg);
  const pb::Dt dt = dt_of(cfg);
  const pb::EpiArgs none;
  if (block == 0) {
    const ParallelBwdGemms g = parallel_bwd_gemms(d, nullptr, nullptr, nullptr, nullptr, nullptr,
                                                  nullptr, none, none, none, none);
    paired[0] = pb::gemm_pair_supported(dt, g.dc, g.dw_out);
    paired[1] = pb::gemm_pair_supported(dt, g.dh, g.dw_in);
  } else {
    const SerialBwdGemms g =
        serial_bwd_gemms(d, SerialBwdOperands{}, none, none, none, none, none, none, none, none);
    paired[0] = pb::gemm_pair_supported(dt, g.dg, g.dw_down);
    paired[1] = pb::gemm_pair_supported(dt, g.dh2, g.dw_up);
    paired[2] = pb::gemm_pair_supported(dt, g.d_o, g.dw_o);
    paired[3] = pb::gemm_pair_supported(dt, g.dh1, g.dw_qkv);
  }
  return PB_OK;
}

pb_status pblock_backward(const pb_config* cfg, const void* x, const void* ln_gamma,
                          const void* ln_beta, const void* w_in, const void* b_in,
                          const void* w_out, const void* b_out, const void* saved,
                          const void* dy, void* dx, float* dgamma, float* dbeta, float* dw_in,
                          float* db_in, float* dw_out, float* db_out, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
  return pblock_backward_timed(cfg, x, ln_gamma, ln_beta, w_in, b_in, w_out, b_out, saved, dy, dx,
                               dgamma, dbeta, dw_in, db_in, dw_out, db_out, ws, ws_bytes, stream,
                               nullptr);
}

pb_status pblock_backward_timed(const pb_config* cfg, const void* x, const void* ln_gamma,
                                const void* ln_beta, const void* w_in, const void* b_in,
                                const void* w_out, const void* b_out, const void* saved,
                                const void* dy, void* dx, float* dgamma, float* dbeta,
                                float* dw_in, float* db_in, float* dw_out, float* db_out, void* ws,
                                size_t ws_bytes, hipStream_t stream,
                                const pb_step_events* step_ev) {
  PB_CHECK(check_config(cfg));
  PB_CHECK(check_ptr(x, "x"));
  PB_CHECK(check_ptr(ln_gamma, "ln_gamma"));
  PB_CHECK(check_ptr(ln_beta, "ln_beta"));
  PB_CHECK(check_ptr(w_in, "w_in"));
  PB_CHECK(check_ptr(b_in, "b_in"));
  PB_CHECK(check_ptr(w_out, "w_out"));
  PB_CHECK(check_ptr(b_out, "b_out"));
  PB_CHECK(check_ptr(saved, "saved"));
  PB_CHECK(check_ptr(dy, "dy"));
  PB_CHECK(check_ptr(dx, "dx"));
  PB_CHECK(check_ptr(dgamma, "dgamma"));
  PB_CHECK(check_ptr(dbeta, "dbeta"));
  PB_CHECK(check_ptr(dw_in, "dw_in"));
  PB_CHECK(check_ptr(db_in, "db_in"));
  PB_CHECK(check_ptr(dw_out, "dw_out"));
  PB_CHECK(check_ptr(db_out, "db_out"));
  PB_CHECK(check_ptr(ws, "ws"));
  const Dims d = dims_of(cfg);
  const BwdLayout W = bwd_layout(d);
  if (ws_bytes < W.base)
    return fail(PB_ERR_WORKSPACE, "ws_bytes=%zu < %zu needed", ws_bytes, W.base);
  const SavedLayout L = saved_layout(d);
  const pb::Dt dt = dt_of(cfg);
  const size_t e = d.esz;
  const char* sb = (const char*)saved;
  const void* h = sb + L.off[0];
  const void* z = sb + L.off[1];
  const void* c = sb + L.off[2];
  const float* mean = (const float*)(sb + L.off[3]);
  const float* rstd = (const float*)(sb + L.off[4]);
  const float* lse = (const float*)(sb + L.off[5]);
  char* wb = (char*)ws;
  void* d_o = wb + W.d_o;
  void* dz = wb + W.dz;
  void* dh = wb + W.dh;
  float* delta = (float*)(wb + W.delta);
  float2* rowpart = (float2*)(wb + W.rowpart);
  float* pdg = (float*)(wb + W.pdg);
  float* pdb = (float*)(wb + W.pdb);
  float* pdy = (float*)(wb + W.pdy);
  float* part = (float*)(wb + W.part);
  int* queue = (int*)(wb + W.queue);
  float* split_ws = (float*)(wb + W.split);
  const size_t split_f = ws_bytes >= W.total ? (W.total - W.split) / 4 : 0;
  const int T = (int)d.T, H = (int)d.H, A = (int)d.A, N_in = (int)d.N_in, K_out = (int)d.K_out;
  (void)ln_beta;
  (void)b_in;
  (void)b_out;

  // Order: the chain dC -> attention -> dh -> LayerNorm, each step reading
  // what the previous one just wrote.  Where the two weight-gradient GEMMs can
  // share a launch with the GEMM before them (dW_out with dC, dW_in with dh:
  // see launch_gemm_pair), they do, and their short tiles fill the CUs the
  // long-K tiles leave idle; otherwise they come last, so their write-back
  // does not compete with the chain.
  pb::EpiArgs e2;  // B2: dW_out = dy^T C (contraction over tokens)
  e2.out = dw_out;
  e2.ld_out = K_out;
  pb::EpiArgs e5;  // B5: dW_in = dZ^T h
  e5.out = dw_in;
  e5.ld_out = H;

  // B1: dC = dy W_out; dO = dC[:, :A]; dU = dC[:, A:] * gelu'(U) -> dZ[:, 3A:]
  pb::EpiArgs e1;
  e1.out = d_o;
  e1.ld_out = A;
  e1.out2 = dz;
  e1.ld_out2 = N_in;
  e1.aux = z;
  e1.split = A;
  e1.col2 = 3 * A;
  e1.gelu_tanh = cfg->gelu_tanh;
  pb::EpiArgs e4;  // B4 (below): dh = dZ W_in with the LayerNorm backward's row terms
  e4.out = dh;
  e4.ld_out = H;
  e4.aux = x;
  e4.bias = ln_gamma;
  e4.mean = mean;
  e4.rstd = rstd;
  e4.rowpart = rowpart;
  e4.rowpart_ld = pb::ln_row_groups(H);
  ParallelBwdGemms G = parallel_bwd_gemms(d, dy, w_out, c, dz, w_in, h, e1, e2, e4, e5);
  const pb::GemmSpec &g_dc = G.dc, &g_dwo = G.dw_out, &g_dh = G.dh, &g_dwi = G.dw_in;
  auto run = [&](const pb::GemmSpec& g) {
    pb::launch_gemm(dt, g.epi, g.a_kcontig, g.b_kcontig, g.A, g.lda, g.B, g.ldb, g.M, g.N, g.K,
                    g.ep, split_ws, split_f, stream);
  };
  const bool pair_out = pb::gemm_pair_supported(dt, g_dc, g_dwo);
  // The attention backward's row terms delta = rowsum(dO * O) per head are
  // formed in dC's epilogue (the shared launch's LDS-staged path), where dO
  // leaves the accumulators, instead of re-reading dO and O in a launch of
  // their own: heads of 64 or 128 columns whose blocks align with the
  // epilogue's 128-column wave blocks.
  const bool delta_in_dc = pair_out && (d.d == 64 || d.d == 128) && A % 128 == 0;
  // db_in = sum over tokens of dZ: the row sums of dW_in's A operand (dZ^T),
  // formed by the shared launch's first tile column of dW_in
  const bool pair_in = pb::gemm_pair_supported(dt, g_dh, g_dwi);
  if (pair_in) G.dw_in.ep.rowsum = db_in;
  if (delta_in_dc) {
    G.dc.ep.o_rows = c;  // O = C[:, :A]
    G.dc.ep.ld_o_rows = K_out;
    G.dc.ep.delta = delta;
    G.dc.ep.delta_seq = (int)d.S;
    G.dc.ep.delta_heads = (int)d.heads;
    G.dc.ep.delta_hd = (int)d.d;
  }
  {
    StepScope sc(step_ev, PB_STEP_DC, stream);  // with dW_out when they share a launch
    // the shared launches are persistent: their queue heads start at zero
    if (pair_out || pair_in) pb::launch_queue_reset(queue, 2 * pb::kQueueInts, stream);
    if (pair_out)
      pb::launch_gemm_pair(dt, g_dc, g_dwo, queue, stream);
    else
      run(g_dc);
  }
  // B3: attention backward -> dQ, dK, dV into dZ[:, :3A]
  {
    StepScope sc(step_ev, PB_STEP_ATTN_BWD, stream);
    pb::launch_attn_backward(dt, attn_shape(d), z, at(z, A, e), at(z, 2LL * A, e), N_in, c,
                             K_out, d_o, A, lse, delta, delta_in_dc, dz, at(dz, A, e),
                             at(dz, 2LL * A, e), N_in, split_ws, split_f * 4, stream);
  }
  // B4: dh = dZ W_in, stored in the activation type; its epilogue also forms
  // the LayerNorm backward's row terms (sums of gamma dh and gamma dh xhat per
  // 64 columns) from the fp32 accumulators
  {
    StepScope sc(step_ev, PB_STEP_DH, stream);  // with dW_in when they share a launch
    if (pair_in)
      pb::launch_gemm_pair(dt, g_dh, g_dwi, queue + pb::kQueueInts, stream);
    else
      run(g_dh);
  }
  // B6: LN backward plus the residual path: dx = dy + LN'(dh); dgamma, dbeta
  {
    StepScope sc(step_ev, PB_STEP_LN_BWD, stream);
    pb::launch_ln_backward(dt, x, mean, rstd, ln_gamma, dh, rowpart, dy, dx, pdg, pdb, pdy, T, H,
                           stream);
    // dgamma, dbeta and db_out (= sum over tokens of dy) from the LN
    // backward's per-chunk partial sums, in one launch
    pb::launch_colsum3_f32(pdg, pdb, pdy, H, pb::ln_backward_chunks(T), H, dgamma, dbeta, db_out,
                           stream);
  }
  {
    StepScope sc(step_ev, PB_STEP_DB_OUT, stream);  // now inside the LN backward's column sums
  }
  // db_in = sum over tokens of dZ (already formed in dW_in's launch when
  // it shared dh's)
  {
    StepScope sc(step_ev, PB_STEP_DB_IN, stream);
    if (!pair_in) pb::launch_colsum(dt, dz, N_in, T, N_in, part, db_in, stream);
  }
  {
    StepScope sc(step_ev, PB_STEP_DW_OUT, stream);  // empty when it shared dC's launch
    if (!pair_out)
      run(g_dwo);
  }
  {
    StepScope sc(step_ev, PB_STEP_DW_IN, stream);  // empty when it shared dh's launch
    if (!pair_in)
      run(g_dwi);
  }
  return finish_launches();
}

pb_status pblock_swattn_forward(const pb_config* cfg, const void* q, const void* k,
                                const void* v, int ld_qkv, void* o, int ld_o, float* lse,
                                void* ws, size_t ws_bytes, hipStream_t stream) {
  PB_CHECK(check_attn_config(cfg));
  PB_CHECK(check_ptr(q, "q"));
  PB_CHECK(check_ptr(k, "k"));
  PB_CHECK(check_ptr(v, "v"));
  PB_CHECK(check_ptr(o, "o"));
  PB_CHECK(check_ptr(lse, "lse"));
  PB_CHECK(check_ld(ld_qkv, cfg, "ld_qkv"));
  PB_CHECK(check_ld(ld_o, cfg, "ld_o"));
  pb::AttnShape a;
  a.batch = cfg->batch;
  a.seq = cfg->seq;
  a.heads = cfg->heads;
  a.head_dim = cfg->head_dim;
  a.window = cfg->window < cfg->seq ? cfg->window : cfg->seq;
  if (ws) PB_CHECK(check_ptr(ws, "ws"));
  pb::launch_attn_forward(dt_of(cfg), a, q, k, v, ld_qkv, o, ld_o, lse, ws, ws ? ws_bytes : 0,
                          stream);
  return finish_launches();
}

}  // extern "C"

namespace {

// Scratch of pblock_swattn_forward_noalloc: the split forward's fp32 chunk
// partials live in this file-scope device array instead of a caller
// workspace.  Every GPU the library runs on holds its own copy, at its own
// address, until the process ends.  Host code never passes the array's name
// to a kernel or a copy (on the host it is a stand-in, not a device
// address); it uses the address hipGetSymbolAddress returns for the current
// device, looked up once per device.
constexpr size_t kNoallocScratchBytes = PB_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

std::atomic<void*> g_scratch_addr[kMaxDevices];
std::mutex g_scratch_mu;

pb_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(PB_ERR_HIP, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(PB_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_addr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return fail(PB_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d failed: %s", dev,
                    hipGetErrorString(e));
      g_scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return PB_OK;
}

}  // namespace

extern "C" {

pb_status pblock_swattn_forward_noalloc(const pb_config* cfg, const void* q, const void* k,
                                        const void* v, int ld_qkv, void* o, int ld_o,
                                        float* lse, hipStream_t stream) {
  PB_CHECK(check_attn_config(cfg));
  PB_CHECK(check_ptr(q, "q"));
  PB_CHECK(check_ptr(k, "k"));
  PB_CHECK(check_ptr(v, "v"));
  PB_CHECK(check_ptr(o, "o"));
  PB_CHECK(check_ptr(lse, "lse"));
  PB_CHECK(check_ld(ld_qkv, cfg, "ld_qkv"));
  PB_CHECK(check_ld(ld_o, cfg, "ld_o"));
  pb::AttnShape a;
  a.batch = cfg->batch;
  a.seq = cfg->seq;
  a.heads = cfg->heads;
  a.head_dim = cfg->head_dim;
  a.window = cfg->window < cfg->seq ? cfg->window : cfg->seq;
  const size_t need = pb::attn_fwd_partial_bytes(a, pb::attn_split_plan(dt_of(cfg), a));
  if (need > kNoallocScratchBytes)
    return fail(PB_ERR_UNSUPPORTED,
                "this shape's split forward needs %zu bytes of scratch, more than the %zu the "
                "allocation-free entry point holds; use pblock_swattn_forward with a workspace",
                need, kNoallocScratchBytes);
  void* ws = nullptr;
  if (need) PB_CHECK(scratch_address(&ws));
  pb::launch_attn_forward(dt_of(cfg), a, q, k, v, ld_qkv, o, ld_o, lse, ws, need, stream);
  return finish_launches();
}

size_t pblock_swattn_workspace_bytes(const pb_config* cfg, int mode) {
  if (check_attn_config(cfg) != PB_OK) return 0;
  pb::AttnShape a;
  a.batch = cfg->batch;
  a.seq = cfg->seq;
  a.heads = cfg->heads;
  a.head_dim = cfg->head_dim;
  a.window = cfg->window < cfg->seq ? cfg->window : cfg->seq;
  const pb::AttnSplit p = pb::attn_split_plan(dt_of(cfg), a);
  switch (mode) {
    case PB_ATTN_WS_FORWARD: return pb::attn_fwd_partial_bytes(a, p);
    case PB_ATTN_WS_BACKWARD_MIN: return swattn_delta_bytes(cfg);
    case PB_ATTN_WS_BACKWARD:
      return swattn_delta_bytes(cfg) +
             align256(pb::attn_bwd_partial_bytes(a, pb::attn_bwd_split_plan(dt_of(cfg), a)));
    default: return 0;
  }
}

pb_status pblock_swattn_backward(const pb_config* cfg, const void* q, const void* k,
                                 const void* v, int ld_qkv, const void* o, int ld_o,
                                 const void* d_o, int ld_do, const float* lse, void* dq, void* dk,
                                 void* dv, int ld_dqkv, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  PB_CHECK(check_attn_config(cfg));
  PB_CHECK(check_ptr(q, "q"));
  PB_CHECK(check_ptr(k, "k"));
  PB_CHECK(check_ptr(v, "v"));
  PB_CHECK(check_ptr(o, "o"));
  PB_CHECK(check_ptr(d_o, "d_o"));
  PB_CHECK(check_ptr(lse, "lse"));
  PB_CHECK(check_ptr(dq, "dq"));
  PB_CHECK(check_ptr(dk, "dk"));
  PB_CHECK(check_ptr(dv, "dv"));
  PB_CHECK(check_ptr(ws, "ws"));
  PB_CHECK(check_ld(ld_qkv, cfg, "ld_qkv"));
  PB_CHECK(check_ld(ld_o, cfg, "ld_o"));
  PB_CHECK(check_ld(ld_do, cfg, "ld_do"));
  PB_CHECK(check_ld(ld_dqkv, cfg, "ld_dqkv"));
  const size_t need = swattn_delta_bytes(cfg);
  if (ws_bytes < need) return fail(PB_ERR_WORKSPACE, "ws_bytes=%zu < %zu needed", ws_bytes, need);
  pb::AttnShape a;
  a.batch = cfg->batch;
  a.seq = cfg->seq;
  a.heads = cfg->heads;
  a.head_dim = cfg->head_dim;
  a.window = cfg->window < cfg->seq ? cfg->window : cfg->seq;
  pb::launch_attn_backward(dt_of(cfg), a, q, k, v, ld_qkv, o, ld_o, d_o, ld_do, lse, (float*)ws,
                           false, dq, dk, dv, ld_dqkv, (char*)ws + need, ws_bytes - need, stream);
  return finish_launches();
}

size_t pblock_serial_saved_bytes(const pb_config* cfg) {
  if (check_config(cfg) != PB_OK) return 0;
  return serial_layout(dims_of(cfg)).total;
}

pb_status pblock_serial_saved_offsets(const pb_config* cfg, size_t* offsets) {
  PB_CHECK(check_config(cfg));
  if (!offsets) return fail(PB_ERR_INVALID_ARG, "offsets is NULL");
  const SerialLayout L = serial_layout(dims_of(cfg));
  for (int i = 0; i < 10; ++i) offsets[i] = L.off[i];
  return PB_OK;
}

size_t pblock_serial_workspace_bytes(const pb_config* cfg, int mode) {
  if (check_config(cfg) != PB_OK) return 0;
  const Dims d = dims_of(cfg);
  const size_t split = align256(serial_split_fwd(d, dt_of(cfg)));
  switch (mode) {
    case PB_WS_FORWARD_WITH_STASH: return serial_layout(d).total + split;
    case PB_WS_BACKWARD: return serial_bwd_layout(d).total;
    case PB_WS_FORWARD: return split;
    default: return 0;
  }
}

pb_status pblock_serial_forward(const pb_config* cfg, const void* x, const void* ln1_gamma,
                                const void* ln1_beta, const void* ln2_gamma,
                                const void* ln2_beta, const void* w_in, const void* b_in,
                                const void* w_out, const void* b_o, const void* b_down, void* y,
                                void* saved, void* ws, size_t ws_bytes, hipStream_t stream) {
  PB_CHECK(check_config(cfg));
  PB_CHECK(check_ptr(x, "x"));
  PB_CHECK(check_ptr(ln1_gamma, "ln1_gamma"));
  PB_CHECK(check_ptr(ln1_beta, "ln1_beta"));
  PB_CHECK(check_ptr(ln2_gamma, "ln2_gamma"));
  PB_CHECK(check_ptr(ln2_beta, "ln2_beta"));
  PB_CHECK(check_ptr(w_in, "w_in"));
  PB_CHECK(check_ptr(b_in, "b_in"));
  PB_CHECK(check_ptr(w_out, "w_out"));
  PB_CHECK(check_ptr(b_o, "b_o"));
  PB_CHECK(check_ptr(b_down, "b_down"));
  PB_CHECK(check_ptr(y, "y"));
  const Dims d = dims_of(cfg);
  const SerialLayout L = serial_layout(d);
  const pb::Dt dt = dt_of(cfg);
  void* stash = saved;
  char* split_base = (char*)ws;
  size_t split_bytes = ws ? ws_bytes : 0;
  if (stash) {
    PB_CHECK(check_ptr(stash, "saved"));
    if (ws) PB_CHECK(check_ptr(ws, "ws"));
  } else {
    PB_CHECK(check_ptr(ws, "ws (needed when saved is NULL)"));
    if (ws_bytes < L.total)
      return fail(PB_ERR_WORKSPACE, "ws_bytes=%zu < %zu needed to hold the stash", ws_bytes,
                  L.total);
    stash = ws;
    split_base = (char*)ws + L.total;
    split_bytes = ws_bytes - L.total;
  }
  float* split_ws = (float*)split_base;
  const size_t split_f = split_bytes / 4;
  const size_t e = d.esz;
  char* sb = (char*)stash;
  void* h1 = sb + L.off[0];
  void* z = sb + L.off[1];
  void* c = sb + L.off[2];
  float* mean1 = (float*)(sb + L.off[3]);
  float* rstd1 = (float*)(sb + L.off[4]);
  float* lse = (float*)(sb + L.off[5]);
  void* x1 = sb + L.off[6];
  void* h2 = sb + L.off[7];
  float* mean2 = (float*)(sb + L.off[8]);
  float* rstd2 = (float*)(sb + L.off[9]);
  const int T = (int)d.T, H = (int)d.H, A = (int)d.A, F = (int)d.F, N_in = (int)d.N_in,
            K_out = (int)d.K_out;

  // x1 = x + Attention(LN1(x)) W_o^T + b_o
  pb::launch_ln_forward(dt, x, ln1_gamma, ln1_beta, h1, mean1, rstd1, T, H, cfg->ln_eps, stream);
  pb::EpiArgs eq;  // Q | K | V = h1 W_qkv^T + b_qkv -> Z[:, :3A] (no GeLU columns)
  eq.out = z;
  eq.ld_out = N_in;
  eq.out2 = c;
  eq.ld_out2 = K_out;
  eq.bias = b_in;
  eq.split = 3 * A;
  eq.gelu_tanh = cfg->gelu_tanh;
  pb::launch_gemm(dt, pb::Epi::BiasGelu, true, true, h1, H, w_in, H, T, 3 * A, H, eq, split_ws,
                  split_f, stream);
  pb::launch_attn_forward(dt, attn_shape(d), z, at(z, A, e), at(z, 2LL * A, e), N_in, c, K_out,
                          lse, split_base, split_bytes, stream);
  pb::EpiArgs eo;
  eo.out = x1;
  eo.ld_out = H;
  eo.bias = b_o;
  eo.resid = x;
  pb::launch_gemm(dt, pb::Epi::BiasResid, true, true, c, K_out, w_out, K_out, T, H, A, eo,
                  split_ws, split_f, stream);
  // y = x1 + GeLU(LN2(x1) W_up^T + b_up) W_down^T + b_down
  pb::launch_ln_forward(dt, x1, ln2_gamma, ln2_beta, h2, mean2, rstd2, T, H, cfg->ln_eps,
                        stream);
  pb::EpiArgs eu;  // U -> Z[:, 3A:], G = GeLU(U) -> C[:, A:]
  eu.out = at(z, 3LL * A, e);
  eu.ld_out = N_in;
  eu.out2 = c;
  eu.ld_out2 = K_out;
  eu.bias = at(b_in, 3LL * A, e);
  eu.split = 0;
  eu.col2 = A;
  eu.gelu_tanh = cfg->gelu_tanh;
  pb::launch_gemm(dt, pb::Epi::BiasGelu, true, true, h2, H, at(w_in, 3LL * A * H, e), H, T, F,
                  H, eu, split_ws, split_f, stream);
  pb::EpiArgs ed;
  ed.out = y;
  ed.ld_out = H;
  ed.bias = b_down;
  ed.resid = x1;
  pb::launch_gemm(dt, pb::Epi::BiasResid, true, true, at(c, A, e), K_out, at(w_out, A, e), K_out,
                  T, H, F, ed, split_ws, split_f, stream);
  return finish_launches();
}

pb_status pblock_serial_backward(const pb_config* cfg, const void* x, const void* ln1_gamma,
                                 const void* ln1_beta, const void* ln2_gamma,
                                 const void* ln2_beta, const void* w_in, const void* b_in,
                                 const void* w_out, const void* b_o, const void* b_down,
                                 const void* saved, const void* dy, void* dx,
                                 float* dln1_gamma, float* dln1_beta, float* dln2_gamma,
                                 float* dln2_beta, float* dw_in, float* db_in, float* dw_out,
                                 float* db_o, float* db_down, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  PB_CHECK(check_config(cfg));
  PB_CHECK(check_ptr(x, "x"));
  PB_CHECK(check_ptr(ln1_gamma, "ln1_gamma"));
  PB_CHECK(check_ptr(ln1_beta, "ln1_beta"));
  PB_CHECK(check_ptr(ln2_gamma, "ln2_gamma"));
  PB_CHECK(check_ptr(ln2_beta, "ln2_beta"));
  PB_CHECK(check_ptr(w_in, "w_in"));
  PB_CHECK(check_ptr(b_in, "b_in"));
  PB_CHECK(check_ptr(w_out, "w_out"));
  PB_CHECK(check_ptr(b_o, "b_o"));
  PB_CHECK(check_ptr(b_down, "b_down"));
  PB_CHECK(check_ptr(saved, "saved"));
  PB_CHECK(check_ptr(dy, "dy"));
  PB_CHECK(check_ptr(dx, "dx"));
  PB_CHECK(check_ptr(dln1_gamma, "dln1_gamma"));
  PB_CHECK(check_ptr(dln1_beta, "dln1_beta"));
  PB_CHECK(check_ptr(dln2_gamma, "dln2_gamma"));
  PB_CHECK(check_ptr(dln2_beta, "dln2_beta"));
  PB_CHECK(check_ptr(dw_in, "dw_in"));
  PB_CHECK(check_ptr(db_in, "db_in"));
  PB_CHECK(check_ptr(dw_out, "dw_out"));
  PB_CHECK(check_ptr(db_o, "db_o"));
  PB_CHECK(check_ptr(db_down, "db_down"));
  PB_CHECK(check_ptr(ws, "ws"));
  const Dims d = dims_of(cfg);
  const SerialBwdLayout W = serial_bwd_layout(d);
  if (ws_bytes < W.base)
    return fail(PB_ERR_WORKSPACE, "ws_bytes=%zu < %zu needed", ws_bytes, W.base);
  const SerialLayout L = serial_layout(d);
  const pb::Dt dt = dt_of(cfg);
  const size_t e = d.esz;
  const char* sb = (const char*)saved;
  const void* h1 = sb + L.off[0];
  const void* z = sb + L.off[1];
  const void* c = sb + L.off[2];
  const float* mean1 = (const float*)(sb + L.off[3]);
  const float* rstd1 = (const float*)(sb + L.off[4]);
  const float* lse = (const float*)(sb + L.off[5]);
  const void* x1 = sb + L.off[6];
  const void* h2 = sb + L.off[7];
  const float* mean2 = (const float*)(sb + L.off[8]);
  const float* rstd2 = (const float*)(sb + L.off[9]);
  char* wb = (char*)ws;
  void* d_o = wb + W.d_o;
  void* dz = wb + W.dz;
  void* dh = wb + W.dh;
  void* dx1 = wb + W.dx1;
  float* delta = (float*)(wb + W.delta);
  float2* rowpart = (float2*)(wb + W.rowpart);
  float* pdg = (float*)(wb + W.pdg);
  float* pdb = (float*)(wb + W.pdb);
  float* pdy = (float*)(wb + W.pdy);
  float* part = (float*)(wb + W.part);
  int* queue = (int*)(wb + W.queue);
  float* split_ws = (float*)(wb + W.split);
  const size_t split_f = ws_bytes >= W.total ? (W.total - W.split) / 4 : 0;
  const int T = (int)d.T, H = (int)d.H, A = (int)d.A, F = (int)d.F, N_in = (int)d.N_in,
            K_out = (int)d.K_out;
  const int nblk = pb::ln_backward_chunks(T);
  (void)ln1_beta;
  (void)ln2_beta;
  (void)b_in;
  (void)b_o;
  (void)b_down;

  // Each weight gradient (a token contraction, fp32) shares one launch with
  // the GEMM before it where launch_gemm_pair takes the pair, so its short
  // tiles fill the CUs the other leaves idle; any other runs at the end.
  pb::EpiArgs wd, wo, wu, wq;
  wd.out = at(dw_out, A, 4);  // dW_down = dy^T G
  wd.ld_out = K_out;
  wo.out = dw_out;  // dW_o = dx1^T O
  wo.ld_out = K_out;
  wu.out = at(dw_in, 3LL * A * H, 4);  // dW_up = dU^T h2
  wu.ld_out = H;
  wq.out = dw_in;  // dW_qkv = dQKV^T h1
  wq.ld_out = H;
  // dG = dy W_down, dU = dG * gelu'(U) -> dZ[:, 3A:]
  pb::EpiArgs e1;
  e1.out = dz;
  e1.ld_out = N_in;
  e1.out2 = dz;
  e1.ld_out2 = N_in;
  e1.aux = z;
  e1.split = 0;
  e1.col2 = 3 * A;
  e1.gelu_tanh = cfg->gelu_tanh;
  // dh2 = dU W_up, with LN2's row terms
  pb::EpiArgs e2;
  e2.out = dh;
  e2.ld_out = H;
  e2.aux = x1;
  e2.bias = ln2_gamma;
  e2.mean = mean2;
  e2.rstd = rstd2;
  e2.rowpart = rowpart;
  e2.rowpart_ld = pb::ln_row_groups(H);
  // dO = dx1 W_o
  pb::EpiArgs e3;
  e3.out = d_o;
  e3.ld_out = A;
  e3.split = A;  // every column is dO
  e3.gelu_tanh = cfg->gelu_tanh;
  // dh1 = dQKV W_qkv, with LN1's row terms
  pb::EpiArgs e4;
  e4.out = dh;
  e4.ld_out = H;
  e4.aux = x;
  e4.bias = ln1_gamma;
  e4.mean = mean1;
  e4.rstd = rstd1;
  e4.rowpart = rowpart;
  e4.rowpart_ld = pb::ln_row_groups(H);
  SerialBwdGemms G = serial_bwd_gemms(
      d, SerialBwdOperands{dy, dx1, c, dz, h1, h2, w_in, w_out}, e1, wd, e2, wu, e3, wo, e4, wq);
  // As in the parallel block: db_in from the row sums of the weight
  // gradients' A operands (dU^T in dW_up, dQKV^T in dW_qkv) when both share
  // launches, and the attention backward's delta from the dO GEMM's epilogue
  const bool db_in_fused = pb::gemm_pair_supported(dt, G.dh2, G.dw_up) &&
                           pb::gemm_pair_supported(dt, G.dh1, G.dw_qkv);
  if (db_in_fused) {
    G.dw_up.ep.rowsum = db_in + 3LL * A;
    G.dw_qkv.ep.rowsum = db_in;
  }
  const bool delta_in_do = pb::gemm_pair_supported(dt, G.d_o, G.dw_o) &&
                           (d.d == 64 || d.d == 128) && A % 128 == 0;
  if (delta_in_do) {
    G.d_o.ep.o_rows = c;  // O = C[:, :A]
    G.d_o.ep.ld_o_rows = K_out;
    G.d_o.ep.delta = delta;
    G.d_o.ep.delta_seq = (int)d.S;
    G.d_o.ep.delta_heads = (int)d.heads;
    G.d_o.ep.delta_hd = (int)d.d;
  }
  auto run = [&](const pb::GemmSpec& g) {
    pb::launch_gemm(dt, g.epi, g.a_kcontig, g.b_kcontig, g.A, g.lda, g.B, g.ldb, g.M, g.N, g.K,
                    g.ep, split_ws, split_f, stream);
  };
  const pb::GemmSpec* deferred[4];
  int n_deferred = 0;
  // the shared launches are persistent, each with its own queue heads,
  // zeroed here
  static_assert(kBwdQueueSets >= 4, "one queue per shared launch");
  if (pb::gemm_pair_supported(dt, G.dg, G.dw_down) || pb::gemm_pair_supported(dt, G.dh2, G.dw_up) ||
      pb::gemm_pair_supported(dt, G.d_o, G.dw_o) || pb::gemm_pair_supported(dt, G.dh1, G.dw_qkv))
    pb::launch_queue_reset(queue, 4 * pb::kQueueInts, stream);
  int n_pairs = 0;
  auto run_with = [&](const pb::GemmSpec& g, const pb::GemmSpec& wg) {
    if (!pb::launch_gemm_pair(dt, g, wg, queue + pb::kQueueInts * n_pairs++, stream)) {
      run(g);
      deferred[n_deferred++] = &wg;
    }
  };

  // MLP: dG and dU, then dh2
  run_with(G.dg, G.dw_down);
  run_with(G.dh2, G.dw_up);
  // dx1 = dy + LN2'(dh2); dgamma2, dbeta2, and db_down = sum dy
  pb::launch_ln_backward(dt, x1, mean2, rstd2, ln2_gamma, dh, rowpart, dy, dx1, pdg, pdb, pdy, T,
                         H, stream);
  pb::launch_colsum3_f32(pdg, pdb, pdy, H, nblk, H, dln2_gamma, dln2_beta, db_down, stream);
  // attention: dO = dx1 W_o, then dQ, dK, dV -> dZ[:, :3A]
  run_with(G.d_o, G.dw_o);
  pb::launch_attn_backward(dt, attn_shape(d), z, at(z, A, e), at(z, 2LL * A, e), N_in, c, K_out,
                           d_o, A, lse, delta, delta_in_do, dz, at(dz, A, e), at(dz, 2LL * A, e),
                           N_in, split_ws, split_f * 4, stream);
  run_with(G.dh1, G.dw_qkv);
  // dx = dx1 + LN1'(dh1); dgamma1, dbeta1, and db_o = sum dx1
  pb::launch_ln_backward(dt, x, mean1, rstd1, ln1_gamma, dh, rowpart, dx1, dx, pdg, pdb, pdy, T,
                         H, stream);
  pb::launch_colsum3_f32(pdg, pdb, pdy, H, nblk, H, dln1_gamma, dln1_beta, db_o, stream);
  // bias gradients of the input projections: db_in = sum over tokens of dZ
  if (!db_in_fused) pb::launch_colsum(dt, dz, N_in, T, N_in, part, db_in, stream);
  // weight gradients that did not share a launch, last
  for (int i = 0; i < n_deferred; ++i) run(*deferred[i]);
  return finish_launches();
}

// -------------------------------------------- tensor-parallel context
namespace {
constexpr int kAgMaxComm = 8;
constexpr int kAgMaxTp = 64;
}  // namespace

// Events of the pipelined all-gather and reduce-scatter calls, tp of each
// kind plus one, on one device.
struct pb_tp_context {
  int device;
  int tp;
  hipEvent_t start;             // AG: the work on `stream` before the copies
  hipEvent_t landed[kAgMaxTp];  // AG: per position in the ring order
  hipEvent_t computed[kAgMaxTp];// RS: per launch group, on `stream`
  hipEvent_t sent[kAgMaxTp];    // RS: per chunk, on its comm stream
};

pb_status pblock_tp_context_create(int tp, pb_tp_context** ctx) {
  if (!ctx) return fail(PB_ERR_INVALID_ARG, "ctx is NULL");
  *ctx = nullptr;
  if (tp < 1 || tp > kAgMaxTp) return fail(PB_ERR_INVALID_ARG, "tp=%d must be in 1..64", tp);
  pb_tp_context* c = new (std::nothrow) pb_tp_context{};
  if (!c) return fail(PB_ERR_INVALID_ARG, "out of host memory");
  c->tp = tp;
  bool ok = hipGetDevice(&c->device) == hipSuccess;
  auto make = [&](hipEvent_t* ev) {
    ok = ok && hipEventCreateWithFlags(ev, hipEventDisableTiming) == hipSuccess;
  };
  make(&c->start);
  for (int i = 0; i < tp; ++i) {
    make(&c->landed[i]);
    make(&c->computed[i]);
    make(&c->sent[i]);
  }
  if (!ok) {
    pblock_tp_context_destroy(c);
    return fail(PB_ERR_HIP, "hipEventCreateWithFlags failed");
  }
  *ctx = c;
  return PB_OK;
}

void pblock_tp_context_destroy(pb_tp_context* ctx) {
  if (!ctx) return;
  auto drop = [](hipEvent_t e) {
    if (e) (void)hipEventDestroy(e);
  };
  drop(ctx->start);
  for (int i = 0; i < ctx->tp; ++i) {
    drop(ctx->landed[i]);
    drop(ctx->computed[i]);
    drop(ctx->sent[i]);
  }
  delete ctx;
}

// ------------------------- all-gather / reduce-scatter pipelined with GEMMs
namespace {
pb_status check_tp_streams(int tp, int rank, long long T, int per_launch, int n_comm,
                           const hipStream_t* comm_streams, hipStream_t stream) {
  if (tp < 1 || tp > kAgMaxTp) return fail(PB_ERR_INVALID_ARG, "tp=%d must be in 1..64", tp);
  if (rank < 0 || rank >= tp) return fail(PB_ERR_INVALID_ARG, "rank=%d not in 0..tp-1", rank);
  if (T % tp) return fail(PB_ERR_INVALID_ARG, "tokens=%lld not divisible by tp=%d", T, tp);
  if (per_launch < 1 || per_launch > tp)
    return fail(PB_ERR_INVALID_ARG, "shards_per_launch=%d must be in 1..tp", per_launch);
  if (n_comm < 1 || n_comm > kAgMaxComm)
    return fail(PB_ERR_INVALID_ARG, "n_comm=%d must be in 1..%d", n_comm, kAgMaxComm);
  if (!comm_streams) return fail(PB_ERR_INVALID_ARG, "comm_streams is NULL");
  for (int i = 0; i < n_comm; ++i) {
    if (comm_streams[i] == stream)
      return fail(PB_ERR_INVALID_ARG, "comm_streams[%d] equals stream", i);
    for (int k = 0; k < i; ++k)
      if (comm_streams[k] == comm_streams[i])
        return fail(PB_ERR_INVALID_ARG, "comm_streams[%d] repeats comm_streams[%d]", i, k);
  }
  return PB_OK;
}
// Checked after every other argument: the one check that asks HIP (for the
// current device).
pb_status check_ctx(const pb_tp_context* ctx, int tp) {
  if (!ctx) return fail(PB_ERR_INVALID_ARG, "ctx is NULL");
  if (ctx->tp != tp)
    return fail(PB_ERR_INVALID_ARG, "ctx was made for tp=%d, called with tp=%d", ctx->tp, tp);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(PB_ERR_HIP, "hipGetDevice failed");
  if (dev != ctx->device)
    return fail(PB_ERR_INVALID_ARG, "ctx belongs to device %d, the current device is %d",
                ctx->device, dev);
  return PB_OK;
}
}  // namespace

}  // extern "C"

namespace {
// Largest GEMM split region over the launches of a pipelined call: row
// ranges of m whole shards, m = 1 .. per_launch, of an (rows m) x N x K GEMM.
size_t rows_split_bytes(pb::Dt dt, int rows, int N, int K, int per_launch) {
  size_t m = 0;
  for (int k = 1; k <= per_launch; ++k)
    m = std::max(m, pb::gemm_split_floats(pb::gemm_split_plan(dt, rows * k, N, K)) * 4);
  return align256(m);
}
bool tp_args_ok(const pb_config* cfg, int tp, int per_launch) {
  return check_config(cfg) == PB_OK && tp >= 1 && tp <= kAgMaxTp && per_launch >= 1 &&
         per_launch <= tp && dims_of(cfg).T % tp == 0;
}

// All-gather pipelined into a row-parallel GEMM: the shards are copied into
// `gathered` on the comm streams in ring order from `rank` (the k-th on
// comm_streams[k % n_comm]); gemm_rows(j0, n) computes the GEMM over the
// rows of shards j0 .. j0 + n - 1 on `stream`, each launch of per_launch
// shards waiting (by event) only for its own.  Shards already in place at
// the head of that order are not copied and form a first launch of their
// own unless the call is unpipelined.
template <class F>
pb_status ag_pipeline(int tp, int rank, const void* const* shards, void* gathered,
                      size_t shard_bytes, int per_launch, hipStream_t stream, int n_comm,
                      const hipStream_t* comm_streams, pb_tp_context& ev, F gemm_rows) {
  auto ok = [](hipError_t e) { return e == hipSuccess; };
  auto in_place = [&](int j) {
    return shards[j] == (const char*)gathered + (size_t)j * shard_bytes;
  };
  // Only shards that are copied involve the comm streams and events: a
  // shard already in place needs no wait (cross-stream waits cost ~0.1 ms
  // per call when every shard went through them).
  bool any_copy = false;
  for (int j = 0; j < tp; ++j) any_copy = any_copy || !in_place(j);
  if (any_copy) {
    // the copies start after the work already on `stream` (which may produce
    // the local shard)
    if (!ok(hipEventRecord(ev.start, stream))) return fail(PB_ERR_HIP, "hipEventRecord failed");
    for (int i = 0; i < n_comm; ++i)
      if (!ok(hipStreamWaitEvent(comm_streams[i], ev.start, 0)))
        return fail(PB_ERR_HIP, "hipStreamWaitEvent failed");
  }
  for (int k = 0; k < tp; ++k) {
    const int j = (rank + k) % tp;
    if (in_place(j)) continue;
    hipStream_t cs = comm_streams[k % n_comm];
    char* dst = (char*)gathered + (size_t)j * shard_bytes;
    if (!ok(hipMemcpyAsync(dst, shards[j], shard_bytes, hipMemcpyDeviceToDeviceNoCU, cs)))
      return fail(PB_ERR_HIP, "hipMemcpyAsync of shard %d failed", j);
    if (!ok(hipEventRecord(ev.landed[k], cs))) return fail(PB_ERR_HIP, "hipEventRecord failed");
  }
  int ready = 0;
  while (ready < tp && in_place((rank + ready) % tp)) ++ready;
  auto launch_group = [&](int k0, int k1, bool wait) -> bool {
    if (wait)
      for (int k = k0; k < k1; ++k)
        if (!in_place((rank + k) % tp) && !ok(hipStreamWaitEvent(stream, ev.landed[k], 0)))
          return false;
    const int j0 = (rank + k0) % tp, n = k1 - k0;
    if (j0 + n <= tp) {
      gemm_rows(j0, n);
    } else {
      gemm_rows(j0, tp - j0);
      gemm_rows(0, j0 + n - tp);
    }
    return true;
  };
  int k0 = 0;
  if (ready > 0 && ready < tp && per_launch < tp) {
    if (!launch_group(0, ready, false)) return fail(PB_ERR_HIP, "hipStreamWaitEvent failed");
    k0 = ready;
  }
  for (; k0 < tp; k0 += per_launch)
    if (!launch_group(k0, std::min(tp, k0 + per_launch), true))
      return fail(PB_ERR_HIP, "hipStreamWaitEvent failed");
  return PB_OK;
}

// A row-parallel GEMM pipelined into a reduce-scatter: gemm_rows(j0, n)
// writes the rows of chunks j0 .. j0 + n - 1 of `partial` on `stream`, in
// ring order from rank + 1 (this rank's own chunk last), per_launch chunks
// per launch; chunk j goes to dst[j] on comm_streams[k % n_comm] (k its
// position) as soon as its launch has finished.  Later work on `stream`
// follows every send.
template <class F>
pb_status rs_pipeline(int tp, int rank, const void* partial, void* const* dst, size_t chunk_bytes,
                      int per_launch, hipStream_t stream, int n_comm,
                      const hipStream_t* comm_streams, pb_tp_context& ev, F gemm_rows) {
  auto ok = [](hipError_t e) { return e == hipSuccess; };
  int group = 0;
  for (int k0 = 0; k0 < tp; k0 += per_launch, ++group) {
    const int k1 = std::min(tp, k0 + per_launch);
    const int j0 = (rank + 1 + k0) % tp, n = k1 - k0;
    if (j0 + n <= tp) {
      gemm_rows(j0, n);
    } else {
      gemm_rows(j0, tp - j0);
      gemm_rows(0, j0 + n - tp);
    }
    bool recorded = false;
    for (int k = k0; k < k1; ++k) {
      const int j = (rank + 1 + k) % tp;
      const char* src = (const char*)partial + (size_t)j * chunk_bytes;
      if (dst[j] == src) continue;  // in place: nothing to send or wait for
      if (!recorded) {
        if (!ok(hipEventRecord(ev.computed[group], stream)))
          return fail(PB_ERR_HIP, "hipEventRecord failed");
        recorded = true;
      }
      hipStream_t cs = comm_streams[k % n_comm];
      if (!ok(hipStreamWaitEvent(cs, ev.computed[group], 0)))
        return fail(PB_ERR_HIP, "hipStreamWaitEvent failed");
      if (!ok(hipMemcpyAsync(dst[j], src, chunk_bytes, hipMemcpyDeviceToDeviceNoCU, cs)))
        return fail(PB_ERR_HIP, "hipMemcpyAsync of chunk %d failed", j);
      if (!ok(hipEventRecord(ev.sent[k], cs))) return fail(PB_ERR_HIP, "hipEventRecord failed");
    }
  }
  for (int k = 0; k < tp; ++k) {
    const int j = (rank + 1 + k) % tp;
    if (dst[j] == (const char*)partial + (size_t)j * chunk_bytes) continue;
    if (!ok(hipStreamWaitEvent(stream, ev.sent[k], 0)))
      return fail(PB_ERR_HIP, "hipStreamWaitEvent failed");
  }
  return PB_OK;
}

pb_status check_list(const void* const* p, int n, const char* name) {
  if (!p) return fail(PB_ERR_INVALID_ARG, "%s is NULL", name);
  for (int j = 0; j < n; ++j)
    if (!p[j] || (uintptr_t)p[j] % 16)
      return fail(PB_ERR_INVALID_ARG, "%s[%d] is NULL or not 16-byte aligned", name, j);
  return PB_OK;
}
pb_status check_ws(const void* ws, size_t ws_bytes) {
  if (ws_bytes && (!ws || (uintptr_t)ws % 256))
    return fail(PB_ERR_INVALID_ARG, "ws is NULL or not 256-byte aligned");
  return PB_OK;
}
}  // namespace

extern "C" {

size_t pblock_ag_in_proj_workspace_bytes(const pb_config* cfg, int tp, int shards_per_launch) {
  if (!tp_args_ok(cfg, tp, shards_per_launch)) return 0;
  const Dims d = dims_of(cfg);
  return rows_split_bytes(dt_of(cfg), (int)(d.T / tp), (int)d.N_in, (int)d.H, shards_per_launch);
}

pb_status pblock_ag_in_proj(const pb_config* cfg, int tp, int rank, const void* const* shards,
                            void* h, const void* w_in, const void* b_in, void* z, void* c,
                            int shards_per_launch, void* ws, size_t ws_bytes, hipStream_t stream,
                            int n_comm, const hipStream_t* comm_streams, pb_tp_context* ctx) {
  PB_CHECK(check_config(cfg));
  const Dims d = dims_of(cfg);
  PB_CHECK(check_tp_streams(tp, rank, d.T, shards_per_launch, n_comm, comm_streams, stream));
  PB_CHECK(check_list(shards, tp, "shards"));
  PB_CHECK(check_ptr(h, "h"));
  PB_CHECK(check_ptr(w_in, "w_in"));
  PB_CHECK(check_ptr(b_in, "b_in"));
  PB_CHECK(check_ptr(z, "z"));
  PB_CHECK(check_ptr(c, "c"));
  PB_CHECK(check_ws(ws, ws_bytes));
  PB_CHECK(check_ctx(ctx, tp));
  const pb::Dt dt = dt_of(cfg);
  const int H = (int)d.H, A = (int)d.A, N_in = (int)d.N_in, K_out = (int)d.K_out;
  const int rows = (int)(d.T / tp);
  const size_t e = d.esz;
  float* split_ws = (float*)ws;
  const size_t split_f = ws_bytes / 4;
  // the in-projection of rows of h: Z (bias) and G = gelu(U) as the forward
  auto gemm_rows = [&](int j0, int nsh) {
    const int r0 = j0 * rows, m = nsh * rows;
    pb::EpiArgs e1;
    e1.out = at(z, (long long)r0 * N_in, e);
    e1.ld_out = N_in;
    e1.out2 = at(c, (long long)r0 * K_out, e);
    e1.ld_out2 = K_out;
    e1.bias = b_in;
    e1.split = 3 * A;
    e1.col2 = A;
    e1.gelu_tanh = cfg->gelu_tanh;
    pb::launch_gemm(dt, pb::Epi::BiasGelu, true, true, at(h, (long long)r0 * H, e), H, w_in, H,
                    m, N_in, H, e1, split_ws, split_f, stream);
  };
  PB_CHECK(ag_pipeline(tp, rank, shards, h, (size_t)rows * H * e, shards_per_launch, stream,
                       n_comm, comm_streams, *ctx, gemm_rows));
  return finish_launches();
}

size_t pblock_ag_dc_workspace_bytes(const pb_config* cfg, int tp, int shards_per_launch) {
  if (!tp_args_ok(cfg, tp, shards_per_launch)) return 0;
  const Dims d = dims_of(cfg);
  return rows_split_bytes(dt_of(cfg), (int)(d.T / tp), (int)d.K_out, (int)d.H, shards_per_launch);
}

pb_status pblock_ag_dc(const pb_config* cfg, int tp, int rank, const void* const* dy_shards,
                       void* dy, const void* w_out, const void* z, void* d_o, void* dz,
                       int shards_per_launch, void* ws, size_t ws_bytes, hipStream_t stream,
                       int n_comm, const hipStream_t* comm_streams, pb_tp_context* ctx) {
  PB_CHECK(check_config(cfg));
  const Dims d = dims_of(cfg);
  PB_CHECK(check_tp_streams(tp, rank, d.T, shards_per_launch, n_comm, comm_streams, stream));
  PB_CHECK(check_list(dy_shards, tp, "dy_shards"));
  PB_CHECK(check_ptr(dy, "dy"));
  PB_CHECK(check_ptr(w_out, "w_out"));
  PB_CHECK(check_ptr(z, "z"));
  PB_CHECK(check_ptr(d_o, "d_o"));
  PB_CHECK(check_ptr(dz, "dz"));
  PB_CHECK(check_ws(ws, ws_bytes));
  PB_CHECK(check_ctx(ctx, tp));
  const pb::Dt dt = dt_of(cfg);
  const int H = (int)d.H, A = (int)d.A, N_in = (int)d.N_in, K_out = (int)d.K_out;
  const int rows = (int)(d.T / tp);
  const size_t e = d.esz;
  float* split_ws = (float*)ws;
  const size_t split_f = ws_bytes / 4;
  // dC = dy W_out over rows of dy: dO = dC[:, :A], dU = dC[:, A:] * gelu'(U)
  // -> dZ[:, 3A:], as the backward pass writes them
  auto gemm_rows = [&](int j0, int nsh) {
    const int r0 = j0 * rows, m = nsh * rows;
    pb::EpiArgs e1;
    e1.out = at(d_o, (long long)r0 * A, e);
    e1.ld_out = A;
    e1.out2 = at(dz, (long long)r0 * N_in, e);
    e1.ld_out2 = N_in;
    e1.aux = at(z, (long long)r0 * N_in, e);
    e1.split = A;
    e1.col2 = 3 * A;
    e1.gelu_tanh = cfg->gelu_tanh;
    pb::launch_gemm(dt, pb::Epi::DgeluSplit, true, false, at(dy, (long long)r0 * H, e), H, w_out,
                    K_out, m, K_out, H, e1, split_ws, split_f, stream);
  };
  PB_CHECK(ag_pipeline(tp, rank, dy_shards, dy, (size_t)rows * H * e, shards_per_launch, stream,
                       n_comm, comm_streams, *ctx, gemm_rows));
  return finish_launches();
}

size_t pblock_rs_out_proj_workspace_bytes(const pb_config* cfg, int tp, int shards_per_launch) {
  if (!tp_args_ok(cfg, tp, shards_per_launch)) return 0;
  const Dims d = dims_of(cfg);
  return rows_split_bytes(dt_of(cfg), (int)(d.T / tp), (int)d.H, (int)d.K_out, shards_per_launch);
}

pb_status pblock_rs_out_proj(const pb_config* cfg, int tp, int rank, const void* c,
                             const void* w_out, void* partial, void* const* dst,
                             int shards_per_launch, void* ws, size_t ws_bytes, hipStream_t stream,
                             int n_comm, const hipStream_t* comm_streams, pb_tp_context* ctx) {
  PB_CHECK(check_config(cfg));
  const Dims d = dims_of(cfg);
  PB_CHECK(check_tp_streams(tp, rank, d.T, shards_per_launch, n_comm, comm_streams, stream));
  PB_CHECK(check_list(dst, tp, "dst"));
  PB_CHECK(check_ptr(c, "c"));
  PB_CHECK(check_ptr(w_out, "w_out"));
  PB_CHECK(check_ptr(partial, "partial"));
  PB_CHECK(check_ws(ws, ws_bytes));
  PB_CHECK(check_ctx(ctx, tp));
  const pb::Dt dt = dt_of(cfg);
  const int H = (int)d.H, K_out = (int)d.K_out;
  const int rows = (int)(d.T / tp);
  const size_t e = d.esz;
  float* split_ws = (float*)ws;
  const size_t split_f = ws_bytes / 4;
  // P = C W_out^T over a row range, stored in the activation type
  auto gemm_rows = [&](int j0, int nsh) {
    const int r0 = j0 * rows, m = nsh * rows;
    pb::EpiArgs ep;
    ep.out = at(partial, (long long)r0 * H, e);
    ep.ld_out = H;
    ep.split = H;  // every column is a plain store
    pb::launch_gemm(dt, pb::Epi::DgeluSplit, true, true, at(c, (long long)r0 * K_out, e), K_out,
                    w_out, K_out, m, H, K_out, ep, split_ws, split_f, stream);
  };
  PB_CHECK(rs_pipeline(tp, rank, partial, dst, (size_t)rows * H * e, shards_per_launch, stream,
                       n_comm, comm_streams, *ctx, gemm_rows));
  return finish_launches();
}

size_t pblock_rs_dh_workspace_bytes(const pb_config* cfg, int tp, int shards_per_launch) {
  if (!tp_args_ok(cfg, tp, shards_per_launch)) return 0;
  const Dims d = dims_of(cfg);
  return rows_split_bytes(dt_of(cfg), (int)(d.T / tp), (int)d.H, (int)d.N_in, shards_per_launch);
}

pb_status pblock_rs_dh(const pb_config* cfg, int tp, int rank, const void* dz, const void* w_in,
                       void* partial, void* const* dst, int shards_per_launch, void* ws,
                       size_t ws_bytes, hipStream_t stream, int n_comm,
                       const hipStream_t* comm_streams, pb_tp_context* ctx) {
  PB_CHECK(check_config(cfg));
  const Dims d = dims_of(cfg);
  PB_CHECK(check_tp_streams(tp, rank, d.T, shards_per_launch, n_comm, comm_streams, stream));
  PB_CHECK(check_list(dst, tp, "dst"));
  PB_CHECK(check_ptr(dz, "dz"));
  PB_CHECK(check_ptr(w_in, "w_in"));
  PB_CHECK(check_ptr(partial, "partial"));
  PB_CHECK(check_ws(ws, ws_bytes));
  PB_CHECK(check_ctx(ctx, tp));
  const pb::Dt dt = dt_of(cfg);
  const int H = (int)d.H, N_in = (int)d.N_in;
  const int rows = (int)(d.T / tp);
  const size_t e = d.esz;
  float* split_ws = (float*)ws;
  const size_t split_f = ws_bytes / 4;
  // this rank's partial dh = dZ W_in over a row range (W_in's rows are
  // MN-contiguous here), stored in the activation type
  auto gemm_rows = [&](int j0, int nsh) {
    const int r0 = j0 * rows, m = nsh * rows;
    pb::EpiArgs ep;
    ep.out = at(partial, (long long)r0 * H, e);
    ep.ld_out = H;
    ep.split = H;  // every column is a plain store
    pb::launch_gemm(dt, pb::Epi::DgeluSplit, true, false, at(dz, (long long)r0 * N_in, e), N_in,
                    w_in, H, m, H, N_in, ep, split_ws, split_f, stream);
  };
  PB_CHECK(rs_pipeline(tp, rank, partial, dst, (size_t)rows * H * e, shards_per_launch, stream,
                       n_comm, comm_streams, *ctx, gemm_rows));
  return finish_launches();
}

pb_status pblock_rs_reduce(const pb_config* cfg, int tp, const void* const* parts,
                           const void* x_shard, const void* b_out, void* y_shard,
                           hipStream_t stream) {
  PB_CHECK(check_config(cfg));
  const Dims d = dims_of(cfg);
  if (tp < 1 || tp > pb::kRsMaxParts)
    return fail(PB_ERR_INVALID_ARG, "tp=%d must be in 1..%d", tp, pb::kRsMaxParts);
  if (d.T % tp) return fail(PB_ERR_INVALID_ARG, "tokens=%lld not divisible by tp=%d", d.T, tp);
  if (!parts) return fail(PB_ERR_INVALID_ARG, "parts is NULL");
  pb::RsParts rp{};
  rp.n = tp;
  for (int q = 0; q < tp; ++q) {
    if (!parts[q] || (uintptr_t)parts[q] % 16)
      return fail(PB_ERR_INVALID_ARG, "parts[%d] is NULL or not 16-byte aligned", q);
    rp.p[q] = parts[q];
  }
  // x_shard and b_out may be NULL (the sum alone: the backward's dh)
  if (x_shard) PB_CHECK(check_ptr(x_shard, "x_shard"));
  if (b_out) PB_CHECK(check_ptr(b_out, "b_out"));
  PB_CHECK(check_ptr(y_shard, "y_shard"));
  pb::launch_rs_reduce(dt_of(cfg), rp, x_shard, b_out, y_shard, (int)(d.T / tp), (int)d.H,
                       stream);
  return finish_launches();
}

// ---------------------------------------------------------------- LAMB step
static_assert(PB_LAMB_MAX_TENSORS == pb::kLambMaxTensors, "tensor limit");

size_t pblock_lamb_workspace_bytes(int n_tensors, const pb_lamb_tensor* tensors) {
  if (n_tensors < 1 || n_tensors > PB_LAMB_MAX_TENSORS || !tensors) return 0;
  long long chunks = 0;
  for (int i = 0; i < n_tensors; ++i) chunks += pb::lamb_padded_chunks((long long)tensors[i].numel);
  if (chunks > INT32_MAX) return 0;
  return align256((size_t)chunks * sizeof(float2)) +
         align256((size_t)(chunks / pb::kLambGroup) * sizeof(double2)) +
         align256((size_t)n_tensors * 4);
}

pb_status pblock_lamb_step(const pb_lamb_config* cfg, int n_tensors,
                           const pb_lamb_tensor* tensors, pb_dtype copy_dtype,
                           float* trust_ratio, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!cfg) return fail(PB_ERR_INVALID_ARG, "cfg is NULL");
  if (!std::isfinite(cfg->lr)) return fail(PB_ERR_INVALID_ARG, "lr is not finite");
  if (!(cfg->beta1 >= 0.f && cfg->beta1 < 1.f) || !(cfg->beta2 >= 0.f && cfg->beta2 < 1.f))
    return fail(PB_ERR_INVALID_ARG, "beta1=%g, beta2=%g: each must be in [0, 1)",
                (double)cfg->beta1, (double)cfg->beta2);
  if (!(cfg->eps > 0.f) || !std::isfinite(cfg->eps))
    return fail(PB_ERR_INVALID_ARG, "eps=%g must be positive and finite", (double)cfg->eps);
  if (!std::isfinite(cfg->grad_scale)) return fail(PB_ERR_INVALID_ARG, "grad_scale is not finite");
  if (cfg->step < 1) return fail(PB_ERR_INVALID_ARG, "step=%d must be >= 1", cfg->step);
  if (cfg->bias_correction != 0 && cfg->bias_correction != 1)
    return fail(PB_ERR_INVALID_ARG, "bias_correction must be 0 or 1");
  if (copy_dtype != PB_BF16 && copy_dtype != PB_F32)
    return fail(PB_ERR_INVALID_ARG, "copy_dtype=%d", (int)copy_dtype);
  if (n_tensors < 1 || n_tensors > PB_LAMB_MAX_TENSORS)
    return fail(PB_ERR_INVALID_ARG, "n_tensors=%d must be in 1..%d", n_tensors,
                PB_LAMB_MAX_TENSORS);
  if (!tensors) return fail(PB_ERR_INVALID_ARG, "tensors is NULL");
  pb::LambTable t{};
  t.n = n_tensors;
  long long chunks = 0;
  for (int i = 0; i < n_tensors; ++i) {
    const pb_lamb_tensor& x = tensors[i];
    if (!(x.weight_decay >= 0.f) || !std::isfinite(x.weight_decay))
      return fail(PB_ERR_INVALID_ARG, "tensor %d: weight_decay=%g", i, (double)x.weight_decay);
    if (x.numel > 0) {
      const char* names[4] = {"param", "grad", "exp_avg", "exp_avg_sq"};
      const void* ptrs[4] = {x.param, x.grad, x.exp_avg, x.exp_avg_sq};
      for (int k = 0; k < 4; ++k)
        if (!ptrs[k] || (uintptr_t)ptrs[k] % 16)
          return fail(PB_ERR_INVALID_ARG, "tensor %d: %s is NULL or not 16-byte aligned", i,
                      names[k]);
      if (x.param_copy && (uintptr_t)x.param_copy % 16)
        return fail(PB_ERR_INVALID_ARG, "tensor %d: param_copy is not 16-byte aligned", i);
    }
    t.w[i] = x.param;
    t.g[i] = x.grad;
    t.m[i] = x.exp_avg;
    t.v[i] = x.exp_avg_sq;
    t.copy[i] = x.numel > 0 ? x.param_copy : nullptr;
    t.numel[i] = (long long)x.numel;
    t.wd[i] = x.weight_decay;
    t.chunk0[i] = (int)chunks;
    t.chunk_end[i] = (int)std::min<long long>(chunks + pb::lamb_chunks((long long)x.numel),
                                              INT32_MAX);
    chunks += pb::lamb_padded_chunks((long long)x.numel);
    if (chunks > INT32_MAX) return fail(PB_ERR_INVALID_ARG, "too many elements in one call");
  }
  t.chunk0[n_tensors] = (int)chunks;
  if (trust_ratio && (uintptr_t)trust_ratio % 4)
    return fail(PB_ERR_INVALID_ARG, "trust_ratio is not 4-byte aligned");
  const size_t need = pblock_lamb_workspace_bytes(n_tensors, tensors);
  if (!ws || (uintptr_t)ws % 256)
    return fail(PB_ERR_INVALID_ARG, "ws is NULL or not 256-byte aligned");
  if (ws_bytes < need) return fail(PB_ERR_WORKSPACE, "ws_bytes=%zu < %zu needed", ws_bytes, need);
  pb::LambScalars sc;
  sc.lr = cfg->lr;
  sc.beta1 = cfg->beta1;
  sc.beta2 = cfg->beta2;
  sc.eps = cfg->eps;
  sc.grad_scale = cfg->grad_scale;
  sc.c1 = cfg->bias_correction ? (float)(1.0 / (1.0 - pow((double)cfg->beta1, cfg->step))) : 1.f;
  sc.c2 = cfg->bias_correction ? (float)(1.0 / (1.0 - pow((double)cfg->beta2, cfg->step))) : 1.f;
  char* wsb = (char*)ws;
  float2* partial = (float2*)wsb;
  wsb += align256((size_t)chunks * sizeof(float2));
  double2* group = (double2*)wsb;
  wsb += align256((size_t)(chunks / pb::kLambGroup) * sizeof(double2));
  float* ratio = (float*)wsb;
  pb::launch_lamb(t, sc, copy_dtype == PB_BF16 ? pb::Dt::BF16 : pb::Dt::F32, partial, group,
                  ratio, trust_ratio, stream);
  return finish_launches();
}


const char* pblock_status_string(pb_status status) {
  switch (status) {
    case PB_OK: return "PB_OK";
    case PB_ERR_INVALID_ARG: return "PB_ERR_INVALID_ARG";
    case PB_ERR_UNSUPPORTED: return "PB_ERR_UNSUPPORTED";
    case PB_ERR_WORKSPACE: return "PB_ERR_WORKSPACE";
    case PB_ERR_HIP: return "PB_ERR_HIP";
  }
  return "PB_ERR_UNKNOWN";
}

const char* pblock_last_error(void) { return g_err; }

}  // extern "C"
