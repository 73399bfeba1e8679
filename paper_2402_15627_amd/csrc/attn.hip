// Causal sliding-window attention (MegaScale Section 3.1, "Sliding window
// attention"), evaluated flash-style as Section 3.3 adopts FlashAttention-2:
// scores never reach HBM, softmax is computed online, and key tiles that lie
// wholly outside a query block's window are never visited, so the work is
// O(seq * window).  Query i sees key j iff 0 <= i - j < window.
//
// bf16 kernels (gfx950 MFMA 32x32x16).  Everything is computed transposed:
// the MFMA's "A" operand is the key (or d) side, so the 32 output columns a
// lane owns are 32 queries (forward, dQ) or 32 keys (dK/dV).  Each lane then
// holds all scores of ONE query; the softmax rescale is a per-lane scalar,
// the row maximum needs a single cross-half exchange, and the probabilities
// feed the next MFMA straight from the accumulator registers (the k-index
// order of that MFMA is permuted to match, and the LDS copy of the other
// operand is written in the same permuted order).
//   forward : S^T = K Q^T, O^T += V^T P^T         (LDS: K, V^T)
//   dK, dV  : S = Q K^T, dP = dO V^T,
//             dV^T += dO^T P, dK^T += Q^T dS       (LDS: Q, Q^T, dO, dO^T)
//   dQ      : S^T = K Q^T, dP^T = V dO^T,
//             dQ^T += K^T dS^T                     (LDS: K, K^T, V)
// The backward pass is split in two kernels so that no gradient needs atomic
// accumulation: results are deterministic.
//
// fp32 kernels: one thread per query (or key), plain loops; parity path.
#include "common.h"
#include "kernels.h"

namespace pb {
namespace {

constexpr int kAttnThreads = 256;  // four waves
constexpr int kTile = 64;          // keys (forward, dQ) or queries (dK/dV) per LDS tile
constexpr float kNegInf = -__builtin_huge_valf();

// ------------------------------------------------------------ LDS tiles
// Natural tile: 64 token rows x D, row r chunk c (8 elements) at
// r * (D/8) + (c ^ (r & 7)).
template <int D>
PB_DEV void load_nat(const bf16* __restrict__ base, int ld, int row0, int rows_valid, int tid,
                     u32x4* r) {
  constexpr int CPR = D / 8;
#pragma unroll
  for (int u = 0; u < CPR / 4; ++u) {
    const int ci = tid + kAttnThreads * u;
    const int row = ci / CPR, c = ci % CPR;
    const int t = row0 + row;
    r[u] = t < rows_valid ? *reinterpret_cast<const u32x4*>(base + (size_t)t * ld + 8 * c)
                          : u32x4{0, 0, 0, 0};
  }
}
template <int D>
PB_DEV void store_nat(u32x4* __restrict__ lds, int tid, const u32x4* r) {
  constexpr int CPR = D / 8;
#pragma unroll
  for (int u = 0; u < CPR / 4; ++u) {
    const int ci = tid + kAttnThreads * u;
    const int row = ci / CPR, c = ci % CPR;
    lds[row * CPR + (c ^ (row & 7))] = r[u];
  }
}
template <int D>
PB_DEV bf16x8 frag_nat(const u32x4* lds, int row, int c) {
  return __builtin_bit_cast(bf16x8, lds[row * (D / 8) + (c ^ (row & 7))]);
}

// Transposed tile: D rows (one per feature e) x 64 tokens.  Chunk c of row e
// holds tokens 16(c/2) + 4(c%2) + {0,1,2,3} then 16(c/2) + 8 + 4(c%2) +
// {0,1,2,3}: the k order in which an MFMA consumes probabilities straight
// from its accumulator registers.  Stored at e * 8 + (c ^ (e & 7)).
// Block bi (0 <= bi < D) = chunk bi & 7 of rows 8 (bi >> 3) .. +7.
PB_DEV int perm_token(int c, int e) { return 16 * (c >> 1) + 4 * (c & 1) + (e & 3) + 8 * (e >> 2); }

template <int D>
PB_DEV void load_t(const bf16* __restrict__ base, int ld, int row0, int rows_valid, int bi,
                   u32x4* r) {
  const int c = bi & 7, dg = bi >> 3;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int t = row0 + perm_token(c, e);
    r[e] = t < rows_valid ? *reinterpret_cast<const u32x4*>(base + (size_t)t * ld + 8 * dg)
                          : u32x4{0, 0, 0, 0};
  }
}
template <int D>
PB_DEV void store_t(u32x4* __restrict__ lds, int bi, const u32x4* r) {
  const int c = bi & 7, dg = bi >> 3;
  u32x4 t[8];
  transpose8x8(r, t);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int e = 8 * dg + i;
    lds[e * 8 + (c ^ (e & 7))] = t[i];
  }
}
PB_DEV bf16x8 frag_t(const u32x4* lds, int e, int c) {
  return __builtin_bit_cast(bf16x8, lds[e * 8 + (c ^ (e & 7))]);
}

// Probabilities for MFMA k-step s (16 tokens) from two 32-token accumulators.
PB_DEV bf16x8 probs_frag(const f32x16* p, int s) {
  const f32x16& a = p[s >> 1];
  const int o = 8 * (s & 1);
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (bf16)a[o + e];
  return r;
}

PB_DEV f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int e = 0; e < 16; ++e) z[e] = 0.f;
  return z;
}

// ============================================================== forward
template <int D>
__global__ __launch_bounds__(kAttnThreads, 1) void attn_fwd_bf16(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V, int ld,
    bf16* __restrict__ O, int ld_o, float* __restrict__ lse, int S, int H, int W, float scale) {
  constexpr int NB = 32 * 4;                 // queries per workgroup
  constexpr int NAT = kTile * D / 8;         // u32x4 per natural tile
  constexpr int TT = D * 8;                  // u32x4 per transposed tile
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  u32x4* const lds0 = (u32x4*)smem;
  auto kn = [&](int s) { return lds0 + s * (NAT + TT); };
  auto vt = [&](int s) { return lds0 + s * (NAT + TT) + NAT; };

  const int nqb = (S + NB - 1) / NB;
  const int q0 = (nqb - 1 - (int)blockIdx.x) * NB;  // longest rows first
  const int head = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 31, fh = lane >> 5;
  const size_t tok0 = (size_t)b * S;
  const bf16* qb = Q + tok0 * ld + head * D;
  const bf16* kb = K + tok0 * ld + head * D;
  const bf16* vb = V + tok0 * ld + head * D;

  const int qw0 = q0 + 32 * wave;
  const int q = qw0 + fr;
  bf16x8 qf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
    qf[ks] = q < S ? __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                    qb + (size_t)q * ld + 16 * ks + 8 * fh))
                   : bf16x8{};

  const float c2 = scale * kLog2e;
  float m_run = kNegInf, l_run = 0.f;
  f32x16 o[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) o[i] = zero16();

  const int q_last = min(q0 + NB - 1, S - 1);
  const int kv_begin = (max(0, q0 - W + 1) / kTile) * kTile;
  const int ntiles = (q_last - kv_begin) / kTile + 1;
  // wave's own key range
  const int w_lo = qw0 - W + 1, w_hi = min(qw0 + 31, S - 1);

  u32x4 rk[D / 32], rv[8];
  load_nat<D>(kb, ld, kv_begin, S, tid, rk);
  if (tid < D) load_t<D>(vb, ld, kv_begin, S, tid, rv);
  store_nat<D>(kn(0), tid, rk);
  if (tid < D) store_t<D>(vt(0), tid, rv);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int cur = t & 1;
    const int kv0 = kv_begin + t * kTile;
    if (t + 1 < ntiles) {
      load_nat<D>(kb, ld, kv0 + kTile, S, tid, rk);
      if (tid < D) load_t<D>(vb, ld, kv0 + kTile, S, tid, rv);
    }
    if (qw0 < S && kv0 <= w_hi && kv0 + kTile - 1 >= w_lo) {
      f32x16 s[2];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        s[h2] = zero16();
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks)
          s[h2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              frag_nat<D>(kn(cur), 32 * h2 + fr, 2 * ks + fh), qf[ks], s[h2], 0, 0, 0);
      }
      const bool full = (kv0 + kTile - 1 <= qw0) && (qw0 + 31 - kv0 < W) &&
                        (kv0 + kTile <= S) && (qw0 + 32 <= S);
      float mx = kNegInf;
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float x = s[h2][r] * c2;
          if (!full) {
            const int key = kv0 + 32 * h2 + 8 * (r >> 2) + 4 * fh + (r & 3);
            const int dist = q - key;
            if (dist < 0 || dist >= W || key >= S) x = kNegInf;
          }
          s[h2][r] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);
      const float m_use = m_new == kNegInf ? 0.f : m_new;
      const float alpha = exp2f(m_run - m_use);
      m_run = m_new;
      float ls = 0.f;
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = exp2f(s[h2][r] - m_use);
          s[h2][r] = p;
          ls += p;
        }
      l_run = l_run * alpha + ls;
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
#pragma unroll
        for (int e = 0; e < 16; ++e) o[db][e] *= alpha;
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2)
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_t(vt(cur), 32 * db + fr, 2 * s2 + fh),
                                                          probs_frag(s, s2), o[db], 0, 0, 0);
      }
    }
    if (t + 1 < ntiles) {
      store_nat<D>(kn(cur ^ 1), tid, rk);
      if (tid < D) store_t<D>(vt(cur ^ 1), tid, rv);
    }
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (q < S) {
    const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    bf16* orow = O + (tok0 + q) * ld_o + head * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v[4] = {o[db][4 * j] * inv, o[db][4 * j + 1] * inv, o[db][4 * j + 2] * inv,
                      o[db][4 * j + 3] * inv};
        store4(orow + 32 * db + 8 * j + 4 * fh, v);
      }
    if (fh == 0) {
      const float m_use = m_run == kNegInf ? 0.f : m_run;
      lse[((size_t)b * H + head) * S + q] = (m_use + log2f(l_tot)) * kLn2;
    }
  }
}

// ===================================================== backward: delta
template <typename T>
__global__ __launch_bounds__(256) void attn_delta_kernel(const T* __restrict__ O, int ld_o,
                                                         const T* __restrict__ dO, int ld_do,
                                                         float* __restrict__ delta, int B, int S,
                                                         int H, int D) {
  const int idx = blockIdx.x * 256 + threadIdx.x;  // (b, t, head)
  if (idx >= B * S * H) return;
  const int head = idx % H, bt = idx / H;
  const int b = bt / S, t = bt % S;
  const T* o = O + (size_t)bt * ld_o + head * D;
  const T* g = dO + (size_t)bt * ld_do + head * D;
  float acc = 0.f;
  for (int e = 0; e < D; e += 8) {
    float a[8], c[8];
    load8(o + e, a);
    load8(g + e, c);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc += a[i] * c[i];
  }
  delta[((size_t)b * H + head) * S + t] = acc;
}

// ====================================================== backward: dK, dV
template <int D>
__global__ __launch_bounds__(kAttnThreads, 1) void attn_dkdv_bf16(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V, int ld,
    const bf16* __restrict__ dO, int ld_o, const float* __restrict__ lse,
    const float* __restrict__ delta, bf16* __restrict__ dK, bf16* __restrict__ dV, int ld_d,
    int S, int H, int W, float scale) {
  constexpr int NB = 32 * 4;  // keys per workgroup
  constexpr int NAT = kTile * D / 8, TT = D * 8;
  constexpr int STAGE = 2 * NAT + 2 * TT + 2 * kTile / 4;  // in u32x4
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  auto qn = [&](int s) { return (u32x4*)smem + s * STAGE; };
  auto don = [&](int s) { return (u32x4*)smem + s * STAGE + NAT; };
  auto qt = [&](int s) { return (u32x4*)smem + s * STAGE + 2 * NAT; };
  auto dot_ = [&](int s) { return (u32x4*)smem + s * STAGE + 2 * NAT + TT; };
  auto lsd = [&](int s) { return (float*)((u32x4*)smem + s * STAGE + 2 * NAT + 2 * TT); };

  const int nkb = (S + NB - 1) / NB;
  const int k0 = (int)blockIdx.x * NB;
  (void)nkb;
  const int head = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 31, fh = lane >> 5;
  const size_t tok0 = (size_t)b * S;
  const bf16* qb = Q + tok0 * ld + head * D;
  const bf16* kb = K + tok0 * ld + head * D;
  const bf16* vb = V + tok0 * ld + head * D;
  const bf16* gb = dO + tok0 * ld_o + head * D;
  const float* lseb = lse + ((size_t)b * H + head) * S;
  const float* delb = delta + ((size_t)b * H + head) * S;

  const int kw0 = k0 + 32 * wave;
  const int key = kw0 + fr;
  bf16x8 kf[D / 16], vf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const size_t off = (size_t)key * ld + 16 * ks + 8 * fh;
    kf[ks] = key < S ? __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(kb + off)) : bf16x8{};
    vf[ks] = key < S ? __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(vb + off)) : bf16x8{};
  }
  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) dk[i] = dv[i] = zero16();

  const float c2 = scale * kLog2e;
  const int k_last = min(k0 + NB - 1, S - 1);
  const int q_end = min(S - 1, k_last + W - 1);
  const int ntiles = (q_end - k0) / kTile + 1;
  const int w_lo = kw0, w_hi = min(S - 1, kw0 + 31 + W - 1);  // queries this wave needs

  u32x4 rq[D / 32], rg[D / 32], rt[8];
  float rl = 0.f;
  auto load_stage = [&](int qs) {
    load_nat<D>(qb, ld, qs, S, tid, rq);
    load_nat<D>(gb, ld_o, qs, S, tid, rg);
    if (tid < D) load_t<D>(qb, ld, qs, S, tid, rt);
    else if (tid >= 128 && tid < 128 + D) load_t<D>(gb, ld_o, qs, S, tid - 128, rt);
    if (tid < kTile) rl = qs + tid < S ? lseb[qs + tid] * kLog2e : __builtin_huge_valf();
    else if (tid < 2 * kTile) rl = qs + tid - kTile < S ? delb[qs + tid - kTile] : 0.f;
  };
  auto store_stage = [&](int s) {
    store_nat<D>(qn(s), tid, rq);
    store_nat<D>(don(s), tid, rg);
    if (tid < D) store_t<D>(qt(s), tid, rt);
    else if (tid >= 128 && tid < 128 + D) store_t<D>(dot_(s), tid - 128, rt);
    if (tid < 2 * kTile) lsd(s)[tid] = rl;
  };
  load_stage(k0);
  store_stage(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int cur = t & 1;
    const int qs = k0 + t * kTile;
    if (t + 1 < ntiles) load_stage(qs + kTile);
    if (kw0 < S && qs <= w_hi && qs + kTile - 1 >= w_lo) {
      f32x16 p[2], ds[2];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        p[h2] = zero16();
        ds[h2] = zero16();
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          p[h2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              frag_nat<D>(qn(cur), 32 * h2 + fr, 2 * ks + fh), kf[ks], p[h2], 0, 0, 0);
          ds[h2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              frag_nat<D>(don(cur), 32 * h2 + fr, 2 * ks + fh), vf[ks], ds[h2], 0, 0, 0);
        }
      }
      // lane holds key `key` and queries qs + 32 h2 + 8 j + 4 fh + i (r = 4 j + i)
      const bool full = (qs >= kw0 + 31) && (qs + kTile - 1 - kw0 < W) && (qs + kTile <= S) &&
                        (kw0 + 32 <= S);
      const float* ls = lsd(cur);
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int ql = 32 * h2 + 8 * j + 4 * fh;
          const f32x4 L4 = *reinterpret_cast<const f32x4*>(ls + ql);
          const f32x4 D4 = *reinterpret_cast<const f32x4*>(ls + kTile + ql);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = 4 * j + i;
            float pv = exp2f(p[h2][r] * c2 - L4[i]);
            if (!full) {
              const int dist = qs + ql + i - key;
              if (dist < 0 || dist >= W || qs + ql + i >= S) pv = 0.f;
            }
            p[h2][r] = pv;
            ds[h2][r] = pv * (ds[h2][r] - D4[i]);
          }
        }
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
          dv[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_t(dot_(cur), 32 * db + fr, 2 * s2 + fh),
                                                           probs_frag(p, s2), dv[db], 0, 0, 0);
          dk[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_t(qt(cur), 32 * db + fr, 2 * s2 + fh),
                                                           probs_frag(ds, s2), dk[db], 0, 0, 0);
        }
    }
    if (t + 1 < ntiles) store_stage(cur ^ 1);
    __syncthreads();
  }

  if (key < S) {
    bf16* dkr = dK + (tok0 + key) * ld_d + head * D;
    bf16* dvr = dV + (tok0 + key) * ld_d + head * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float a[4], c[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          a[i] = dk[db][4 * j + i] * scale;
          c[i] = dv[db][4 * j + i];
        }
        store4(dkr + 32 * db + 8 * j + 4 * fh, a);
        store4(dvr + 32 * db + 8 * j + 4 * fh, c);
      }
  }
}

// ============================================================ backward: dQ
template <int D>
__global__ __launch_bounds__(kAttnThreads, 1) void attn_dq_bf16(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V, int ld,
    const bf16* __restrict__ dO, int ld_o, const float* __restrict__ lse,
    const float* __restrict__ delta, bf16* __restrict__ dQ, int ld_d, int S, int H, int W,
    float scale) {
  constexpr int NB = 32 * 4;
  constexpr int NAT = kTile * D / 8, TT = D * 8;
  constexpr int STAGE = 2 * NAT + TT;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  auto kn = [&](int s) { return (u32x4*)smem + s * STAGE; };
  auto vn = [&](int s) { return (u32x4*)smem + s * STAGE + NAT; };
  auto kt = [&](int s) { return (u32x4*)smem + s * STAGE + 2 * NAT; };

  const int nqb = (S + NB - 1) / NB;
  const int q0 = (nqb - 1 - (int)blockIdx.x) * NB;
  const int head = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 31, fh = lane >> 5;
  const size_t tok0 = (size_t)b * S;
  const bf16* qb = Q + tok0 * ld + head * D;
  const bf16* kb = K + tok0 * ld + head * D;
  const bf16* vb = V + tok0 * ld + head * D;
  const bf16* gb = dO + tok0 * ld_o + head * D;

  const int qw0 = q0 + 32 * wave;
  const int q = qw0 + fr;
  bf16x8 qf[D / 16], gf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    qf[ks] = q < S ? __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                    qb + (size_t)q * ld + 16 * ks + 8 * fh))
                   : bf16x8{};
    gf[ks] = q < S ? __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                    gb + (size_t)q * ld_o + 16 * ks + 8 * fh))
                   : bf16x8{};
  }
  const size_t row_off = ((size_t)b * H + head) * S;
  const float L2 = q < S ? lse[row_off + q] * kLog2e : 0.f;
  const float Dq = q < S ? delta[row_off + q] : 0.f;
  const float c2 = scale * kLog2e;

  f32x16 dq[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) dq[i] = zero16();

  const int q_last = min(q0 + NB - 1, S - 1);
  const int kv_begin = (max(0, q0 - W + 1) / kTile) * kTile;
  const int ntiles = (q_last - kv_begin) / kTile + 1;
  const int w_lo = qw0 - W + 1, w_hi = min(qw0 + 31, S - 1);

  u32x4 rk[D / 32], rv[D / 32], rt[8];
  auto load_stage = [&](int ks0) {
    load_nat<D>(kb, ld, ks0, S, tid, rk);
    load_nat<D>(vb, ld, ks0, S, tid, rv);
    if (tid < D) load_t<D>(kb, ld, ks0, S, tid, rt);
  };
  auto store_stage = [&](int s) {
    store_nat<D>(kn(s), tid, rk);
    store_nat<D>(vn(s), tid, rv);
    if (tid < D) store_t<D>(kt(s), tid, rt);
  };
  load_stage(kv_begin);
  store_stage(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int cur = t & 1;
    const int kv0 = kv_begin + t * kTile;
    if (t + 1 < ntiles) load_stage(kv0 + kTile);
    if (qw0 < S && kv0 <= w_hi && kv0 + kTile - 1 >= w_lo) {
      f32x16 p[2], ds[2];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        p[h2] = zero16();
        ds[h2] = zero16();
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          p[h2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              frag_nat<D>(kn(cur), 32 * h2 + fr, 2 * ks + fh), qf[ks], p[h2], 0, 0, 0);
          ds[h2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              frag_nat<D>(vn(cur), 32 * h2 + fr, 2 * ks + fh), gf[ks], ds[h2], 0, 0, 0);
        }
      }
      const bool full = (kv0 + kTile - 1 <= qw0) && (qw0 + 31 - kv0 < W) &&
                        (kv0 + kTile <= S) && (qw0 + 32 <= S);
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float pv = exp2f(p[h2][r] * c2 - L2);
          if (!full) {
            const int k = kv0 + 32 * h2 + 8 * (r >> 2) + 4 * fh + (r & 3);
            const int dist = q - k;
            if (dist < 0 || dist >= W || k >= S) pv = 0.f;
          }
          ds[h2][r] = pv * (ds[h2][r] - Dq);
        }
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2)
          dq[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_t(kt(cur), 32 * db + fr, 2 * s2 + fh),
                                                           probs_frag(ds, s2), dq[db], 0, 0, 0);
    }
    if (t + 1 < ntiles) store_stage(cur ^ 1);
    __syncthreads();
  }

  if (q < S) {
    bf16* dqr = dQ + (tok0 + q) * ld_d + head * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float a[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = dq[db][4 * j + i] * scale;
        store4(dqr + 32 * db + 8 * j + 4 * fh, a);
      }
  }
}

// ============================================================ fp32 path
template <int D>
__global__ __launch_bounds__(64) void attn_fwd_f32(const float* __restrict__ Q,
                                                   const float* __restrict__ K,
                                                   const float* __restrict__ V, int ld,
                                                   float* __restrict__ O, int ld_o,
                                                   float* __restrict__ lse, int S, int H, int W,
                                                   float scale) {
  const int q = blockIdx.x * 64 + threadIdx.x, head = blockIdx.y, b = blockIdx.z;
  if (q >= S) return;
  const size_t tok0 = (size_t)b * S;
  const float* qr = Q + (tok0 + q) * ld + head * D;
  float qv[D], acc[D];
  for (int e = 0; e < D; ++e) { qv[e] = qr[e]; acc[e] = 0.f; }
  float m = kNegInf, l = 0.f;
  for (int j = max(0, q - W + 1); j <= q; ++j) {
    const float* kr = K + (tok0 + j) * ld + head * D;
    const float* vr = V + (tok0 + j) * ld + head * D;
    float s = 0.f;
    for (int e = 0; e < D; ++e) s = fmaf(qv[e], kr[e], s);
    s *= scale;
    const float mn = fmaxf(m, s);
    const float a = expf(m - mn), p = expf(s - mn);
    l = l * a + p;
    for (int e = 0; e < D; ++e) acc[e] = acc[e] * a + p * vr[e];
    m = mn;
  }
  float* orow = O + (tok0 + q) * ld_o + head * D;
  for (int e = 0; e < D; ++e) orow[e] = acc[e] / l;
  lse[((size_t)b * H + head) * S + q] = m + logf(l);
}

template <int D>
__global__ __launch_bounds__(64) void attn_dq_f32(const float* __restrict__ Q,
                                                  const float* __restrict__ K,
                                                  const float* __restrict__ V, int ld,
                                                  const float* __restrict__ dO, int ld_o,
                                                  const float* __restrict__ lse,
                                                  const float* __restrict__ delta,
                                                  float* __restrict__ dQ, int ld_d, int S, int H,
                                                  int W, float scale) {
  const int q = blockIdx.x * 64 + threadIdx.x, head = blockIdx.y, b = blockIdx.z;
  if (q >= S) return;
  const size_t tok0 = (size_t)b * S;
  const float* qr = Q + (tok0 + q) * ld + head * D;
  const float* gr = dO + (tok0 + q) * ld_o + head * D;
  float qv[D], gv[D], acc[D];
  for (int e = 0; e < D; ++e) { qv[e] = qr[e]; gv[e] = gr[e]; acc[e] = 0.f; }
  const size_t ro = ((size_t)b * H + head) * S + q;
  const float L = lse[ro], Dq = delta[ro];
  for (int j = max(0, q - W + 1); j <= q; ++j) {
    const float* kr = K + (tok0 + j) * ld + head * D;
    const float* vr = V + (tok0 + j) * ld + head * D;
    float s = 0.f, dp = 0.f;
    for (int e = 0; e < D; ++e) {
      s = fmaf(qv[e], kr[e], s);
      dp = fmaf(gv[e], vr[e], dp);
    }
    const float ds = expf(s * scale - L) * (dp - Dq);
    for (int e = 0; e < D; ++e) acc[e] = fmaf(ds, kr[e], acc[e]);
  }
  float* out = dQ + (tok0 + q) * ld_d + head * D;
  for (int e = 0; e < D; ++e) out[e] = acc[e] * scale;
}

template <int D>
__global__ __launch_bounds__(64) void attn_dkdv_f32(const float* __restrict__ Q,
                                                    const float* __restrict__ K,
                                                    const float* __restrict__ V, int ld,
                                                    const float* __restrict__ dO, int ld_o,
                                                    const float* __restrict__ lse,
                                                    const float* __restrict__ delta,
                                                    float* __restrict__ dK, float* __restrict__ dV,
                                                    int ld_d, int S, int H, int W, float scale) {
  const int j = blockIdx.x * 64 + threadIdx.x, head = blockIdx.y, b = blockIdx.z;
  if (j >= S) return;
  const size_t tok0 = (size_t)b * S;
  const float* kr = K + (tok0 + j) * ld + head * D;
  const float* vr = V + (tok0 + j) * ld + head * D;
  float kv[D], vv[D], dk[D], dv[D];
  for (int e = 0; e < D; ++e) { kv[e] = kr[e]; vv[e] = vr[e]; dk[e] = 0.f; dv[e] = 0.f; }
  const size_t ro = ((size_t)b * H + head) * S;
  const int i_end = min(S - 1, j + W - 1);
  for (int i = j; i <= i_end; ++i) {
    const float* qr = Q + (tok0 + i) * ld + head * D;
    const float* gr = dO + (tok0 + i) * ld_o + head * D;
    float s = 0.f, dp = 0.f;
    for (int e = 0; e < D; ++e) {
      s = fmaf(qr[e], kv[e], s);
      dp = fmaf(gr[e], vv[e], dp);
    }
    const float p = expf(s * scale - lse[ro + i]);
    const float ds = p * (dp - delta[ro + i]);
    for (int e = 0; e < D; ++e) {
      dv[e] = fmaf(p, gr[e], dv[e]);
      dk[e] = fmaf(ds, qr[e], dk[e]);
    }
  }
  float* dko = dK + (tok0 + j) * ld_d + head * D;
  float* dvo = dV + (tok0 + j) * ld_d + head * D;
  for (int e = 0; e < D; ++e) {
    dko[e] = dk[e] * scale;
    dvo[e] = dv[e];
  }
}

template <int D>
size_t fwd_lds() { return 2 * ((size_t)kTile * D / 8 + (size_t)D * 8) * 16; }
template <int D>
size_t dkdv_lds() { return 2 * (2 * (size_t)kTile * D / 8 + 2 * (size_t)D * 8 + 2 * kTile / 4) * 16; }
template <int D>
size_t dq_lds() { return 2 * (2 * (size_t)kTile * D / 8 + (size_t)D * 8) * 16; }

template <int D>
void fwd_d(Dt dt, const AttnShape& a, const void* q, const void* k, const void* v, int ld,
           void* o, int ld_o, float* lse, hipStream_t s) {
  const float scale = 1.0f / sqrtf((float)D);
  if (dt == Dt::BF16) {
    dim3 g((a.seq + 127) / 128, a.heads, a.batch);
    attn_fwd_bf16<D><<<g, kAttnThreads, fwd_lds<D>(), s>>>(
        (const bf16*)q, (const bf16*)k, (const bf16*)v, ld, (bf16*)o, ld_o, lse, a.seq, a.heads,
        a.window, scale);
  } else {
    dim3 g((a.seq + 63) / 64, a.heads, a.batch);
    attn_fwd_f32<D><<<g, 64, 0, s>>>((const float*)q, (const float*)k, (const float*)v, ld,
                                     (float*)o, ld_o, lse, a.seq, a.heads, a.window, scale);
  }
}

template <int D>
void bwd_d(Dt dt, const AttnShape& a, const void* q, const void* k, const void* v, int ld,
           const void* o, int ld_o, const void* d_o, int ld_do, const float* lse, float* delta,
           void* dq, void* dk, void* dv, int ld_d, hipStream_t s) {
  const float scale = 1.0f / sqrtf((float)D);
  const int nrows = a.batch * a.seq * a.heads;
  if (dt == Dt::BF16) {
    attn_delta_kernel<bf16><<<(nrows + 255) / 256, 256, 0, s>>>(
        (const bf16*)o, ld_o, (const bf16*)d_o, ld_do, delta, a.batch, a.seq, a.heads, D);
    dim3 g((a.seq + 127) / 128, a.heads, a.batch);
    attn_dkdv_bf16<D><<<g, kAttnThreads, dkdv_lds<D>(), s>>>(
        (const bf16*)q, (const bf16*)k, (const bf16*)v, ld, (const bf16*)d_o, ld_do, lse, delta,
        (bf16*)dk, (bf16*)dv, ld_d, a.seq, a.heads, a.window, scale);
    attn_dq_bf16<D><<<g, kAttnThreads, dq_lds<D>(), s>>>(
        (const bf16*)q, (const bf16*)k, (const bf16*)v, ld, (const bf16*)d_o, ld_do, lse, delta,
        (bf16*)dq, ld_d, a.seq, a.heads, a.window, scale);
  } else {
    attn_delta_kernel<float><<<(nrows + 255) / 256, 256, 0, s>>>(
        (const float*)o, ld_o, (const float*)d_o, ld_do, delta, a.batch, a.seq, a.heads, D);
    dim3 g((a.seq + 63) / 64, a.heads, a.batch);
    attn_dq_f32<D><<<g, 64, 0, s>>>((const float*)q, (const float*)k, (const float*)v, ld,
                                    (const float*)d_o, ld_do, lse, delta, (float*)dq, ld_d,
                                    a.seq, a.heads, a.window, scale);
    attn_dkdv_f32<D><<<g, 64, 0, s>>>((const float*)q, (const float*)k, (const float*)v, ld,
                                      (const float*)d_o, ld_do, lse, delta, (float*)dk,
                                      (float*)dv, ld_d, a.seq, a.heads, a.window, scale);
  }
}

}  // namespace

void launch_attn_forward(Dt dt, const AttnShape& a, const void* q, const void* k, const void* v,
                         int ld_qkv, void* o, int ld_o, float* lse, hipStream_t s) {
  if (a.head_dim == 64) fwd_d<64>(dt, a, q, k, v, ld_qkv, o, ld_o, lse, s);
  else fwd_d<128>(dt, a, q, k, v, ld_qkv, o, ld_o, lse, s);
}

void launch_attn_backward(Dt dt, const AttnShape& a, const void* q, const void* k, const void* v,
                          int ld_qkv, const void* o, int ld_o, const void* d_o, int ld_do,
                          const float* lse, float* delta, void* dq, void* dk, void* dv, int ld_d,
                          hipStream_t s) {
  if (a.head_dim == 64)
    bwd_d<64>(dt, a, q, k, v, ld_qkv, o, ld_o, d_o, ld_do, lse, delta, dq, dk, dv, ld_d, s);
  else
    bwd_d<128>(dt, a, q, k, v, ld_qkv, o, ld_o, d_o, ld_do, lse, delta, dq, dk, dv, ld_d, s);
}

}  // namespace pb
