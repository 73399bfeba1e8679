// LayerNorm forward / backward (fused, one pass over HBM each) and
// deterministic column sums for the bias and LN-parameter gradients.
//
// LN is the shared normalisation of the parallel block (MegaScale Section 3.1,
// Eq. 2); Section 3.3 fuses its fine-grained kernels into one.  Forward: one
// workgroup normalises one row held in registers: one HBM read of x, one
// write of h, statistics from wavefront reductions.  Backward: the two row
// reductions it needs are formed by the dh GEMM's epilogue (Epi::LnGrad), so
// the kernel here is column-parallel and streams x, dh and dy once.
#include "common.h"
#include "kernels.h"

namespace pb {
namespace {

// Eight elements of data read once and not again soon (x in the forward;
// x, dh and dy in the backward): non-temporal loads keep them from pushing
// out of the caches what the next kernels reuse (h for the in-projection,
// dZ for the column sums and dW_in).  Measured: LN forward 34 -> 27 us,
// db_in 20 -> 15 us at the 175B share.
template <typename T> PB_DEV void load8_stream(const T* p, float* v);
template <> PB_DEV void load8_stream<bf16>(const bf16* p, float* v) {
  const u32x4 w = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
#pragma unroll
  for (int i = 0; i < 4; ++i) { v[2 * i] = lo_bf(w[i]); v[2 * i + 1] = hi_bf(w[i]); }
}
template <> PB_DEV void load8_stream<float>(const float* p, float* v) {
  const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
  const f32x4 b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + 4));
#pragma unroll
  for (int i = 0; i < 4; ++i) { v[i] = a[i]; v[4 + i] = b[i]; }
}

// Eight elements as loaded (packed bf16, or two fp32 quads, read once:
// non-temporal), unpacked where they are used: packed, a bf16 batch of rows
// takes half the registers.
template <typename T> struct Raw8;
template <> struct Raw8<bf16> {
  u32x4 w;
  PB_DEV void load(const bf16* p) {
    w = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  }
  PB_DEV float operator[](int e) const { return (e & 1) ? hi_bf(w[e >> 1]) : lo_bf(w[e >> 1]); }
};
template <> struct Raw8<float> {
  f32x4 a, b;
  PB_DEV void load(const float* p) {
    a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
    b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + 4));
  }
  PB_DEV float operator[](int e) const { return e < 4 ? a[e] : b[e - 4]; }
};

constexpr int kLnThreads = 512;
constexpr int kLnWaves = kLnThreads / 64;

// Sum of v over the workgroup; every thread gets the result.
template <int NW>
PB_DEV float block_sum(float v, float* scratch) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) scratch[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) t += scratch[i];
  __syncthreads();
  return t;
}

template <typename T, int NV>
__global__ __launch_bounds__(kLnThreads) void ln_fwd_kernel(const T* __restrict__ x,
                                                            const T* __restrict__ gamma,
                                                            const T* __restrict__ beta,
                                                            T* __restrict__ h,
                                                            float* __restrict__ mean_out,
                                                            float* __restrict__ rstd_out, int H,
                                                            float eps) {
  __shared__ float red[kLnWaves];
  const size_t row = blockIdx.x;
  const T* xr = x + row * H;
  float v[NV][8];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = (threadIdx.x + j * kLnThreads) * 8;
    if (c < H) {
      load8_stream(xr + c, v[j]);
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[j][e];
    }
  }
  const float mu = block_sum<kLnWaves>(s, red) / (float)H;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = (threadIdx.x + j * kLnThreads) * 8;
    if (c < H) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = v[j][e] - mu;
        q += d * d;
      }
    }
  }
  const float var = block_sum<kLnWaves>(q, red) / (float)H;
  const float rs = 1.0f / sqrtf(var + eps);
  T* hr = h + row * H;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = (threadIdx.x + j * kLnThreads) * 8;
    if (c < H) {
      float g[8], b[8], o[8];
      load8(gamma + c, g);
      load8(beta + c, b);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (v[j][e] - mu) * rs * g[e] + b[e];
      store8(hr + c, o);
    }
  }
  if (threadIdx.x == 0) {
    mean_out[row] = mu;
    rstd_out[row] = rs;
  }
}

// One wave per row for bf16 rows of NC * 512 columns: the row stays in
// registers as packed bf16 (NC 16-byte chunks per lane, each load
// instruction covering 1 KB of the row), the statistics come from wave
// reductions with no workgroup barrier, and a 2048-row input has every row
// in flight at once (2048 waves on 256 CUs) instead of two rounds of
// 512-thread workgroups.  Same two passes as above (mean, then the sum of
// squared deviations), fp32 throughout.
// An empty asm that claims to rewrite the packed row, so values unpacked
// from it before this point are not reused after it.
template <int NC>
PB_DEV void keep_packed(u32x4 (&w)[NC]) {
#pragma unroll
  for (int j = 0; j < NC; ++j) asm volatile("" : "+v"(w[j]));
}

template <int NC>
__global__ __launch_bounds__(256) void ln_fwd_wave_bf16(const bf16* __restrict__ x,
                                                        const bf16* __restrict__ gamma,
                                                        const bf16* __restrict__ beta,
                                                        bf16* __restrict__ h,
                                                        float* __restrict__ mean_out,
                                                        float* __restrict__ rstd_out, int rows,
                                                        float eps) {
  constexpr int H = NC * 512;
  const int lane = threadIdx.x & 63;
  const int row = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6);
  if (row >= rows) return;  // wave-uniform
  const bf16* xr = x + (size_t)row * H;
  u32x4 w[NC];
#pragma unroll
  for (int j = 0; j < NC; ++j)
    w[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(xr + (j * 64 + lane) * 8));
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NC; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) s += lo_bf(w[j][i]) + hi_bf(w[j][i]);
  const float mu = wave_sum(s) / (float)H;
  // each pass unpacks the row again: kept unpacked from one pass to the
  // next, the row would need twice the registers
  keep_packed<NC>(w);
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < NC; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float d0 = lo_bf(w[j][i]) - mu, d1 = hi_bf(w[j][i]) - mu;
      q += d0 * d0 + d1 * d1;
    }
  const float rs = 1.0f / sqrtf(wave_sum(q) / (float)H + eps);
  keep_packed<NC>(w);
  bf16* hr = h + (size_t)row * H;
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int c = (j * 64 + lane) * 8;
    float g[8], b[8], o[8];
    load8(gamma + c, g);
    load8(beta + c, b);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = (lo_bf(w[j][i]) - mu) * rs * g[2 * i] + b[2 * i];
      o[2 * i + 1] = (hi_bf(w[j][i]) - mu) * rs * g[2 * i + 1] + b[2 * i + 1];
    }
    store8(hr + c, o);
  }
  if (lane == 0) {
    mean_out[row] = mu;
    rstd_out[row] = rs;
  }
}

// Column-parallel LayerNorm backward.  The row terms sum gamma dh and
// sum gamma dh xhat arrive as 64-column group partials from the dh GEMM's
// epilogue, so no row-wide reduction is left here: each workgroup owns 16
// rows x 2048 columns, first folds its rows' partials (in a fixed order) into
// mean(g) and mean(g xhat), then streams x, dh and dy once, writes dx, and
// keeps the column sums of dh xhat (dgamma), dh (dbeta) and dy (db_out) of
// its 16 rows in registers, written once as a partial row.
constexpr int kApplyRows = 16;
constexpr int kApplyThreads = 256;
constexpr int kApplyCols = kApplyThreads * 8;

template <typename T>
__global__ __launch_bounds__(kApplyThreads) void ln_bwd_apply(
    const T* __restrict__ x, const float* __restrict__ mean, const float* __restrict__ rstd,
    const T* __restrict__ gamma, const T* __restrict__ dh, const float2* __restrict__ rowpart,
    int ngroups, const T* __restrict__ dy, T* __restrict__ dx, float* __restrict__ part_dg,
    float* __restrict__ part_db, float* __restrict__ part_dy, int rows, int H) {
  __shared__ float stat[kApplyRows][4];  // mean(g), mean(g xhat), mean, rstd
  const int ncb = (H + kApplyCols - 1) / kApplyCols;
  const int cb = (int)blockIdx.x % ncb, chunk = (int)blockIdx.x / ncb;
  const int r0 = chunk * kApplyRows;
  const int nr = min(kApplyRows, rows - r0);
  const int c = (cb * kApplyThreads + threadIdx.x) * 8;
  const bool col_ok = c < H;
  float gm[8], adg[8], adb[8], ady[8];
  // the first rows' loads go out before the row terms are folded (they do
  // not depend on them), so their latency overlaps the fold and its barrier
  if (col_ok) load8(gamma + c, gm);
#pragma unroll
  for (int e = 0; e < 8; ++e) adg[e] = adb[e] = ady[e] = 0.f;
  // Rows in batches of kBatch, double-buffered: the next batch's loads are
  // issued before this batch's dx stores, so waiting for them never waits for
  // a store as well (one counter covers both; loaded one batch at a time
  // after the previous stores, every batch paid the full load latency).
  // bf16 rows are held packed, four to a batch (four batches per workgroup
  // instead of eight, with the same registers).
  constexpr int kBatch = sizeof(T) == 2 ? 4 : 2, kBatches = kApplyRows / kBatch;
  Raw8<T> xv[2][kBatch], dv[2][kBatch], yv[2][kBatch];
  auto load_batch = [&](int buf, int rb) {
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const size_t off = (size_t)(r0 + min(rb + i, nr - 1)) * H + c;
      xv[buf][i].load(x + off);
      dv[buf][i].load(dh + off);
      yv[buf][i].load(dy + off);
    }
  };
  if (col_ok) load_batch(0, 0);
  {
    // 16 threads per row, each summing every 16th group, then a butterfly
    const int rr = threadIdx.x >> 4, l = threadIdx.x & 15;
    float s1 = 0.f, s2 = 0.f;
    if (rr < nr)
      for (int g = l; g < ngroups; g += 16) {
        const float2 p = rowpart[(size_t)(r0 + rr) * ngroups + g];
        s1 += p.x;
        s2 += p.y;
      }
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) {
      s1 += __shfl_xor(s1, off, 16);
      s2 += __shfl_xor(s2, off, 16);
    }
    if (l == 0 && rr < kApplyRows) {
      stat[rr][0] = s1 / (float)H;
      stat[rr][1] = s2 / (float)H;
      stat[rr][2] = rr < nr ? mean[r0 + rr] : 0.f;
      stat[rr][3] = rr < nr ? rstd[r0 + rr] : 0.f;
    }
  }
  __syncthreads();
  if (!col_ok) return;

#pragma unroll
  for (int bt = 0; bt < kBatches; ++bt) {
    const int cur = bt & 1;
    if (bt + 1 < kBatches && (bt + 1) * kBatch < nr) load_batch(cur ^ 1, (bt + 1) * kBatch);
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int rr = bt * kBatch + i;
      if (rr < nr) {
        const size_t off = (size_t)(r0 + rr) * H + c;
        const float m1 = stat[rr][0], m2 = stat[rr][1], mu = stat[rr][2], rs = stat[rr][3];
        float o[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = dv[cur][i][e];
          const float xh = (xv[cur][i][e] - mu) * rs;
          adg[e] += d * xh;
          adb[e] += d;
          ady[e] += yv[cur][i][e];
          o[e] = yv[cur][i][e] + rs * (gm[e] * d - m1 - xh * m2);
        }
        {
          u32x4 wv;
#pragma unroll
          for (int q = 0; q < 4; ++q) wv[q] = pack_bf2(o[2 * q], o[2 * q + 1]);
          // dx is not read again here: streamed past the caches
          if constexpr (sizeof(T) == 2)
            __builtin_nontemporal_store(wv, reinterpret_cast<u32x4*>(dx + off));
          else
            store8(dx + off, o);
        }
      }
    }
  }
  const size_t prow = (size_t)chunk * H + c;
  store8(part_dg + prow, adg);
  store8(part_db + prow, adb);
  store8(part_dy + prow, ady);
}

// ------------------------------------------------------------ column sums
constexpr int kColThreads = 256;
constexpr int kColWidth = 512;  // columns per workgroup (8 per lane, 64 lanes)

int colsum_chunks(int rows) {
  int c = (rows + 63) / 64;
  return c < 1 ? 1 : (c > 32 ? 32 : c);
}

template <typename T>
__global__ __launch_bounds__(kColThreads) void colsum_stage1(const T* __restrict__ src, int ld,
                                                            int rows, int cols, int rows_per_chunk,
                                                            float* __restrict__ part) {
  __shared__ float red[kColThreads / 64][64][9];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = blockIdx.x * kColWidth + lane * 8;
  const int r0 = blockIdx.y * rows_per_chunk;
  const int r1 = min(rows, r0 + rows_per_chunk);
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (c < cols) {
    for (int r = r0 + w; r < r1; r += kColThreads / 64) {
      float v[8];
      load8(src + (size_t)r * ld + c, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += v[e];
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[w][lane][e] = acc[e];
  __syncthreads();
  if (w == 0 && c < cols) {
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float t = 0.f;
#pragma unroll
      for (int i = 0; i < kColThreads / 64; ++i) t += red[i][lane][e];
      o[e] = t;
    }
    store8(part + (size_t)blockIdx.y * cols + c, o);
  }
}

// Column sums of up to three fp32 [rows, cols] arrays (cols a multiple of
// 4), blockIdx.y picking the array: a workgroup covers 64 columns as 16
// column quads x 16 row groups; each thread adds rows g, g + 16, ... of its
// four columns, and the 16 group sums are added in a fixed order.  Many
// short, independent row walks keep enough loads in flight for the few
// hundred rows these arrays have.
struct Colsum3 {
  const float* src[3];
  float* out[3];
};
__global__ __launch_bounds__(256) void colsum_rows_f32(Colsum3 a, int ld, int rows, int cols) {
  __shared__ f32x4 red[16][16];
  const float* __restrict__ src = a.src[blockIdx.y];
  const int q = threadIdx.x & 15, g = threadIdx.x >> 4;
  const int c = (blockIdx.x * 16 + q) * 4;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (c < cols) {
#pragma unroll 8
    for (int r = g; r < rows; r += 16)
      acc += *reinterpret_cast<const f32x4*>(src + (size_t)r * ld + c);
  }
  red[g][q] = acc;
  __syncthreads();
  if (g == 0 && c < cols) {
    f32x4 t = red[0][q];
#pragma unroll
    for (int i = 1; i < 16; ++i) t += red[i][q];
    *reinterpret_cast<f32x4*>(a.out[blockIdx.y] + c) = t;
  }
}

template <typename T>
void colsum_impl(const T* src, int ld, int rows, int cols, float* part, float* out,
                 hipStream_t s) {
  const int chunks = colsum_chunks(rows);
  const int rpc = (rows + chunks - 1) / chunks;
  dim3 g1((cols + kColWidth - 1) / kColWidth, chunks);
  colsum_stage1<T><<<g1, kColThreads, 0, s>>>(src, ld, rows, cols, rpc, part);
  Colsum3 a{{part, nullptr, nullptr}, {out, nullptr, nullptr}};
  colsum_rows_f32<<<dim3((cols + 63) / 64, 1), 256, 0, s>>>(a, cols, chunks, cols);
}

template <typename T, int NV>
void ln_fwd_nv(const void* x, const void* gamma, const void* beta, void* h, float* mean,
               float* rstd, int rows, int H, float eps, hipStream_t s) {
  ln_fwd_kernel<T, NV><<<rows, kLnThreads, 0, s>>>((const T*)x, (const T*)gamma,
                                                   (const T*)beta, (T*)h, mean, rstd, H, eps);
}

template <int NC>
void ln_fwd_wave(const void* x, const void* gamma, const void* beta, void* h, float* mean,
                 float* rstd, int rows, float eps, hipStream_t s) {
  ln_fwd_wave_bf16<NC><<<(rows + 3) / 4, 256, 0, s>>>((const bf16*)x, (const bf16*)gamma,
                                                      (const bf16*)beta, (bf16*)h, mean, rstd,
                                                      rows, eps);
}

// bf16 rows of 512 NC columns for the NC instantiated here (H = 5120 and
// 12288 among them) take the wave-per-row kernel; true if launched.
bool ln_fwd_wave_dispatch(const void* x, const void* gamma, const void* beta, void* h,
                          float* mean, float* rstd, int rows, int H, float eps, hipStream_t s) {
  if (H % 512 != 0) return false;
  switch (H / 512) {
    case 4: ln_fwd_wave<4>(x, gamma, beta, h, mean, rstd, rows, eps, s); return true;
    case 8: ln_fwd_wave<8>(x, gamma, beta, h, mean, rstd, rows, eps, s); return true;
    case 10: ln_fwd_wave<10>(x, gamma, beta, h, mean, rstd, rows, eps, s); return true;
    case 12: ln_fwd_wave<12>(x, gamma, beta, h, mean, rstd, rows, eps, s); return true;
    case 16: ln_fwd_wave<16>(x, gamma, beta, h, mean, rstd, rows, eps, s); return true;
    case 24: ln_fwd_wave<24>(x, gamma, beta, h, mean, rstd, rows, eps, s); return true;
    default: return false;
  }
}

template <typename T>
void ln_fwd_t(const void* x, const void* gamma, const void* beta, void* h, float* mean,
              float* rstd, int rows, int H, float eps, hipStream_t s) {
  if constexpr (sizeof(T) == 2)
    if (ln_fwd_wave_dispatch(x, gamma, beta, h, mean, rstd, rows, H, eps, s)) return;
  const int nv = (H + kLnThreads * 8 - 1) / (kLnThreads * 8);
  switch (nv) {
    case 1: ln_fwd_nv<T, 1>(x, gamma, beta, h, mean, rstd, rows, H, eps, s); break;
    case 2: ln_fwd_nv<T, 2>(x, gamma, beta, h, mean, rstd, rows, H, eps, s); break;
    case 3: ln_fwd_nv<T, 3>(x, gamma, beta, h, mean, rstd, rows, H, eps, s); break;
    case 4: ln_fwd_nv<T, 4>(x, gamma, beta, h, mean, rstd, rows, H, eps, s); break;
    case 5: ln_fwd_nv<T, 5>(x, gamma, beta, h, mean, rstd, rows, H, eps, s); break;
    case 6: ln_fwd_nv<T, 6>(x, gamma, beta, h, mean, rstd, rows, H, eps, s); break;
    case 7: ln_fwd_nv<T, 7>(x, gamma, beta, h, mean, rstd, rows, H, eps, s); break;
    default: ln_fwd_nv<T, 8>(x, gamma, beta, h, mean, rstd, rows, H, eps, s); break;
  }
}

}  // namespace

void launch_ln_forward(Dt dt, const void* x, const void* gamma, const void* beta, void* h,
                       float* mean, float* rstd, int rows, int H, float eps, hipStream_t s) {
  if (dt == Dt::BF16)
    ln_fwd_t<bf16>(x, gamma, beta, h, mean, rstd, rows, H, eps, s);
  else
    ln_fwd_t<float>(x, gamma, beta, h, mean, rstd, rows, H, eps, s);
}

int ln_backward_chunks(int rows) { return (rows + kApplyRows - 1) / kApplyRows; }

void launch_ln_backward(Dt dt, const void* x, const float* mean, const float* rstd,
                        const void* gamma, const void* dh, const float2* rowpart,
                        const void* dy, void* dx, float* part_dgamma, float* part_dbeta,
                        float* part_dy, int rows, int H, hipStream_t s) {
  const unsigned grid = (unsigned)((H + kApplyCols - 1) / kApplyCols) * ln_backward_chunks(rows);
  const int ng = ln_row_groups(H);
  if (dt == Dt::BF16)
    ln_bwd_apply<bf16><<<grid, kApplyThreads, 0, s>>>(
        (const bf16*)x, mean, rstd, (const bf16*)gamma, (const bf16*)dh, rowpart, ng,
        (const bf16*)dy,
        (bf16*)dx, part_dgamma, part_dbeta, part_dy, rows, H);
  else
    ln_bwd_apply<float><<<grid, kApplyThreads, 0, s>>>(
        (const float*)x, mean, rstd, (const float*)gamma, (const float*)dh, rowpart, ng,
        (const float*)dy,
        (float*)dx, part_dgamma, part_dbeta, part_dy, rows, H);
}

size_t colsum_partial_floats(int rows, int cols) {
  return (size_t)colsum_chunks(rows) * (size_t)cols;
}

void launch_colsum(Dt dt, const void* src, int ld, int rows, int cols, float* part, float* out,
                   hipStream_t s) {
  if (dt == Dt::BF16)
    colsum_impl<bf16>((const bf16*)src, ld, rows, cols, part, out, s);
  else
    colsum_impl<float>((const float*)src, ld, rows, cols, part, out, s);
}

void launch_colsum_f32(const float* src, int ld, int rows, int cols, float* part, float* out,
                       hipStream_t s) {
  colsum_impl<float>(src, ld, rows, cols, part, out, s);
}

void launch_colsum3_f32(const float* a, const float* b, const float* c, int ld, int rows,
                        int cols, float* out_a, float* out_b, float* out_c, hipStream_t s) {
  Colsum3 args{{a, b, c}, {out_a, out_b, out_c}};
  colsum_rows_f32<<<dim3((cols + 63) / 64, 3), 256, 0, s>>>(args, ld, rows, cols);
}

}  // namespace pb
