// LayerNorm forward / backward (fused, one pass over HBM each) and
// deterministic column sums for the bias and LN-parameter gradients.
//
// LN is the shared normalisation of the parallel block (MegaScale Section 3.1,
// Eq. 2); Section 3.3 fuses its fine-grained kernels into one.  Here one
// workgroup normalises one row held in registers: one HBM read of x, one
// write of h, statistics from wavefront reductions.
#include "common.h"
#include "kernels.h"

namespace pb {
namespace {

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
      load8(xr + c, v[j]);
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

// Rows are strided over the grid; each workgroup keeps running column sums of
// dh * xhat, dh and dy in registers and writes them once as a partial row
// (dy's column sum is db_out, the output bias gradient).  The raw loads of
// the next row are issued before the current row's reductions, so the
// memory latency of one row hides behind the arithmetic of the previous.
template <typename T>
struct RowRaw;
template <>
struct RowRaw<bf16> {
  u32x4 v;
  PB_DEV void load(const bf16* p) { v = *reinterpret_cast<const u32x4*>(p); }
  PB_DEV void get(float* o) const {
#pragma unroll
    for (int i = 0; i < 4; ++i) { o[2 * i] = lo_bf(v[i]); o[2 * i + 1] = hi_bf(v[i]); }
  }
};
template <>
struct RowRaw<float> {
  f32x4 a, b;
  PB_DEV void load(const float* p) {
    a = *reinterpret_cast<const f32x4*>(p);
    b = *reinterpret_cast<const f32x4*>(p + 4);
  }
  PB_DEV void get(float* o) const {
#pragma unroll
    for (int i = 0; i < 4; ++i) { o[i] = a[i]; o[4 + i] = b[i]; }
  }
};

template <typename T, int NV>
__global__ __launch_bounds__(kLnThreads) void ln_bwd_kernel(
    const T* __restrict__ x, const float* __restrict__ mean, const float* __restrict__ rstd,
    const T* __restrict__ gamma, const float* __restrict__ dh, const T* __restrict__ dy,
    T* __restrict__ dx, float* __restrict__ part_dg, float* __restrict__ part_db,
    float* __restrict__ part_dy, int rows, int H) {
  __shared__ float red[2][kLnWaves];
  float adg[NV][8], adb[NV][8], ady[NV][8];
  RowRaw<T> graw[NV];  // gamma, kept packed to save registers
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = (threadIdx.x + j * kLnThreads) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) adg[j][e] = adb[j][e] = ady[j][e] = 0.f;
    if (c < H) graw[j].load(gamma + c);
  }
  const float inv_h = 1.0f / (float)H;
  RowRaw<T> nx[NV], ny[NV];
  RowRaw<float> nd[NV];
  auto fetch = [&](int row) {
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int c = (threadIdx.x + j * kLnThreads) * 8;
      if (c < H) {
        nx[j].load(x + (size_t)row * H + c);
        nd[j].load(dh + (size_t)row * H + c);
        ny[j].load(dy + (size_t)row * H + c);
      }
    }
  };
  int row = blockIdx.x;
  if (row < rows) fetch(row);
  for (; row < rows; row += gridDim.x) {
    // the current row stays packed; values are unpacked where they are used
    RowRaw<T> cx[NV], cy[NV];
    RowRaw<float> cd[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      cx[j] = nx[j];
      cd[j] = nd[j];
      cy[j] = ny[j];
    }
    if (row + (int)gridDim.x < rows) fetch(row + gridDim.x);
    const float mu = mean[row], rs = rstd[row];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int c = (threadIdx.x + j * kLnThreads) * 8;
      if (c < H) {
        float xv[8], d[8], r[8], gm[8];
        cx[j].get(xv);
        cd[j].get(d);
        cy[j].get(r);
        graw[j].get(gm);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xh = (xv[e] - mu) * rs;
          adg[j][e] += d[e] * xh;
          adb[j][e] += d[e];
          ady[j][e] += r[e];
          const float g = gm[e] * d[e];
          s1 += g;
          s2 += g * xh;
        }
      }
    }
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
      red[0][w] = s1;
      red[1][w] = s2;
    }
    __syncthreads();
    float t1 = 0.f, t2 = 0.f;
#pragma unroll
    for (int i = 0; i < kLnWaves; ++i) {
      t1 += red[0][i];
      t2 += red[1][i];
    }
    __syncthreads();
    const float m1 = t1 * inv_h, m2 = t2 * inv_h;
    T* dxr = dx + (size_t)row * H;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int c = (threadIdx.x + j * kLnThreads) * 8;
      if (c < H) {
        float xv[8], d[8], r[8], gm[8], o[8];
        cx[j].get(xv);
        cd[j].get(d);
        cy[j].get(r);
        graw[j].get(gm);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xh = (xv[e] - mu) * rs;
          o[e] = r[e] + rs * (gm[e] * d[e] - m1 - xh * m2);
        }
        store8(dxr + c, o);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = (threadIdx.x + j * kLnThreads) * 8;
    if (c < H) {
      store8(part_dg + (size_t)blockIdx.x * H + c, adg[j]);
      store8(part_db + (size_t)blockIdx.x * H + c, adb[j]);
      store8(part_dy + (size_t)blockIdx.x * H + c, ady[j]);
    }
  }
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

__global__ __launch_bounds__(256) void colsum_stage2(const float* __restrict__ part, int chunks,
                                                     int cols, float* __restrict__ out) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= cols) return;
  float t = 0.f;
  for (int i = 0; i < chunks; ++i) t += part[(size_t)i * cols + c];
  out[c] = t;
}

template <typename T>
void colsum_impl(const T* src, int ld, int rows, int cols, float* part, float* out,
                 hipStream_t s) {
  const int chunks = colsum_chunks(rows);
  const int rpc = (rows + chunks - 1) / chunks;
  dim3 g1((cols + kColWidth - 1) / kColWidth, chunks);
  colsum_stage1<T><<<g1, kColThreads, 0, s>>>(src, ld, rows, cols, rpc, part);
  colsum_stage2<<<(cols + 255) / 256, 256, 0, s>>>(part, chunks, cols, out);
}

template <typename T, int NV>
void ln_fwd_nv(const void* x, const void* gamma, const void* beta, void* h, float* mean,
               float* rstd, int rows, int H, float eps, hipStream_t s) {
  ln_fwd_kernel<T, NV><<<rows, kLnThreads, 0, s>>>((const T*)x, (const T*)gamma,
                                                   (const T*)beta, (T*)h, mean, rstd, H, eps);
}

template <typename T, int NV>
void ln_bwd_nv(const void* x, const float* mean, const float* rstd, const void* gamma,
               const float* dh, const void* dy, void* dx, float* pdg, float* pdb, float* pdy,
               int rows, int H, hipStream_t s) {
  ln_bwd_kernel<T, NV><<<ln_backward_blocks(rows), kLnThreads, 0, s>>>(
      (const T*)x, mean, rstd, (const T*)gamma, dh, (const T*)dy, (T*)dx, pdg, pdb, pdy, rows,
      H);
}

template <typename T>
void ln_fwd_t(const void* x, const void* gamma, const void* beta, void* h, float* mean,
              float* rstd, int rows, int H, float eps, hipStream_t s) {
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

template <typename T>
void ln_bwd_t(const void* x, const float* mean, const float* rstd, const void* gamma,
              const float* dh, const void* dy, void* dx, float* pdg, float* pdb, float* pdy,
              int rows, int H, hipStream_t s) {
  const int nv = (H + kLnThreads * 8 - 1) / (kLnThreads * 8);
  switch (nv) {
    case 1: ln_bwd_nv<T, 1>(x, mean, rstd, gamma, dh, dy, dx, pdg, pdb, pdy, rows, H, s); break;
    case 2: ln_bwd_nv<T, 2>(x, mean, rstd, gamma, dh, dy, dx, pdg, pdb, pdy, rows, H, s); break;
    case 3: ln_bwd_nv<T, 3>(x, mean, rstd, gamma, dh, dy, dx, pdg, pdb, pdy, rows, H, s); break;
    case 4: ln_bwd_nv<T, 4>(x, mean, rstd, gamma, dh, dy, dx, pdg, pdb, pdy, rows, H, s); break;
    case 5: ln_bwd_nv<T, 5>(x, mean, rstd, gamma, dh, dy, dx, pdg, pdb, pdy, rows, H, s); break;
    case 6: ln_bwd_nv<T, 6>(x, mean, rstd, gamma, dh, dy, dx, pdg, pdb, pdy, rows, H, s); break;
    case 7: ln_bwd_nv<T, 7>(x, mean, rstd, gamma, dh, dy, dx, pdg, pdb, pdy, rows, H, s); break;
    default: ln_bwd_nv<T, 8>(x, mean, rstd, gamma, dh, dy, dx, pdg, pdb, pdy, rows, H, s); break;
  }
}

}  // namespace

int ln_backward_blocks(int rows) { return rows < 256 ? rows : 256; }

void launch_ln_forward(Dt dt, const void* x, const void* gamma, const void* beta, void* h,
                       float* mean, float* rstd, int rows, int H, float eps, hipStream_t s) {
  if (dt == Dt::BF16)
    ln_fwd_t<bf16>(x, gamma, beta, h, mean, rstd, rows, H, eps, s);
  else
    ln_fwd_t<float>(x, gamma, beta, h, mean, rstd, rows, H, eps, s);
}

void launch_ln_backward(Dt dt, const void* x, const float* mean, const float* rstd,
                        const void* gamma, const float* dh, const void* dy, void* dx,
                        float* part_dgamma, float* part_dbeta, float* part_dy, int rows, int H,
                        hipStream_t s) {
  if (dt == Dt::BF16)
    ln_bwd_t<bf16>(x, mean, rstd, gamma, dh, dy, dx, part_dgamma, part_dbeta, part_dy, rows, H,
                   s);
  else
    ln_bwd_t<float>(x, mean, rstd, gamma, dh, dy, dx, part_dgamma, part_dbeta, part_dy, rows,
                    H, s);
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

}  // namespace pb
