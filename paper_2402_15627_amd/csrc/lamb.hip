// One LAMB optimizer step over up to kLambMaxTensors fp32 tensors (the
// layer-wise trust-ratio method the paper trains with, Section 3.1 "LAMB
// optimizer"; You et al. 2020).  HBM-bound: two streaming passes over the
// concatenated elements (chunks of kLambChunk elements, one float4 of each
// array per thread), with a two-level norm reduction between them.
//
//   1. moments: g = grad_scale grad; m, v updated in place; the direction
//      u = m^ / (sqrt(v^) + eps) + lambda w is formed and the chunk's sums
//      of w^2 and u^2 are written as one partial per chunk (u itself is not
//      stored).
//   2. ratio:   the partials are summed in groups of kLambGroup chunks
//      (each tensor's chunks start at a group boundary), then one workgroup
//      per tensor folds its groups, in fixed orders and in fp64, into
//      ratio = ||w|| / ||u|| (1 if either is 0).
//   3. apply:   u is recomputed from the stored m, v and the unchanged w by
//      the same code as in 1, w -= lr ratio u, and the updated weights are
//      also written in the model's storage type when a copy is requested.
//
// Per element: 16 bytes read and 8 written in 1; 12 read and 4 (+2 or 4
// for the copy) written in 3.  Results do not depend on timing: no atomics,
// fixed reduction orders.
#include "common.h"
#include "kernels.h"

namespace pb {
namespace {

constexpr int kLambThreads = 256;
static_assert(kLambChunk == 4 * kLambThreads, "one float4 per thread and array");

PB_DEV int tensor_of(const LambTable& t, int chunk) {
  int ti = 0;
#pragma unroll 1
  for (int i = 1; i < t.n; ++i)
    if (chunk >= t.chunk0[i]) ti = i;
  return ti;
}

// The update direction of one element (shared by both passes so that the
// recomputed u is bit-identical to the one whose norm was taken).
PB_DEV float lamb_dir(const LambScalars& sc, float m1, float v1, float w, float wd) {
  const float mh = m1 * sc.c1;
  const float vh = v1 * sc.c2;
  return __builtin_fmaf(wd, w, mh / (__builtin_sqrtf(vh) + sc.eps));
}

// Streaming accesses: every element is touched once per pass, so loads and
// stores bypass the caches' normal retention (measured +10% over ordinary
// accesses on these passes).
PB_DEV f32x4 ld_stream(const float* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
}
PB_DEV void st_stream(float* p, const f32x4& v) {
  __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(p));
}

template <typename T>
PB_DEV T block_sum(T v, T* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  T s = 0;
  if (threadIdx.x == 0) {
#pragma unroll
    for (int i = 0; i < kLambThreads / 64; ++i) s += red[i];
  }
  __syncthreads();
  return s;  // valid in thread 0
}

__global__ __launch_bounds__(kLambThreads) void lamb_moments_kernel(LambTable t, LambScalars sc,
                                                                    float2* __restrict__ partial) {
  __shared__ float red[2][kLambThreads / 64];
  const int c = blockIdx.x;
  const int ti = tensor_of(t, c);
  if (c >= t.chunk_end[ti]) {  // padding up to the next group of chunks
    if (threadIdx.x == 0) partial[c] = float2{0.f, 0.f};
    return;
  }
  const long long n = t.numel[ti];
  const long long e = (long long)(c - t.chunk0[ti]) * kLambChunk + 4 * threadIdx.x;
  const float* __restrict__ gp = t.g[ti];
  const float* __restrict__ wp = t.w[ti];
  float* __restrict__ mp = t.m[ti];
  float* __restrict__ vp = t.v[ti];
  const float wd = t.wd[ti];
  const float b1 = sc.beta1, b2 = sc.beta2, a1 = 1.0f - sc.beta1, a2 = 1.0f - sc.beta2;
  float sw = 0.f, su = 0.f;
  if (e + 4 <= n) {
    const f32x4 g4 = ld_stream(gp + e);
    const f32x4 w4 = ld_stream(wp + e);
    f32x4 m4 = ld_stream(mp + e);
    f32x4 v4 = ld_stream(vp + e);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float g = g4[k] * sc.grad_scale;
      m4[k] = b1 * m4[k] + a1 * g;
      v4[k] = b2 * v4[k] + a2 * (g * g);
      const float u = lamb_dir(sc, m4[k], v4[k], w4[k], wd);
      sw += w4[k] * w4[k];
      su += u * u;
    }
    st_stream(mp + e, m4);
    st_stream(vp + e, v4);
  } else {
    for (long long k = e; k < n; ++k) {
      const float g = gp[k] * sc.grad_scale;
      const float m1 = b1 * mp[k] + a1 * g;
      const float v1 = b2 * vp[k] + a2 * (g * g);
      const float w = wp[k];
      const float u = lamb_dir(sc, m1, v1, w, wd);
      mp[k] = m1;
      vp[k] = v1;
      sw += w * w;
      su += u * u;
    }
  }
  const float tw = block_sum(sw, red[0]);
  const float tu = block_sum(su, red[1]);
  if (threadIdx.x == 0) partial[c] = float2{tw, tu};
}

// Sum of each group of kLambGroup chunk partials (groups never straddle two
// tensors: every tensor's chunks start at a multiple of kLambGroup).
__global__ __launch_bounds__(kLambThreads) void lamb_group_kernel(const float2* __restrict__ partial,
                                                                  double2* __restrict__ group) {
  static_assert(kLambGroup == kLambThreads, "one partial per thread");
  __shared__ double red[2][kLambThreads / 64];
  const float2 p = partial[(size_t)blockIdx.x * kLambGroup + threadIdx.x];
  const double sw = block_sum<double>(p.x, red[0]);
  const double su = block_sum<double>(p.y, red[1]);
  if (threadIdx.x == 0) group[blockIdx.x] = double2{sw, su};
}

__global__ __launch_bounds__(kLambThreads) void lamb_ratio_kernel(LambTable t,
                                                                  const double2* __restrict__ group,
                                                                  float* __restrict__ ratio,
                                                                  float* __restrict__ ratio_out) {
  __shared__ double red[2][kLambThreads / 64];
  const int ti = blockIdx.x;
  double sw = 0.0, su = 0.0;
  for (int g = t.chunk0[ti] / kLambGroup + threadIdx.x; g < t.chunk0[ti + 1] / kLambGroup;
       g += kLambThreads) {
    const double2 p = group[g];
    sw += p.x;
    su += p.y;
  }
  const double w2 = block_sum(sw, red[0]);
  const double u2 = block_sum(su, red[1]);
  if (threadIdx.x == 0) {
    const float r = (w2 > 0.0 && u2 > 0.0) ? (float)sqrt(w2 / u2) : 1.0f;
    ratio[ti] = r;
    if (ratio_out) ratio_out[ti] = r;
  }
}

template <typename CT>
__global__ __launch_bounds__(kLambThreads) void lamb_apply_kernel(LambTable t, LambScalars sc,
                                                                  const float* __restrict__ ratio) {
  const int c = blockIdx.x;
  const int ti = tensor_of(t, c);
  if (c >= t.chunk_end[ti]) return;
  const long long n = t.numel[ti];
  const long long e = (long long)(c - t.chunk0[ti]) * kLambChunk + 4 * threadIdx.x;
  float* __restrict__ wp = t.w[ti];
  const float* __restrict__ mp = t.m[ti];
  const float* __restrict__ vp = t.v[ti];
  void* copy = t.copy[ti];
  const float wd = t.wd[ti];
  const float step = sc.lr * ratio[ti];
  if (e + 4 <= n) {
    f32x4 w4 = ld_stream(wp + e);
    const f32x4 m4 = ld_stream(mp + e);
    const f32x4 v4 = ld_stream(vp + e);
#pragma unroll
    for (int k = 0; k < 4; ++k) w4[k] = w4[k] - step * lamb_dir(sc, m4[k], v4[k], w4[k], wd);
    st_stream(wp + e, w4);
    if (copy) {
      if constexpr (sizeof(CT) == 2) {
        __builtin_nontemporal_store(u32x2{pack_bf2(w4[0], w4[1]), pack_bf2(w4[2], w4[3])},
                                    reinterpret_cast<u32x2*>((bf16*)copy + e));
      } else {
        st_stream((float*)copy + e, w4);
      }
    }
  } else {
    for (long long k = e; k < n; ++k) {
      const float w = wp[k] - step * lamb_dir(sc, mp[k], vp[k], wp[k], wd);
      wp[k] = w;
      if (copy) {
        if constexpr (sizeof(CT) == 2) ((bf16*)copy)[k] = (bf16)w;
        else ((float*)copy)[k] = w;
      }
    }
  }
}

}  // namespace

int lamb_chunks(long long numel) { return (int)((numel + kLambChunk - 1) / kLambChunk); }

int lamb_padded_chunks(long long numel) {
  return (lamb_chunks(numel) + kLambGroup - 1) / kLambGroup * kLambGroup;
}

void launch_lamb(const LambTable& t, const LambScalars& sc, Dt copy_dt, float2* partial,
                 double2* group, float* ratio, float* ratio_out, hipStream_t s) {
  const int chunks = t.chunk0[t.n];
  if (chunks > 0) {
    lamb_moments_kernel<<<chunks, kLambThreads, 0, s>>>(t, sc, partial);
    lamb_group_kernel<<<chunks / kLambGroup, kLambThreads, 0, s>>>(partial, group);
  }
  lamb_ratio_kernel<<<t.n, kLambThreads, 0, s>>>(t, group, ratio, ratio_out);
  if (chunks > 0) {
    if (copy_dt == Dt::BF16) lamb_apply_kernel<bf16><<<chunks, kLambThreads, 0, s>>>(t, sc, ratio);
    else lamb_apply_kernel<float><<<chunks, kLambThreads, 0, s>>>(t, sc, ratio);
  }
}

}  // namespace pb
