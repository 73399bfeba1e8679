// Receiving side of the reduce-scatter after the row-parallel out-projection
// (Section 3.2, tensor/sequence-parallel overlap; Megatron sequence
// parallelism): each of tp ranks holds a partial sum C_r W_out,r^T of every
// token row, and rank j keeps the sum over ranks of its own rows plus the
// residual and the output bias, y = x + b_out + sum_r P_r.  The same pass,
// without x and b_out, sums the backward's partial LayerNorm-output
// gradients dh_r.
//
// HBM-bound elementwise pass: every thread owns eight consecutive columns of
// one row and adds the partials in rank order in fp32 (deterministic), then
// rounds once to the activation type.  Bytes per element: tp + 1 inputs
// read (plus the bias, cached), one output written.
#include "common.h"
#include "kernels.h"

namespace pb {
namespace {

constexpr int kRsThreads = 256;

template <typename T>
__global__ __launch_bounds__(kRsThreads) void rs_reduce_kernel(RsParts parts, const T* __restrict__ x,
                                                               const T* __restrict__ bias,
                                                               T* __restrict__ y, int rows, int H) {
  const int groups = H / 8;
  const long long g = (long long)blockIdx.x * kRsThreads + threadIdx.x;
  if (g >= (long long)rows * groups) return;
  const int r = (int)(g / groups), c = (int)(g % groups) * 8;
  const size_t off = (size_t)r * H + c;
  float acc[8], v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  if (x) load8<T>(x + off, acc);
  if (bias) {
    load8<T>(bias + c, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += v[e];
  }
  for (int q = 0; q < parts.n; ++q) {
    load8<T>((const T*)parts.p[q] + off, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += v[e];
  }
  store8<T>(y + off, acc);
}

}  // namespace

void launch_rs_reduce(Dt dt, const RsParts& parts, const void* x, const void* bias, void* y,
                      int rows, int H, hipStream_t s) {
  const long long work = (long long)rows * (H / 8);
  if (work == 0) return;
  const int blocks = (int)((work + kRsThreads - 1) / kRsThreads);
  if (dt == Dt::BF16)
    rs_reduce_kernel<bf16><<<blocks, kRsThreads, 0, s>>>(parts, (const bf16*)x, (const bf16*)bias,
                                                        (bf16*)y, rows, H);
  else
    rs_reduce_kernel<float><<<blocks, kRsThreads, 0, s>>>(parts, (const float*)x, (const float*)bias,
                                                         (float*)y, rows, H);
}

}  // namespace pb
