// Device-side helpers shared by the gfx950 kernels of the block library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define PB_DEV __device__ __forceinline__

namespace pb {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// ------------------------------------------------------------ conversions
PB_DEV float bf2f(uint32_t bits16) { return __uint_as_float(bits16 << 16); }
PB_DEV float lo_bf(uint32_t w) { return __uint_as_float(w << 16); }
PB_DEV float hi_bf(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round-to-nearest-even fp32 -> bf16 bits (hardware conversion on gfx950).
PB_DEV uint32_t f2bf(float f) {
  bf16 b = (bf16)f;
  return (uint32_t)__builtin_bit_cast(uint16_t, b);
}
PB_DEV uint32_t pack_bf2(float lo, float hi) { return f2bf(lo) | (f2bf(hi) << 16); }

// ------------------------------------------------- 8-element row chunks
// Load 8 consecutive elements as fp32; T is bf16 (one 16 B load) or float
// (two 16 B loads).
template <typename T> PB_DEV void load8(const T* p, float* v);
template <> PB_DEV void load8<bf16>(const bf16* p, float* v) {
  u32x4 w = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) { v[2 * i] = lo_bf(w[i]); v[2 * i + 1] = hi_bf(w[i]); }
}
template <> PB_DEV void load8<float>(const float* p, float* v) {
  f32x4 a = *reinterpret_cast<const f32x4*>(p);
  f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) { v[i] = a[i]; v[4 + i] = b[i]; }
}
template <typename T> PB_DEV void store8(T* p, const float* v);
template <> PB_DEV void store8<bf16>(bf16* p, const float* v) {
  u32x4 w;
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = pack_bf2(v[2 * i], v[2 * i + 1]);
  *reinterpret_cast<u32x4*>(p) = w;
}
template <> PB_DEV void store8<float>(float* p, const float* v) {
  *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
  *reinterpret_cast<f32x4*>(p + 4) = f32x4{v[4], v[5], v[6], v[7]};
}
// Four consecutive elements.
template <typename T> PB_DEV void load4(const T* p, float* v);
template <> PB_DEV void load4<bf16>(const bf16* p, float* v) {
  u32x2 w = *reinterpret_cast<const u32x2*>(p);
  v[0] = lo_bf(w[0]); v[1] = hi_bf(w[0]); v[2] = lo_bf(w[1]); v[3] = hi_bf(w[1]);
}
template <> PB_DEV void load4<float>(const float* p, float* v) {
  f32x4 a = *reinterpret_cast<const f32x4*>(p);
  v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
}
template <typename T> PB_DEV void store4(T* p, const float* v);
template <> PB_DEV void store4<bf16>(bf16* p, const float* v) {
  *reinterpret_cast<u32x2*>(p) = u32x2{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3])};
}
template <> PB_DEV void store4<float>(float* p, const float* v) {
  *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
}
template <typename T> PB_DEV float load1(const T* p);
template <> PB_DEV float load1<bf16>(const bf16* p) { return (float)*p; }
template <> PB_DEV float load1<float>(const float* p) { return *p; }

// ------------------------------------------------------ 8x8 bf16 transpose
// in[j] holds 8 bf16 of row j (as 4 dwords, element 2q in the low half of
// dword q).  On return out[i] holds column i: element j of out[i] is element i
// of in[j].
PB_DEV void transpose8x8(const u32x4* in, u32x4* out) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int q = i >> 1;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t a = in[2 * p][q], b = in[2 * p + 1][q];
      out[i][p] = (i & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
    }
  }
}

// ------------------------------------------------------------- LDS-DMA
// One 16-byte LDS-DMA per lane: global sbase + voff (a wave-uniform 64-bit
// base and a 32-bit lane offset in bytes) -> LDS lds_byte_addr + 16 * lane.
PB_DEV void dma16s(const void* sbase, uint32_t voff, uint32_t lds_byte_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase),
               "s"(lds_byte_addr)
               : "memory", "m0");
}

// -------------------------------------------------------------- reductions
PB_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
PB_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// ------------------------------------------------------------------- GeLU
// Tanh form: 0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3))); erf form:
// 0.5 u (1 + erf(u / sqrt 2)).  tanh is evaluated from the hardware base-2
// exponential, tanh|a| = (1 - e) / (1 + e) with e = 2^(-2|a| log2 e): a few
// instructions, relative error of a few ulp for |a| > 0.1 and an absolute
// error below 1e-7 near 0 (well inside fp32 parity).  The erf form uses the
// ROCm device erff.
constexpr float kSqrt2OverPi = 0.7978845608028654f;
constexpr float kGeluC = 0.044715f;
constexpr float kInvSqrt2 = 0.7071067811865476f;
constexpr float kInvSqrt2Pi = 0.3989422804014327f;

PB_DEV float tanh_fast(float a) {
  const float e = __builtin_amdgcn_exp2f(-2.0f * kLog2e * fabsf(a));
  const float t = (1.0f - e) * __builtin_amdgcn_rcpf(1.0f + e);
  return __builtin_copysignf(t, a);
}

template <bool TANH>
PB_DEV float gelu(float u) {
  if constexpr (TANH) return 0.5f * u * (1.0f + tanh_fast(kSqrt2OverPi * (u + kGeluC * u * u * u)));
  else return 0.5f * u * (1.0f + erff(u * kInvSqrt2));
}
template <bool TANH>
PB_DEV float gelu_grad(float u) {
  if constexpr (TANH) {
    const float t = tanh_fast(kSqrt2OverPi * (u + kGeluC * u * u * u));
    const float da = kSqrt2OverPi * (1.0f + 3.0f * kGeluC * u * u);
    return 0.5f * (1.0f + t) + 0.5f * u * (1.0f - t * t) * da;
  } else {
    return 0.5f * (1.0f + erff(u * kInvSqrt2)) +
           u * kInvSqrt2Pi * __builtin_amdgcn_exp2f(-0.5f * kLog2e * u * u);
  }
}

}  // namespace pb
