// Shared device helpers for the gfx950 kernels: storage types, conversions,
// 64-lane wavefront reductions and launch checking.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;

#define FAL_WAVE 64

__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(bf16 x) { return static_cast<float>(x); }

template <typename T> __device__ __forceinline__ T from_f(float x);
template <> __device__ __forceinline__ float from_f<float>(float x) { return x; }
// Round to nearest even (gfx950 v_cvt_pk_bf16_f32).
template <> __device__ __forceinline__ bf16 from_f<bf16>(float x) { return static_cast<bf16>(x); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, FAL_WAVE);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, FAL_WAVE));
  return v;
}

// Block-wide sum for blockDim.x == 64 * nwaves; `red` is LDS of >= nwaves floats.
template <int NWAVES>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / FAL_WAVE, l = threadIdx.x % FAL_WAVE;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NWAVES; ++i) s += red[i];
  return s;
}

// GELU (MLP non-linearity).  tanh form 0.5 x (1 + tanh(u)) with
// u = sqrt(2/pi) (x + 0.044715 x^3), evaluated through the identity
// 0.5 (1 + tanh(u)) = 1 / (1 + exp(-2u)) = s, one exp2 and one reciprocal
// (the hardware's: exp2 of a large argument gives inf and s = 0, of a very
// negative one 0 and s = 1, the limits GELU needs); derivative
// s + 2 x s (1 - s) u'.  erf form x * Phi(x) uses the library erff.
// GELU and its derivative at x share the exponential; erf form:
// GELU' = Phi + x phi.
__device__ __forceinline__ void gelu_and_grad(float x, int tanh_form, float& g, float& dg) {
  if (tanh_form) {
    constexpr float kC = 0.7978845608028654f;                 // sqrt(2/pi)
    constexpr float kA = -2.0f * kC * 1.4426950408889634f;    // -2 sqrt(2/pi) log2(e)
    const float x2 = x * x;
    const float arg = x * fmaf(x2, kA * 0.044715f, kA);        // -2u log2(e)
    const float s = __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(arg));
    g = x * s;
    // 2 u' = 2 sqrt(2/pi) (1 + 3 * 0.044715 x^2)
    const float du2 = fmaf(x2, 2.f * kC * 3.f * 0.044715f, 2.f * kC);
    dg = fmaf(g * (1.f - s), du2, s);
    return;
  }
  const float cdf = 0.5f * (1.f + erff(x * 0.7071067811865476f));
  const float pdf = 0.3989422804014327f * expf(-0.5f * x * x);
  g = x * cdf;
  dg = cdf + x * pdf;
}

static inline int cdiv(long a, long b) { return (int)((a + b - 1) / b); }
