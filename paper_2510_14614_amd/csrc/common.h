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
// 0.5 (1 + tanh(u)) = 1 / (1 + exp(-2u)) (one exp2 and one reciprocal);
// derivative s + 2 x s (1 - s) u' with s = 1 / (1 + exp(-2u)).
// erf form x * Phi(x) uses the library erff.
__device__ __forceinline__ float gelu_sig_arg(float x) {
  // -2u * log2(e)
  const float c2 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;
  return c2 * (x + 0.044715f * x * x * x);
}

// GELU and its derivative at x, sharing the exponential: tanh form
// x * s with s = sigmoid(2u), u = sqrt(2/pi) (x + 0.044715 x^3), so
// GELU' = s + 2 x s (1 - s) du/dx; erf form x Phi(x), GELU' = Phi + x phi.
__device__ __forceinline__ void gelu_and_grad(float x, int tanh_form, float& g, float& dg) {
  if (tanh_form) {
    const float s = __builtin_amdgcn_rcpf(1.f + exp2f(gelu_sig_arg(x)));
    const float du = 0.7978845608028654f * (1.f + 3.f * 0.044715f * x * x);
    g = x * s;
    dg = s + 2.f * x * s * (1.f - s) * du;
    return;
  }
  const float cdf = 0.5f * (1.f + erff(x * 0.7071067811865476f));
  const float pdf = 0.3989422804014327f * expf(-0.5f * x * x);
  g = x * cdf;
  dg = cdf + x * pdf;
}

static inline int cdiv(long a, long b) { return (int)((a + b - 1) / b); }
