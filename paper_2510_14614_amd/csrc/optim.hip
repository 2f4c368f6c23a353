// AdamW update with global-norm gradient clipping over one flat fp32
// parameter buffer (the training setups of the paper's appendix: lr 1e-4,
// weight decay 0.001, clipping to norm 1; the optimizer is Adam-type).
//
// Three launches, all HBM-bound streams:
//   1. grad_sumsq_kernel: a fixed grid of kNormBlocks workgroups sweeps the
//      gradient in a grid-stride pattern and writes one fp64 sum of squares
//      per workgroup.  The partition depends on n only, so the result is
//      deterministic.
//   2. grad_norm_kernel: one workgroup adds the partials in a fixed order and
//      writes {norm, clip factor} (and the caller's norm output).
//   3. adamw_kernel: one pass reading master weights, gradient and both
//      moments and writing master, moments and the dtype copy of the
//      weights.  It walks the buffer from the top down, so its first reads
//      find the gradient tail that the norm pass left in the last-level
//      cache.
#include <math.h>

#include <algorithm>
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace fal {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 2;                      // float4 units per thread in the update
constexpr int kChunk = kThreads * 4 * kUnroll;  // elements per update workgroup
static_assert(kAdamwMaxElems == (int64_t)0x7fffffff * kChunk, "update grid limit");

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, FAL_WAVE);
  return v;
}

// Fixed-order block sum (kThreads = 4 waves); every thread gets the total.
__device__ __forceinline__ double block_sum_f64(double v, double* red) {
  v = wave_sum_f64(v);
  const int w = threadIdx.x / FAL_WAVE, l = threadIdx.x % FAL_WAVE;
  if (l == 0) red[w] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ __launch_bounds__(kThreads) void grad_sumsq_kernel(const float* __restrict__ g, int64_t n,
                                                             double* __restrict__ part) {
  __shared__ double red[kThreads / FAL_WAVE];
  const int64_t n4 = n / 4;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  const float4* g4 = reinterpret_cast<const float4*>(g);
  double s0 = 0.0, s1 = 0.0;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  for (; i + stride < n4; i += 2 * stride) {
    const float4 a = g4[i], b = g4[i + stride];
    s0 = fma((double)a.x, (double)a.x, s0); s0 = fma((double)a.y, (double)a.y, s0);
    s0 = fma((double)a.z, (double)a.z, s0); s0 = fma((double)a.w, (double)a.w, s0);
    s1 = fma((double)b.x, (double)b.x, s1); s1 = fma((double)b.y, (double)b.y, s1);
    s1 = fma((double)b.z, (double)b.z, s1); s1 = fma((double)b.w, (double)b.w, s1);
  }
  if (i < n4) {
    const float4 a = g4[i];
    s0 = fma((double)a.x, (double)a.x, s0); s0 = fma((double)a.y, (double)a.y, s0);
    s0 = fma((double)a.z, (double)a.z, s0); s0 = fma((double)a.w, (double)a.w, s0);
  }
  // the n % 4 tail elements go to the first threads of workgroup 0
  if (blockIdx.x == 0 && threadIdx.x < (int)(n - 4 * n4)) {
    const double x = g[4 * n4 + threadIdx.x];
    s1 = fma(x, x, s1);
  }
  const double t = block_sum_f64(s0 + s1, red);
  if (threadIdx.x == 0) part[blockIdx.x] = t;
}

__global__ __launch_bounds__(kThreads) void grad_norm_kernel(const double* __restrict__ part, int nparts,
                                                            float max_norm, float* __restrict__ ctrl,
                                                            float* __restrict__ norm_out) {
  __shared__ double red[kThreads / FAL_WAVE];
  double s = 0.0;
  for (int i = threadIdx.x; i < nparts; i += kThreads) s += part[i];
  const double tot = block_sum_f64(s, red);
  if (threadIdx.x == 0) {
    const double norm = sqrt(tot);
    // scale by min(1, max_norm / (norm + 1e-6)); clipping off when max_norm <= 0
    const double c = max_norm > 0.f ? fmin(1.0, (double)max_norm / (norm + 1e-6)) : 1.0;
    ctrl[0] = (float)norm;
    ctrl[1] = (float)c;
    if (norm_out) *norm_out = (float)norm;
  }
}

struct Lp2 {  // four bf16 values
  uint32_t lo, hi;
};

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  const bf16 x = from_f<bf16>(a), y = from_f<bf16>(b);
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

__device__ __forceinline__ void adamw_elem(float& p, float g, float& m, float& v, float c, const AdamwConsts& k) {
  g *= c;
  m = fmaf(k.beta1, m, k.one_minus_beta1 * g);
  v = fmaf(k.beta2, v, k.one_minus_beta2 * g * g);
  const float denom = sqrtf(v) * k.rsqrt_bc2 + k.eps;
  p = fmaf(p, k.decay, -k.step_size * (m / denom));
}

// LP: 0 no dtype copy (fp32 master is the parameter buffer), 1 fp32 copy, 2 bf16 copy.
template <int LP>
__global__ __launch_bounds__(kThreads) void adamw_kernel(float* __restrict__ master, void* __restrict__ lp,
                                                        const float* __restrict__ g, float* __restrict__ m,
                                                        float* __restrict__ v, int64_t n, AdamwConsts k,
                                                        const float* __restrict__ ctrl) {
  const float c = ctrl[1];
  const int64_t base = (int64_t)(gridDim.x - 1 - blockIdx.x) * kChunk;
  if (base + kChunk <= n) {
    // whole chunk in range: all loads of the thread issued before any math
    float4 p4[kUnroll], g4[kUnroll], m4[kUnroll], v4[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = base + (int64_t)(u * kThreads + threadIdx.x) * 4;
      p4[u] = *reinterpret_cast<const float4*>(master + i);
      g4[u] = *reinterpret_cast<const float4*>(g + i);
      m4[u] = *reinterpret_cast<const float4*>(m + i);
      v4[u] = *reinterpret_cast<const float4*>(v + i);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = base + (int64_t)(u * kThreads + threadIdx.x) * 4;
      adamw_elem(p4[u].x, g4[u].x, m4[u].x, v4[u].x, c, k);
      adamw_elem(p4[u].y, g4[u].y, m4[u].y, v4[u].y, c, k);
      adamw_elem(p4[u].z, g4[u].z, m4[u].z, v4[u].z, c, k);
      adamw_elem(p4[u].w, g4[u].w, m4[u].w, v4[u].w, c, k);
      *reinterpret_cast<float4*>(master + i) = p4[u];
      *reinterpret_cast<float4*>(m + i) = m4[u];
      *reinterpret_cast<float4*>(v + i) = v4[u];
      if (LP == 1) *reinterpret_cast<float4*>(static_cast<float*>(lp) + i) = p4[u];
      if (LP == 2) {
        Lp2 o{pack_bf16(p4[u].x, p4[u].y), pack_bf16(p4[u].z, p4[u].w)};
        *reinterpret_cast<Lp2*>(static_cast<bf16*>(lp) + i) = o;
      }
    }
    return;
  }
  // the last (partial) chunk, element by element
  for (int64_t j = base + threadIdx.x; j < n; j += kThreads) {
    float p = master[j], mm = m[j], vv = v[j];
    adamw_elem(p, g[j], mm, vv, c, k);
    master[j] = p;
    m[j] = mm;
    v[j] = vv;
    if (LP == 1) static_cast<float*>(lp)[j] = p;
    if (LP == 2) static_cast<bf16*>(lp)[j] = from_f<bf16>(p);
  }
}

}  // namespace

hipError_t grad_norm(const float* g, int64_t n, float max_norm, double* part, float* ctrl, float* norm_out,
                     hipStream_t s) {
  hipLaunchKernelGGL(grad_sumsq_kernel, dim3(kNormBlocks), dim3(kThreads), 0, s, g, n, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(grad_norm_kernel, dim3(1), dim3(kThreads), 0, s, part, kNormBlocks, max_norm, ctrl,
                     norm_out);
  return hipGetLastError();
}

hipError_t adamw_update(int lp_mode, float* master, void* lp, const float* g, float* m, float* v, int64_t n,
                        const AdamwConsts& k, const float* ctrl, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + kChunk - 1) / kChunk;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks), block(kThreads);
  if (lp_mode == 2)
    hipLaunchKernelGGL(adamw_kernel<2>, grid, block, 0, s, master, lp, g, m, v, n, k, ctrl);
  else if (lp_mode == 1)
    hipLaunchKernelGGL(adamw_kernel<1>, grid, block, 0, s, master, lp, g, m, v, n, k, ctrl);
  else
    hipLaunchKernelGGL(adamw_kernel<0>, grid, block, 0, s, master, lp, g, m, v, n, k, ctrl);
  return hipGetLastError();
}

// Scratch of the allocation-free update (adamw_static_scratch): the norm
// pass's kNormBlocks fp64 partials, then the two-float control block.
// Every call rewrites all of it before reading it (each norm workgroup
// writes its partial, the norm kernel writes the control block), so nothing
// needs clearing between calls.  16 KiB + 256 B per GPU, held until the
// process ends.
constexpr size_t kScratchPartBytes = (size_t)kNormBlocks * sizeof(double);
constexpr size_t kScratchBytes = kScratchPartBytes + 256;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
// The array's device address per GPU.  In host code the name `scratch` is a
// host-side stand-in, not a device address, so kernels only ever receive the
// address hipGetSymbolAddress returns for the current device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

hipError_t scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}
}  // namespace

hipError_t adamw_static_scratch(int lp_mode, float* master, void* lp, const float* g, float* m, float* v, int64_t n,
                                float max_norm, const AdamwConsts& k, float* norm_out, hipStream_t s) {
  void* base = nullptr;
  hipError_t e = scratch_on_current_device(&base);
  if (e != hipSuccess) return e;
  double* part = static_cast<double*>(base);
  float* ctrl = reinterpret_cast<float*>(static_cast<char*>(base) + kScratchPartBytes);
  e = grad_norm(g, n, max_norm, part, ctrl, norm_out, s);
  if (e != hipSuccess) return e;
  return adamw_update(lp_mode, master, lp, g, m, v, n, k, ctrl, s);
}

}  // namespace fal
