// Measured ceilings for the roofline report (not part of the training path):
// the sustained dense bf16 matrix-core rate of this GPU.  Every wavefront
// runs kChains independent accumulation chains of v_mfma_f32_16x16x32_bf16
// on register operands, with no memory traffic in the loop, and the launch
// puts several wavefronts on every SIMD so issue never waits on a chain.
#include <hip/hip_runtime.h>

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kChains = 8;  // must match the assembly block below

__global__ __launch_bounds__(256) void mfma_bf16_peak(int iters, float* out) {
  bf16x8_t a, b;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    a[j] = static_cast<__bf16>(0.001f * (threadIdx.x % 7 + j));
    b[j] = static_cast<__bf16>(0.001f * (threadIdx.x % 5 + j));
  }
  f32x4_t acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // The chains are written out in assembly with the accumulators pinned to
  // AGPRs: compiled from the builtin, the loop-carried accumulators get
  // shuffled through register moves every iteration.
  for (int i = 0; i < iters; ++i) {
    asm volatile(
        "v_mfma_f32_16x16x32_bf16 %0, %8, %9, %0\n\t"
        "v_mfma_f32_16x16x32_bf16 %1, %8, %9, %1\n\t"
        "v_mfma_f32_16x16x32_bf16 %2, %8, %9, %2\n\t"
        "v_mfma_f32_16x16x32_bf16 %3, %8, %9, %3\n\t"
        "v_mfma_f32_16x16x32_bf16 %4, %8, %9, %4\n\t"
        "v_mfma_f32_16x16x32_bf16 %5, %8, %9, %5\n\t"
        "v_mfma_f32_16x16x32_bf16 %6, %8, %9, %6\n\t"
        "v_mfma_f32_16x16x32_bf16 %7, %8, %9, %7"
        : "+a"(acc[0]), "+a"(acc[1]), "+a"(acc[2]), "+a"(acc[3]), "+a"(acc[4]), "+a"(acc[5]), "+a"(acc[6]),
          "+a"(acc[7])
        : "v"(a), "v"(b));
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  // a value no run produces: keeps every chain live without a real store
  if (s == -1.0f) out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

extern "C" {
// Launches `blocks` workgroups of 256 threads, each running `iters` rounds of
// kChains MFMAs per wavefront, on `stream`.  FLOPs = blocks * 4 * iters *
// kChains * 2*16*16*32.  `out` (blocks*256 floats) is never written in practice.
// Returns the hipError_t of the launch.
int fal_probe_mfma_bf16(int blocks, int iters, float* out, void* stream) {
  if (blocks < 1 || iters < 1 || !out) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(mfma_bf16_peak, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), iters, out);
  return (int)hipGetLastError();
}
int fal_probe_mfma_chains() { return kChains; }
}
