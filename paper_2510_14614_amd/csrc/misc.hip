// Embedding, LM-head cross-entropy and small utility kernels of the GPT-2
// language-model step (token + learned position embedding, tied head,
// mean next-token cross-entropy).  All HBM-bound.
//
// Embedding backward is deterministic without atomics: token positions are
// sorted by (id, position) in one LDS bitonic sort, rows of equal ids are
// summed in position order in chunks of 32 sorted positions, and the chunk
// partials of one id are then summed in chunk order.  This keeps the hot
// ids of a Zipf token stream (id 0 is ~14% of all positions) spread over
// many workgroups.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace fal {

template <typename S>
__global__ __launch_bounds__(256) void embed_fwd_kernel(const int32_t* tok, int T, int V, int d, const S* wte,
                                                        const S* wpe, float* X) {
  const int m = blockIdx.x, b = m / T, t = m % T;
  int id = tok[(int64_t)b * (T + 1) + t];
  id = min(max(id, 0), V - 1);
  const S* we = wte + (int64_t)id * d;
  const S* pe = wpe + (int64_t)t * d;
  float* x = X + (int64_t)m * d;
  for (int j = threadIdx.x; j < d; j += 256) x[j] = to_f(we[j]) + to_f(pe[j]);
}

hipError_t embed_fwd(DType dt, const int32_t* tokens, int B, int T, int V, int d, const void* wte,
                     const void* wpe, float* X, hipStream_t s) {
  const dim3 grid(B * T), block(256);
  if (dt == BF16)
    hipLaunchKernelGGL((embed_fwd_kernel<bf16>), grid, block, 0, s, tokens, T, V, d,
                       static_cast<const bf16*>(wte), static_cast<const bf16*>(wpe), X);
  else
    hipLaunchKernelGGL((embed_fwd_kernel<float>), grid, block, 0, s, tokens, T, V, d,
                       static_cast<const float*>(wte), static_cast<const float*>(wpe), X);
  return hipGetLastError();
}

// ------------------------------------------------------ embedding backward --
constexpr int kSortMax = 16384;  // positions; 64 KB of LDS keys
constexpr int kChunk = 32;

// keys[i] = id << 16 | position, sorted ascending (single workgroup).
__global__ __launch_bounds__(1024) void embed_sort_kernel(const int32_t* tok, int B, int T, int V,
                                                          uint32_t* out) {
  __shared__ uint32_t k[kSortMax];
  const int M = B * T;
  int n = 1;
  while (n < M) n <<= 1;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    uint32_t key = 0xFFFFFFFFu;
    if (i < M) {
      const int b = i / T, t = i % T;
      int id = tok[(int64_t)b * (T + 1) + t];
      id = min(max(id, 0), V - 1);
      key = ((uint32_t)id << 16) | (uint32_t)i;
    }
    k[i] = key;
  }
  __syncthreads();
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < n; i += blockDim.x) {
        const int j = i ^ stride;
        if (j > i) {
          const bool up = (i & size) == 0;
          const uint32_t a = k[i], c = k[j];
          if ((a > c) == up) { k[i] = c; k[j] = a; }
        }
      }
      __syncthreads();
    }
  }
  for (int i = threadIdx.x; i < M; i += blockDim.x) out[i] = k[i];
}

// partial[p] (row p of [M, d]) for every position p that starts a run of
// equal ids inside its chunk of kChunk sorted positions.
__global__ __launch_bounds__(256) void embed_chunk_kernel(const uint32_t* keys, int M, int d, const float* dX,
                                                          float* partial) {
  const int c0 = blockIdx.x * kChunk;
  const int col = blockIdx.y * 256 + threadIdx.x;
  if (col >= d) return;
  const int c1 = min(M, c0 + kChunk);
  float acc = 0.f;
  int start = c0;
  for (int p = c0; p < c1; ++p) {
    const uint32_t key = keys[p];
    acc += dX[(int64_t)(key & 0xFFFFu) * d + col];
    const bool last = (p + 1 == c1) || ((keys[p + 1] >> 16) != (key >> 16));
    if (last) {
      partial[(int64_t)start * d + col] = acc;
      acc = 0.f;
      start = p + 1;
    }
  }
}

// For every sorted position that starts an id's run: sum that id's chunk
// partials in chunk order and add to dwte.
__global__ __launch_bounds__(256) void embed_combine_kernel(const uint32_t* keys, int M, int d,
                                                            const float* partial, float* dwte) {
  const int j = blockIdx.x;
  const int col = blockIdx.y * 256 + threadIdx.x;
  if (col >= d) return;
  const uint32_t id = keys[j] >> 16;
  if (j > 0 && (keys[j - 1] >> 16) == id) return;
  float s = partial[(int64_t)j * d + col];
  for (int p = (j / kChunk + 1) * kChunk; p < M && (keys[p] >> 16) == id; p += kChunk)
    s += partial[(int64_t)p * d + col];
  dwte[(int64_t)id * d + col] += s;
}

__global__ __launch_bounds__(256) void wpe_grad_kernel(const float* dX, int B, int T, int d, float* dwpe) {
  const int t = blockIdx.x;
  const int col = blockIdx.y * 256 + threadIdx.x;
  if (col >= d) return;
  float s = 0.f;
  for (int b = 0; b < B; ++b) s += dX[((int64_t)b * T + t) * d + col];
  dwpe[(int64_t)t * d + col] = s;
}

int64_t embed_bwd_scratch(int M) { return M; }

hipError_t embed_bwd(const int32_t* tokens, int B, int T, int V, int d, const float* dX, float* dwte,
                     float* dwpe, int32_t* sort_scratch, float* partial, hipStream_t s) {
  const int M = B * T;
  if (M > kSortMax) return hipErrorInvalidValue;
  uint32_t* keys = reinterpret_cast<uint32_t*>(sort_scratch);
  hipLaunchKernelGGL(embed_sort_kernel, dim3(1), dim3(1024), 0, s, tokens, B, T, V, keys);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int cb = cdiv(d, 256);
  hipLaunchKernelGGL(embed_chunk_kernel, dim3(cdiv(M, kChunk), cb), dim3(256), 0, s, keys, M, d, dX, partial);
  hipLaunchKernelGGL(embed_combine_kernel, dim3(M, cb), dim3(256), 0, s, keys, M, d, partial, dwte);
  hipLaunchKernelGGL(wpe_grad_kernel, dim3(T, cb), dim3(256), 0, s, dX, B, T, d, dwpe);
  return hipGetLastError();
}

// ---------------------------------------------------------- cross-entropy --
template <typename S>
__global__ __launch_bounds__(256) void ce_kernel(const float* logits, int64_t ldl, const int32_t* tok, int T,
                                                 int V, float inv_n, S* dl, int64_t ldd, float* row_loss) {
  __shared__ float sm[4], ss[4];
  const int m = blockIdx.x, b = m / T, t = m % T;
  int tgt = tok[(int64_t)b * (T + 1) + t + 1];
  tgt = min(max(tgt, 0), V - 1);
  const float* l = logits + (int64_t)m * ldl;
  float mx = -INFINITY, sum = 0.f;
  for (int j = threadIdx.x; j < V; j += 256) {
    const float x = l[j];
    if (x > mx) {
      sum = sum * expf(mx - x) + 1.f;
      mx = x;
    } else {
      sum += expf(x - mx);
    }
  }
  // combine (max, sum) pairs across the wavefront, then across wavefronts
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float om = __shfl_xor(mx, o, FAL_WAVE), os = __shfl_xor(sum, o, FAL_WAVE);
    const float nm = fmaxf(mx, om);
    sum = (mx == -INFINITY ? 0.f : sum * expf(mx - nm)) + (om == -INFINITY ? 0.f : os * expf(om - nm));
    mx = nm;
  }
  const int w = threadIdx.x / FAL_WAVE;
  if (threadIdx.x % FAL_WAVE == 0) { sm[w] = mx; ss[w] = sum; }
  __syncthreads();
  float gm = fmaxf(fmaxf(sm[0], sm[1]), fmaxf(sm[2], sm[3]));
  float gs = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) gs += ss[i] * expf(sm[i] - gm);
  const float lse = gm + logf(gs);
  if (threadIdx.x == 0) row_loss[m] = lse - l[tgt];
  S* drow = dl + (int64_t)m * ldd;
  for (int j = threadIdx.x; j < ldd; j += 256) {
    float g = 0.f;
    if (j < V) g = (expf(l[j] - lse) - (j == tgt ? 1.f : 0.f)) * inv_n;
    drow[j] = from_f<S>(g);
  }
}

// out = scale * sum(x[0..n)), fixed order (single workgroup).
__global__ __launch_bounds__(256) void sum_kernel(const float* x, int64_t n, float scale, float* out) {
  __shared__ float red[256];
  float s = 0.f;
  for (int64_t i = threadIdx.x; i < n; i += 256) s += x[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = red[0] * scale;
}

hipError_t cross_entropy(DType dt, const float* logits, int64_t ldl, const int32_t* tokens, int B, int T,
                         int V, void* dlogits, int64_t ldd, float* row_loss, float* loss, hipStream_t s) {
  const int M = B * T;
  const float inv_n = 1.f / (float)M;
  if (dt == BF16)
    hipLaunchKernelGGL((ce_kernel<bf16>), dim3(M), dim3(256), 0, s, logits, ldl, tokens, T, V, inv_n,
                       static_cast<bf16*>(dlogits), ldd, row_loss);
  else
    hipLaunchKernelGGL((ce_kernel<float>), dim3(M), dim3(256), 0, s, logits, ldl, tokens, T, V, inv_n,
                       static_cast<float*>(dlogits), ldd, row_loss);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (loss) {
    hipLaunchKernelGGL(sum_kernel, dim3(1), dim3(256), 0, s, row_loss, (int64_t)M, inv_n, loss);
    e = hipGetLastError();
  }
  return e;
}

// ------------------------------------------------------------------ misc --
constexpr int kDotBlocks = 256;

__global__ __launch_bounds__(256) void dot_partials(const float* a, const float* b, int64_t n, float* part) {
  __shared__ float red[256];
  float s = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    s += a[i] * b[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[blockIdx.x] = red[0];
}

int64_t dot_scratch(int64_t) { return kDotBlocks; }

hipError_t dot(const float* a, const float* b, int64_t n, float* loss, float* scratch, hipStream_t s) {
  hipLaunchKernelGGL(dot_partials, dim3(kDotBlocks), dim3(256), 0, s, a, b, n, scratch);
  hipLaunchKernelGGL(sum_kernel, dim3(1), dim3(256), 0, s, scratch, (int64_t)kDotBlocks, 1.f, loss);
  return hipGetLastError();
}

__global__ void add_kernel(const float* a, const float* b, float* y, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) y[i] = a[i] + b[i];
}

hipError_t add_f32(const float* a, const float* b, float* y, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(add_kernel, dim3(cdiv(n, 256)), dim3(256), 0, s, a, b, y, n);
  return hipGetLastError();
}

template <typename S>
__global__ void cast_kernel(const float* x, S* y, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) y[i] = from_f<S>(x[i]);
}

hipError_t cast_from_f32(DType dt, const float* x, void* y, int64_t n, hipStream_t s) {
  if (dt == BF16) hipLaunchKernelGGL((cast_kernel<bf16>), dim3(cdiv(n, 256)), dim3(256), 0, s, x, static_cast<bf16*>(y), n);
  else hipLaunchKernelGGL((cast_kernel<float>), dim3(cdiv(n, 256)), dim3(256), 0, s, x, static_cast<float*>(y), n);
  return hipGetLastError();
}

__global__ void zero_kernel(float* y, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) y[i] = 0.f;
}

hipError_t zero_f32(float* y, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(zero_kernel, dim3(cdiv(n, 256)), dim3(256), 0, s, y, n);
  return hipGetLastError();
}

}  // namespace fal
