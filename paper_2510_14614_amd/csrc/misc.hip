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

#include <algorithm>

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

hipError_t embed_sort(const int32_t* tokens, int B, int T, int V, int32_t* sort_scratch, hipStream_t s) {
  if (B * T > kSortMax) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_sort_kernel, dim3(1), dim3(1024), 0, s, tokens, B, T, V,
                     reinterpret_cast<uint32_t*>(sort_scratch));
  return hipGetLastError();
}

hipError_t embed_bwd(int B, int T, int d, const float* dX, float* dwte, float* dwpe, const int32_t* sort_scratch,
                     float* partial, hipStream_t s) {
  const int M = B * T;
  if (M > kSortMax) return hipErrorInvalidValue;
  const uint32_t* keys = reinterpret_cast<const uint32_t*>(sort_scratch);
  const int cb = cdiv(d, 256);
  hipLaunchKernelGGL(embed_chunk_kernel, dim3(cdiv(M, kChunk), cb), dim3(256), 0, s, keys, M, d, dX, partial);
  hipLaunchKernelGGL(embed_combine_kernel, dim3(M, cb), dim3(256), 0, s, keys, M, d, partial, dwte);
  hipLaunchKernelGGL(wpe_grad_kernel, dim3(T, cb), dim3(256), 0, s, dX, B, T, d, dwpe);
  return hipGetLastError();
}

// ---------------------------------------------------------- cross-entropy --
// One 1024-thread workgroup per token row (Sec. 2: next-token cross-entropy
// over the LM-head logits).  The row is read from HBM once, as float4 chunks
// held in registers (chunk c on thread c % 1024); each thread reduces its
// chunks to (max, sum of exp) and keeps exp(x - its max), so the gradient
//   dlogits = (softmax(x) - onehot(target)) / n
// needs one more exponential per thread, not per element.  Columns V..ldd of
// the gradient row are written as zeros.
constexpr int kCeThreads = 1024;

template <typename S>
__device__ __forceinline__ void st4g(S* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void st4g<float>(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
template <>
__device__ __forceinline__ void st4g<bf16>(bf16* p, float a, float b, float c, float d) {
  union { bf16 h[4]; uint2 w; } u;
  u.h[0] = from_f<bf16>(a); u.h[1] = from_f<bf16>(b); u.h[2] = from_f<bf16>(c); u.h[3] = from_f<bf16>(d);
  *reinterpret_cast<uint2*>(p) = u.w;
}

// (m1, s1) <- combination of two (max, sum exp(x - max)) pairs
__device__ __forceinline__ void lse_combine(float& m1, float& s1, float m2, float s2) {
  const float mm = fmaxf(m1, m2);
  if (mm == -INFINITY) return;
  s1 = (m1 == -INFINITY ? 0.f : s1 * __expf(m1 - mm)) + (m2 == -INFINITY ? 0.f : s2 * __expf(m2 - mm));
  m1 = mm;
}

// four consecutive logits as fp32 (16-byte fp32 or 8-byte bf16 load)
__device__ __forceinline__ float4 ld4l(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 ld4l(const bf16* p) {
  const uint2 w = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xFFFF0000u), __uint_as_float(w.y << 16),
                     __uint_as_float(w.y & 0xFFFF0000u));
}

// Logits are stored in the step's dtype (bf16 in mixed precision, as the
// LM-head product produces them); max, log-sum-exp, loss and gradient are
// fp32.
template <typename S, int NPT>
__global__ __launch_bounds__(kCeThreads) void ce_rows(const S* logits, int64_t ldl, const int32_t* tok, int T,
                                                      int V, float inv_n, S* dl, int64_t ldd, float* row_loss) {
  __shared__ float rm[kCeThreads / FAL_WAVE], rs[kCeThreads / FAL_WAVE];
  const int m = blockIdx.x, b = m / T, t = m % T, tid = threadIdx.x;
  int tgt = tok[(int64_t)b * (T + 1) + t + 1];
  tgt = min(max(tgt, 0), V - 1);
  const S* l = logits + (int64_t)m * ldl;
  const int nv = (V + 3) / 4, nd = (int)(ldd / 4);
  float x[NPT][4];
  float lm = -INFINITY;
#pragma unroll
  for (int i = 0; i < NPT; ++i) {
    const int c = tid + kCeThreads * i;
    if (c < nv) {
      const float4 v = ld4l(l + 4 * c);
      x[i][0] = v.x; x[i][1] = 4 * c + 1 < V ? v.y : -INFINITY;
      x[i][2] = 4 * c + 2 < V ? v.z : -INFINITY; x[i][3] = 4 * c + 3 < V ? v.w : -INFINITY;
    } else {
      x[i][0] = x[i][1] = x[i][2] = x[i][3] = -INFINITY;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) lm = fmaxf(lm, x[i][e]);
  }
  float ls = 0.f;
  if (lm != -INFINITY) {
#pragma unroll
    for (int i = 0; i < NPT; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[i][e] = __expf(x[i][e] - lm);  // exp(-inf) = 0 for masked columns
        ls += x[i][e];
      }
  }
  float gm = lm, gs = ls;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) lse_combine(gm, gs, __shfl_xor(gm, o, FAL_WAVE), __shfl_xor(gs, o, FAL_WAVE));
  if ((tid & (FAL_WAVE - 1)) == 0) { rm[tid / FAL_WAVE] = gm; rs[tid / FAL_WAVE] = gs; }
  __syncthreads();
  gm = rm[0]; gs = rs[0];
#pragma unroll
  for (int w = 1; w < kCeThreads / FAL_WAVE; ++w) lse_combine(gm, gs, rm[w], rs[w]);
  const float lse = gm + __logf(gs);
  if (tid == 0) row_loss[m] = lse - to_f(l[tgt]);
  if (!dl) return;  // loss only
  const float sc = lm == -INFINITY ? 0.f : __expf(lm - lse) * inv_n;
  S* drow = dl + (int64_t)m * ldd;
#pragma unroll
  for (int i = 0; i < NPT; ++i) {
    const int c = tid + kCeThreads * i;
    if (c >= nd) continue;
    float g[4] = {0.f, 0.f, 0.f, 0.f};
    if (c < nv) {
#pragma unroll
      for (int e = 0; e < 4; ++e) g[e] = x[i][e] * sc - (4 * c + e == tgt ? inv_n : 0.f);
    }
    st4g<S>(drow + 4 * c, g[0], g[1], g[2], g[3]);
  }
}

// bf16 rows with 16-byte accesses: lane c of the workgroup holds groups of
// eight raw logits (packed, four registers per group) rather than their
// exponentials, and recomputes exp(x - lse) for the gradient.  Packed raw
// values keep the kernel under 64 registers, so two 1024-thread workgroups
// share a compute unit and one row's reduction overlaps another's loads.
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf_at(const uint4& u, int e) {
  const uint32_t w = e < 2 ? u.x : e < 4 ? u.y : e < 6 ? u.z : u.w;
  return (e & 1) ? bf_hi(w) : bf_lo(w);
}
__device__ __forceinline__ uint32_t bf_pack2(float a, float b) {
  return (uint32_t)__builtin_bit_cast(uint16_t, from_f<bf16>(a)) |
         ((uint32_t)__builtin_bit_cast(uint16_t, from_f<bf16>(b)) << 16);
}

template <int NPT>
__global__ __launch_bounds__(kCeThreads) void ce_rows_x8(const bf16* logits, int64_t ldl, const int32_t* tok, int T,
                                                         int V, float inv_n, bf16* dl, int64_t ldd,
                                                         float* row_loss) {
  __shared__ float rm[kCeThreads / FAL_WAVE], rs[kCeThreads / FAL_WAVE];
  const int m = blockIdx.x, b = m / T, t = m % T, tid = threadIdx.x;
  int tgt = tok[(int64_t)b * (T + 1) + t + 1];
  tgt = min(max(tgt, 0), V - 1);
  const bf16* l = logits + (int64_t)m * ldl;
  const int nv = (V + 7) / 8, nd = (int)(ldd / 8);
  uint4 raw[NPT];
#pragma unroll
  for (int i = 0; i < NPT; ++i) {
    const int c = tid + kCeThreads * i;
    raw[i] = c < nv ? *reinterpret_cast<const uint4*>(l + 8 * c) : make_uint4(0u, 0u, 0u, 0u);
  }
  float lm = -INFINITY;
#pragma unroll
  for (int i = 0; i < NPT; ++i) {
    const int c = tid + kCeThreads * i;
    if (c < nv) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (8 * c + e < V) lm = fmaxf(lm, bf_at(raw[i], e));
    }
  }
  float ls = 0.f;
  if (lm != -INFINITY) {
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      const int c = tid + kCeThreads * i;
      if (c < nv) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (8 * c + e < V) ls += __expf(bf_at(raw[i], e) - lm);
      }
    }
  }
  float gm = lm, gs = ls;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) lse_combine(gm, gs, __shfl_xor(gm, o, FAL_WAVE), __shfl_xor(gs, o, FAL_WAVE));
  if ((tid & (FAL_WAVE - 1)) == 0) { rm[tid / FAL_WAVE] = gm; rs[tid / FAL_WAVE] = gs; }
  __syncthreads();
  gm = rm[0]; gs = rs[0];
#pragma unroll
  for (int w = 1; w < kCeThreads / FAL_WAVE; ++w) lse_combine(gm, gs, rm[w], rs[w]);
  const float lse = gm + __logf(gs);
  if (tid == 0) row_loss[m] = lse - to_f(l[tgt]);
  if (!dl) return;  // loss only
  bf16* drow = dl + (int64_t)m * ldd;
#pragma unroll
  for (int i = 0; i < NPT; ++i) {
    const int c = tid + kCeThreads * i;
    if (c >= nd) continue;
    float g[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int col = 8 * c + e;
      g[e] = col < V ? __expf(bf_at(raw[i], e) - lse) * inv_n - (col == tgt ? inv_n : 0.f) : 0.f;
    }
    *reinterpret_cast<uint4*>(drow + 8 * c) =
        make_uint4(bf_pack2(g[0], g[1]), bf_pack2(g[2], g[3]), bf_pack2(g[4], g[5]), bf_pack2(g[6], g[7]));
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

hipError_t cross_entropy(DType dt, const void* logits, int64_t ldl, const int32_t* tokens, int B, int T,
                         int V, void* dlogits, int64_t ldd, float* row_loss, float* loss, hipStream_t s) {
  const int M = B * T;
  const float inv_n = 1.f / (float)M;
  // float4 rows: leading dimensions multiples of 4 covering the vocabulary
  if (ldl % 4 || ldd % 4 || ldl < V || ldd < V) return hipErrorInvalidValue;
  const int64_t nd = ldd / 4;
  const int need = (int)((nd + kCeThreads - 1) / kCeThreads);
  const dim3 grid(M), block(kCeThreads);
#define FAL_CE_LAUNCH(NPT)                                                                                    \
  if (dt == BF16)                                                                                            \
    hipLaunchKernelGGL((ce_rows<bf16, NPT>), grid, block, 0, s, static_cast<const bf16*>(logits), ldl, tokens, \
                       T, V, inv_n,                                                                          \
                       static_cast<bf16*>(dlogits), ldd, row_loss);                                          \
  else                                                                                                       \
    hipLaunchKernelGGL((ce_rows<float, NPT>), grid, block, 0, s, static_cast<const float*>(logits), ldl,      \
                       tokens, T, V, inv_n,                                                                  \
                       static_cast<float*>(dlogits), ldd, row_loss);
  // bf16 rows in 16-byte groups when both row pitches allow it
  const int need8 = (int)((ldd / 8 + kCeThreads - 1) / kCeThreads);
  const bool x8 = dt == BF16 && ldl % 8 == 0 && ldd % 8 == 0 && need8 <= 8 &&
                  reinterpret_cast<uintptr_t>(logits) % 16 == 0 && reinterpret_cast<uintptr_t>(dlogits) % 16 == 0;
#define FAL_CE_X8_LAUNCH(NPT)                                                                              \
  hipLaunchKernelGGL((ce_rows_x8<NPT>), grid, block, 0, s, static_cast<const bf16*>(logits), ldl, tokens, T, V, \
                     inv_n, static_cast<bf16*>(dlogits), ldd, row_loss);
  if (x8) {
    if (need8 <= 1) { FAL_CE_X8_LAUNCH(1) }
    else if (need8 <= 2) { FAL_CE_X8_LAUNCH(2) }
    else if (need8 <= 4) { FAL_CE_X8_LAUNCH(4) }
    else if (need8 <= 7) { FAL_CE_X8_LAUNCH(7) }  // GPT-2 vocabulary (50257 padded to 50304)
    else { FAL_CE_X8_LAUNCH(8) }
  } else if (need <= 1) { FAL_CE_LAUNCH(1) }
  else if (need <= 4) { FAL_CE_LAUNCH(4) }
  else if (need <= 8) { FAL_CE_LAUNCH(8) }
  else if (need <= 13) { FAL_CE_LAUNCH(13) }  // GPT-2 vocabulary (50257 padded to 50304)
  else if (need <= 16) { FAL_CE_LAUNCH(16) }
  else return hipErrorInvalidValue;
#undef FAL_CE_LAUNCH
#undef FAL_CE_X8_LAUNCH
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (loss) {
    hipLaunchKernelGGL(sum_kernel, dim3(1), dim3(256), 0, s, row_loss, (int64_t)M, inv_n, loss);
    e = hipGetLastError();
  }
  return e;
}

// dst[r, c] = src[r, c] as fp32 for r < rows, c < cols (src in dtype).
template <typename S>
__global__ __launch_bounds__(256) void rows_to_f32_kernel(const S* src, int64_t lds, float* dst, int64_t ldd,
                                                          int cols) {
  const int r = blockIdx.y;
  for (int c = blockIdx.x * 256 + threadIdx.x; c < cols; c += gridDim.x * 256)
    dst[(int64_t)r * ldd + c] = to_f(src[(int64_t)r * lds + c]);
}

hipError_t rows_to_f32(DType dt, const void* src, int64_t lds, float* dst, int64_t ldd, int rows, int cols,
                       hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  const dim3 grid(std::min(cdiv(cols, 256), 64), rows), block(256);
  if (dt == BF16)
    hipLaunchKernelGGL(rows_to_f32_kernel<bf16>, grid, block, 0, s, static_cast<const bf16*>(src), lds, dst, ldd, cols);
  else
    hipLaunchKernelGGL(rows_to_f32_kernel<float>, grid, block, 0, s, static_cast<const float*>(src), lds, dst, ldd,
                       cols);
  return hipGetLastError();
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

// Reads n16 16-byte chunks and discards them: brings a read-only operand
// (a block's weights, untouched since the previous step) into the
// last-level cache ahead of the GEMMs that read it.
__global__ __launch_bounds__(256) void cache_warm_kernel(const uint4* p, int64_t n16) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (int64_t)gridDim.x * 256) {
    const uint4 v = p[i];
    asm volatile("" ::"v"(v.x), "v"(v.y), "v"(v.z), "v"(v.w));
  }
}

hipError_t cache_warm(const void* p, int64_t bytes, hipStream_t s) {
  if (!p || bytes <= 0) return hipSuccess;
  // whole 16-byte chunks inside [p, p + bytes)
  const uintptr_t a = (reinterpret_cast<uintptr_t>(p) + 15) & ~static_cast<uintptr_t>(15);
  const int64_t n16 = ((int64_t)(reinterpret_cast<uintptr_t>(p) + bytes) - (int64_t)a) / 16;
  if (n16 <= 0) return hipSuccess;
  p = reinterpret_cast<const void*>(a);
  const int blocks = (int)std::min<int64_t>(2048, cdiv(n16, 256));
  hipLaunchKernelGGL(cache_warm_kernel, dim3(blocks), dim3(256), 0, s, static_cast<const uint4*>(p), n16);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void copy4_kernel(float4* y, const float4* x, int64_t n4) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) y[i] = x[i];
}
__global__ __launch_bounds__(256) void copy_kernel(float* y, const float* x, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) y[i] = x[i];
}

hipError_t copy_f32(float* y, const float* x, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const bool v4 = n % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 && reinterpret_cast<uintptr_t>(y) % 16 == 0;
  const int64_t units = v4 ? n / 4 : n;
  const int blocks = (int)std::min<int64_t>(4096, (units + 255) / 256);
  if (v4)
    hipLaunchKernelGGL(copy4_kernel, dim3(blocks), dim3(256), 0, s, reinterpret_cast<float4*>(y),
                       reinterpret_cast<const float4*>(x), units);
  else
    hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(256), 0, s, y, x, units);
  return hipGetLastError();
}

hipError_t zero_f32(float* y, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(zero_kernel, dim3(cdiv(n, 256)), dim3(256), 0, s, y, n);
  return hipGetLastError();
}

}  // namespace fal
