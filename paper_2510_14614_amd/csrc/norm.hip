// LayerNorm kernels of the block (Eq. 1, Eq. 2 and the FAL+ equation):
//  * ln_fwd: one wavefront per row.  One pass over the fp32 residual row
//    gives mean and rstd and up to two normalised outputs with different
//    affine parameters.  FAL uses both outputs, since its MHA and MLP
//    LayerNorms read the same X_i (H1 = LN1(X_i), H2 = LN2(X_i) + F); FAL+
//    adds the per-block LayerNorm of the shared first-attention
//    normalisation to its MLP input in the same pass.
//  * ln_bwd: the input gradient (both LayerNorms of one input at once) and
//    the gamma/beta gradients: for widths that are a multiple of 256 (up to
//    4096) one pass forms both (partial sums per workgroup of rows); other
//    widths use a row kernel plus a column partial-sum kernel.  Either way a
//    fixed-order reduce finishes the parameter gradients.
//  * norm_bwd: backward of the affine-free normalisation of A_1 (FAL+).
//  * col_sum_batch: bias gradients, up to four matrices per pair of launches.
// All of these are HBM-bound; rows are read with 64 consecutive elements
// per wavefront instruction.
#include <algorithm>
#include <initializer_list>

#include "common.h"
#include "kernels.h"

namespace fal {

constexpr int kRowsPerBlock = 4;  // 4 wavefronts per 256-thread workgroup
// Output chunks of 256 features whose parameter loads ln_fwd_v4 issues as one
// batch; 1 and 2 were measured slower at d = 2048 and 4096.
constexpr int kFwdGroup = 4;

template <typename S, int VPT>
__global__ __launch_bounds__(256) void ln_fwd_kernel(LnFwdArgs a) {
  const int row = blockIdx.x * kRowsPerBlock + threadIdx.x / FAL_WAVE;
  const int lane = threadIdx.x % FAL_WAVE;
  if (row >= a.M) return;
  const int d = a.d;
  const float* x = a.x + (int64_t)row * d;
  float v[VPT];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int j = lane + FAL_WAVE * i;
    v[i] = j < d ? x[j] : 0.f;
    s += v[i];
  }
  const float mean = wave_sum(s) / d;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int j = lane + FAL_WAVE * i;
    const float c = j < d ? v[i] - mean : 0.f;
    q += c * c;
  }
  const float var = wave_sum(q) / d;
  const float rstd = 1.f / sqrtf(var + a.eps);
  if (lane == 0) {
    if (a.mean) a.mean[row] = mean;
    if (a.rstd) a.rstd[row] = rstd;
  }
  const S* g1 = static_cast<const S*>(a.g1);
  const S* b1 = static_cast<const S*>(a.b1);
  const S* g2 = static_cast<const S*>(a.g2);
  const S* b2 = static_cast<const S*>(a.b2);
  const S* add2 = static_cast<const S*>(a.add2);
  const S* xF = static_cast<const S*>(a.xhatF);
  const S* gF = static_cast<const S*>(a.gF);
  const S* bF = static_cast<const S*>(a.bF);
  S* y1 = static_cast<S*>(a.y1);
  S* y2 = static_cast<S*>(a.y2);
  S* xo = static_cast<S*>(a.xhat_out);
  const int64_t off = (int64_t)row * d;
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int j = lane + FAL_WAVE * i;
    if (j >= d) break;
    const float xh = (v[i] - mean) * rstd;
    if (y1) y1[off + j] = from_f<S>(xh * to_f(g1[j]) + to_f(b1[j]));
    if (y2) {
      float o = xh * to_f(g2[j]) + to_f(b2[j]);
      if (add2) o += to_f(add2[off + j]);
      if (xF) o += to_f(gF[j]) * to_f(xF[off + j]) + to_f(bF[j]);
      y2[off + j] = from_f<S>(o);
    }
    if (xo) xo[off + j] = from_f<S>(xh);
  }
}

template <typename S, int VPT>
__global__ __launch_bounds__(256) void ln_bwd_rows(LnBwdArgs a) {
  const int row = blockIdx.x * kRowsPerBlock + threadIdx.x / FAL_WAVE;
  const int lane = threadIdx.x % FAL_WAVE;
  if (row >= a.M) return;
  const int d = a.d;
  const int64_t off = (int64_t)row * d;
  const float mean = a.mean[row], rstd = a.rstd[row];
  const S* g1 = static_cast<const S*>(a.g1);
  const S* g2 = static_cast<const S*>(a.g2);
  const S* gF = static_cast<const S*>(a.gF);
  float xh[VPT], dxh[VPT];
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int j = lane + FAL_WAVE * i;
    xh[i] = 0.f;
    dxh[i] = 0.f;
    if (j < d) {
      xh[i] = (a.x[off + j] - mean) * rstd;
      float t = 0.f;
      if (a.dy1) t += a.dy1[off + j] * to_f(g1[j]);
      if (a.dy2) {
        const float dy2 = a.dy2[off + j];
        t += dy2 * to_f(g2[j]);
        if (a.dacc) a.dacc[off + j] = a.dacc_overwrite ? dy2 : a.dacc[off + j] + dy2;
        if (a.dxhatF_acc) {
          const float c = to_f(gF[j]) * dy2;
          a.dxhatF_acc[off + j] = a.dxhatF_overwrite ? c : a.dxhatF_acc[off + j] + c;
        }
      }
      dxh[i] = t;
      s1 += t;
      s2 += t * xh[i];
    }
  }
  s1 = wave_sum(s1) / d;
  s2 = wave_sum(s2) / d;
  S* lp = static_cast<S*>(a.dx_lp);
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int j = lane + FAL_WAVE * i;
    if (j >= d) break;
    float dx = rstd * (dxh[i] - s1 - xh[i] * s2);
    if (a.dres) dx += a.dres[off + j];
    a.dx[off + j] = dx;
    if (lp) lp[off + j] = from_f<S>(dx);
  }
}

// Column partial sums for the LayerNorm parameter gradients.  Workgroup =
// 256 columns x kPartRows rows: 64 threads across the columns (4 consecutive
// columns each, 16-byte loads) times 4 row groups that each walk
// kPartRows/4 rows in order; the 4 group sums are then added in a fixed
// order through LDS.  partials: [nblk][6][d].  Used for widths that are
// not a multiple of 256 and for the FAL+ terms when the side pass cannot
// take them.  32 rows gave 768 workgroups at M = 8192, d = 768, enough
// loads in flight to beat 64 rows (measured while that width still used
// this pass: LayerNorm kernels of a GPT-2-small step 1.10 -> 1.02 ms).
constexpr int kPartRows = 32;

template <typename S>
__global__ __launch_bounds__(256) void ln_param_partials(LnBwdArgs a) {
  __shared__ float red[3][6][256];
  const int cl = threadIdx.x & 63, rg = threadIdx.x >> 6;
  const int j = blockIdx.x * 256 + cl * 4;
  const int rb = blockIdx.y;
  const int d = a.d;
  const S* xF = static_cast<const S*>(a.xhatF);
  float q[6][4] = {};
  constexpr int RG = kPartRows / 4;  // rows per thread
  const int r0 = rb * kPartRows + rg * RG;
  const int r1 = min(a.M, r0 + RG);
  if (j < d && r1 - r0 == RG && !xF) {
    // a whole row group: every input row requested before the first use
    float4 xv[RG], g1[RG], g2[RG];
    float mu[RG], rs[RG];
#pragma unroll
    for (int r = 0; r < RG; ++r) {
      xv[r] = *reinterpret_cast<const float4*>(a.x + (int64_t)(r0 + r) * d + j);
      mu[r] = a.mean[r0 + r];
      rs[r] = a.rstd[r0 + r];
    }
    if (a.dy1) {
#pragma unroll
      for (int r = 0; r < RG; ++r) g1[r] = *reinterpret_cast<const float4*>(a.dy1 + (int64_t)(r0 + r) * d + j);
    }
    if (a.dy2) {
#pragma unroll
      for (int r = 0; r < RG; ++r) g2[r] = *reinterpret_cast<const float4*>(a.dy2 + (int64_t)(r0 + r) * d + j);
    }
#pragma unroll
    for (int r = 0; r < RG; ++r) {
      const float xh[4] = {(xv[r].x - mu[r]) * rs[r], (xv[r].y - mu[r]) * rs[r], (xv[r].z - mu[r]) * rs[r],
                           (xv[r].w - mu[r]) * rs[r]};
      if (a.dy1) {
        const float gv[4] = {g1[r].x, g1[r].y, g1[r].z, g1[r].w};
#pragma unroll
        for (int c = 0; c < 4; ++c) { q[0][c] += gv[c] * xh[c]; q[1][c] += gv[c]; }
      }
      if (a.dy2) {
        const float gv[4] = {g2[r].x, g2[r].y, g2[r].z, g2[r].w};
#pragma unroll
        for (int c = 0; c < 4; ++c) { q[2][c] += gv[c] * xh[c]; q[3][c] += gv[c]; }
      }
    }
  } else if (j < d) {
    // unrolled so that several rows' loads are in flight at once
#pragma unroll 4
    for (int r = r0; r < r1; ++r) {
      const int64_t o = (int64_t)r * d + j;
      const float mu = a.mean[r], rs = a.rstd[r];
      const float4 x = *reinterpret_cast<const float4*>(a.x + o);
      const float xh[4] = {(x.x - mu) * rs, (x.y - mu) * rs, (x.z - mu) * rs, (x.w - mu) * rs};
      if (a.dy1) {
        const float4 g = *reinterpret_cast<const float4*>(a.dy1 + o);
        const float gv[4] = {g.x, g.y, g.z, g.w};
#pragma unroll
        for (int c = 0; c < 4; ++c) { q[0][c] += gv[c] * xh[c]; q[1][c] += gv[c]; }
      }
      if (a.dy2) {
        const float4 g = *reinterpret_cast<const float4*>(a.dy2 + o);
        const float gv[4] = {g.x, g.y, g.z, g.w};
#pragma unroll
        for (int c = 0; c < 4; ++c) { q[2][c] += gv[c] * xh[c]; q[3][c] += gv[c]; }
        if (xF) {
#pragma unroll
          for (int c = 0; c < 4; ++c) q[4][c] += gv[c] * to_f(xF[o + c]);
        }
      }
    }
  }
  if (rg > 0) {
#pragma unroll
    for (int k = 0; k < 6; ++k)
#pragma unroll
      for (int c = 0; c < 4; ++c) red[rg - 1][k][cl * 4 + c] = q[k][c];
  }
  __syncthreads();
  if (rg == 0 && j < d) {
    float* p = a.partials + (int64_t)rb * 6 * d + j;
#pragma unroll
    for (int k = 0; k < 6; ++k) {
      float v[4];
#pragma unroll
      for (int c = 0; c < 4; ++c)
        v[c] = ((q[k][c] + red[0][k][cl * 4 + c]) + red[1][k][cl * 4 + c]) + red[2][k][cl * 4 + c];
      *reinterpret_cast<float4*>(p + (int64_t)k * d) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

// out_k[j] = sum_b part[b * stride + src_k * d + j] for up to 6 outputs, in
// a fixed order: kRedWaves threads per column (one per wavefront) each sum
// every kRedWaves-th partial in block order, then those sums are added
// pairwise in a fixed tree.  Sixteen wavefronts per workgroup keep enough
// loads in flight over the few workgroups a d-wide reduce has.
constexpr int kRedWaves = 16;
__device__ __forceinline__ float tree_sum(const float (&red)[kRedWaves][64], int c) {
  float t[kRedWaves];
#pragma unroll
  for (int w = 0; w < kRedWaves; ++w) t[w] = red[w][c];
#pragma unroll
  for (int h = kRedWaves / 2; h >= 1; h /= 2)
#pragma unroll
    for (int w = 0; w < h; ++w) t[w] = t[2 * w] + t[2 * w + 1];
  return t[0];
}
struct ColReduceArgs {
  const float* part;
  int nblk;
  int64_t stride;
  int d;
  float* out[6];
  int src[6];
};

__global__ __launch_bounds__(64 * kRedWaves) void col_reduce_multi(ColReduceArgs a) {
  __shared__ float red[kRedWaves][64];
  const int col = blockIdx.x * 64 + (threadIdx.x & 63);
  const int part = threadIdx.x >> 6;
  const int k = blockIdx.y;
  float* out = a.out[k];
  if (!out) return;
  float s = 0.f;
  if (col < a.d) {
    const float* p = a.part + (int64_t)a.src[k] * a.d + col;
#pragma unroll 8
    for (int b = part; b < a.nblk; b += kRedWaves) s += p[(int64_t)b * a.stride];
  }
  red[part][threadIdx.x & 63] = s;
  __syncthreads();
  if (part == 0 && col < a.d) out[col] = tree_sum(red, threadIdx.x & 63);
}

hipError_t col_reduce(const float* part, int nblk, int64_t stride, int d, float* out, hipStream_t s) {
  ColReduceArgs a{};
  a.part = part; a.nblk = nblk; a.stride = stride; a.d = d;
  a.out[0] = out; a.src[0] = 0;
  hipLaunchKernelGGL(col_reduce_multi, dim3(cdiv(d, 64), 1), dim3(64 * kRedWaves), 0, s, a);
  return hipGetLastError();
}

template <typename S, int VPT>
__global__ __launch_bounds__(256) void norm_bwd_kernel(const float* A, const float* mean,
                                                       const float* rstd, const float* dxhat, int M,
                                                       int d, const float* dres, float* da, S* lp) {
  const int row = blockIdx.x * kRowsPerBlock + threadIdx.x / FAL_WAVE;
  const int lane = threadIdx.x % FAL_WAVE;
  if (row >= M) return;
  const int64_t off = (int64_t)row * d;
  const float mu = mean[row], rs = rstd[row];
  float xh[VPT], g[VPT];
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int j = lane + FAL_WAVE * i;
    xh[i] = 0.f;
    g[i] = 0.f;
    if (j < d) {
      xh[i] = (A[off + j] - mu) * rs;
      g[i] = dxhat[off + j];
      s1 += g[i];
      s2 += g[i] * xh[i];
    }
  }
  s1 = wave_sum(s1) / d;
  s2 = wave_sum(s2) / d;
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int j = lane + FAL_WAVE * i;
    if (j >= d) break;
    float v = rs * (g[i] - s1 - xh[i] * s2);
    if (dres) v += dres[off + j];
    da[off + j] = v;
    if (lp) lp[off + j] = from_f<S>(v);
  }
}

// ---------------------------------------------------------------------------
// The same row kernels with 4-element chunks per lane (16-byte fp32 and
// 8-byte bf16 accesses): lane l owns chunks l, l + 64, ... of its row.  Used
// when d is a multiple of 4 and every row and parameter pointer is aligned
// to its chunk; the scalar kernels above serve the rest.
__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ void st4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
template <typename S> __device__ __forceinline__ float4 ld4s(const S* p);
template <> __device__ __forceinline__ float4 ld4s<float>(const float* p) { return ld4(p); }
template <> __device__ __forceinline__ float4 ld4s<bf16>(const bf16* p) {
  const uint2 w = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xFFFF0000u), __uint_as_float(w.y << 16),
                     __uint_as_float(w.y & 0xFFFF0000u));
}
template <typename S> __device__ __forceinline__ void st4s(S* p, float4 v);
template <> __device__ __forceinline__ void st4s<float>(float* p, float4 v) { st4(p, v); }
template <> __device__ __forceinline__ void st4s<bf16>(bf16* p, float4 v) {
  union { bf16 h[4]; uint2 w; } u;
  u.h[0] = from_f<bf16>(v.x); u.h[1] = from_f<bf16>(v.y); u.h[2] = from_f<bf16>(v.z); u.h[3] = from_f<bf16>(v.w);
  *reinterpret_cast<uint2*>(p) = u.w;
}
// Four elements held as stored (bf16: 2 registers), widened at use.
template <typename S> struct Raw4 { float4 v; };
template <> struct Raw4<bf16> { uint2 w; };
template <typename S> __device__ __forceinline__ Raw4<S> raw4(const S* p);
template <> __device__ __forceinline__ Raw4<float> raw4<float>(const float* p) { return {ld4(p)}; }
template <> __device__ __forceinline__ Raw4<bf16> raw4<bf16>(const bf16* p) { return {*reinterpret_cast<const uint2*>(p)}; }
__device__ __forceinline__ float4 val4(Raw4<float> r) { return r.v; }
__device__ __forceinline__ float4 val4(Raw4<bf16> r) {
  return make_float4(__uint_as_float(r.w.x << 16), __uint_as_float(r.w.x & 0xFFFF0000u), __uint_as_float(r.w.y << 16),
                     __uint_as_float(r.w.y & 0xFFFF0000u));
}
__device__ __forceinline__ float4 f4(float a) { return make_float4(a, a, a, a); }
__device__ __forceinline__ float4 operator+(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
__device__ __forceinline__ float4 operator-(float4 a, float4 b) { return make_float4(a.x - b.x, a.y - b.y, a.z - b.z, a.w - b.w); }
__device__ __forceinline__ float4 operator*(float4 a, float4 b) { return make_float4(a.x * b.x, a.y * b.y, a.z * b.z, a.w * b.w); }
__device__ __forceinline__ float hsum(float4 a) { return (a.x + a.y) + (a.z + a.w); }

template <typename S, int NC>
__global__ __launch_bounds__(256) void ln_fwd_v4(LnFwdArgs a) {
  const int row = blockIdx.x * kRowsPerBlock + threadIdx.x / FAL_WAVE;
  const int lane = threadIdx.x % FAL_WAVE;
  if (row >= a.M) return;
  const int d = a.d;
  const int64_t off = (int64_t)row * d;
  float4 v[NC];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int j = 4 * (lane + FAL_WAVE * i);
    v[i] = j < d ? ld4(a.x + off + j) : f4(0.f);
    s += hsum(v[i]);
  }
  const float mean = wave_sum(s) / d;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int j = 4 * (lane + FAL_WAVE * i);
    if (j < d) {
      const float4 c = v[i] - f4(mean);
      q += hsum(c * c);
    }
  }
  const float var = wave_sum(q) / d;
  const float rstd = 1.f / sqrtf(var + a.eps);
  if (lane == 0) {
    if (a.mean) a.mean[row] = mean;
    if (a.rstd) a.rstd[row] = rstd;
  }
  const S* g1 = static_cast<const S*>(a.g1);
  const S* b1 = static_cast<const S*>(a.b1);
  const S* g2 = static_cast<const S*>(a.g2);
  const S* b2 = static_cast<const S*>(a.b2);
  const S* add2 = static_cast<const S*>(a.add2);
  const S* xF = static_cast<const S*>(a.xhatF);
  const S* gF = static_cast<const S*>(a.gF);
  const S* bF = static_cast<const S*>(a.bF);
  S* y1 = static_cast<S*>(a.y1);
  S* y2 = static_cast<S*>(a.y2);
  S* xo = static_cast<S*>(a.xhat_out);
  // Outputs in groups of G chunks: every parameter and addend of a group is
  // requested before any is used, so a group waits for one round trip.
  constexpr int G = NC < kFwdGroup ? NC : kFwdGroup;
#pragma unroll
  for (int i0 = 0; i0 < NC; i0 += G) {
    Raw4<S> rg1[G], rb1[G], rg2[G], rb2[G], ra2[G], rgF[G], rxF[G], rbF[G];
#pragma unroll
    for (int k = 0; k < G; ++k) {
      const int j = 4 * (lane + FAL_WAVE * (i0 + k));
      if (j >= d) break;
      if (y1) {
        rg1[k] = raw4<S>(g1 + j);
        rb1[k] = raw4<S>(b1 + j);
      }
      if (y2) {
        rg2[k] = raw4<S>(g2 + j);
        rb2[k] = raw4<S>(b2 + j);
        if (add2) ra2[k] = raw4<S>(add2 + off + j);
        if (xF) {
          rgF[k] = raw4<S>(gF + j);
          rxF[k] = raw4<S>(xF + off + j);
          rbF[k] = raw4<S>(bF + j);
        }
      }
    }
#pragma unroll
    for (int k = 0; k < G; ++k) {
      const int j = 4 * (lane + FAL_WAVE * (i0 + k));
      if (j >= d) break;
      const float4 xh = (v[i0 + k] - f4(mean)) * f4(rstd);
      if (y1) st4s<S>(y1 + off + j, xh * val4(rg1[k]) + val4(rb1[k]));
      if (y2) {
        float4 o = xh * val4(rg2[k]) + val4(rb2[k]);
        if (add2) o = o + val4(ra2[k]);
        if (xF) o = o + (val4(rgF[k]) * val4(rxF[k]) + val4(rbF[k]));
        st4s<S>(y2 + off + j, o);
      }
      if (xo) st4s<S>(xo + off + j, xh);
    }
  }
}

template <typename S, int NC>
__global__ __launch_bounds__(256) void ln_bwd_v4(LnBwdArgs a) {
  const int row = blockIdx.x * kRowsPerBlock + threadIdx.x / FAL_WAVE;
  const int lane = threadIdx.x % FAL_WAVE;
  if (row >= a.M) return;
  const int d = a.d;
  const int64_t off = (int64_t)row * d;
  const float mean = a.mean[row], rstd = a.rstd[row];
  const S* g1 = static_cast<const S*>(a.g1);
  const S* g2 = static_cast<const S*>(a.g2);
  const S* gF = static_cast<const S*>(a.gF);
  // The inputs of G chunks at a time (all of the row's up to 4 chunks per
  // lane) are requested before any is used, so a group waits for one
  // memory round trip; a lane past the row's end reads the row's first
  // chunk instead and discards it (no load sits behind a branch).  Past 4
  // chunks per lane the residual gradient is read after the reductions,
  // where holding it would cost occupancy.
  constexpr int G = NC <= 4 ? NC : 4;
  constexpr bool PRE = NC <= 4;
  static_assert(NC % G == 0, "whole groups");
  float4 xh[NC], dxh[NC], res[PRE ? NC : 1];
  int jc[NC];
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int j = 4 * (lane + FAL_WAVE * i);
    jc[i] = j < d ? j : 0;
  }
  if (PRE && a.dres) {
#pragma unroll
    for (int i = 0; i < NC; ++i) res[PRE ? i : 0] = ld4(a.dres + off + jc[i]);
  }
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int i0 = 0; i0 < NC; i0 += G) {
    float4 v1[G], v2[G], vacc[G];
    Raw4<S> gv1[G], gv2[G];
#pragma unroll
    for (int k = 0; k < G; ++k) xh[i0 + k] = ld4(a.x + off + jc[i0 + k]);
    if (a.dy1) {
#pragma unroll
      for (int k = 0; k < G; ++k) {
        v1[k] = ld4(a.dy1 + off + jc[i0 + k]);
        gv1[k] = raw4<S>(g1 + jc[i0 + k]);
      }
    }
    if (a.dy2) {
#pragma unroll
      for (int k = 0; k < G; ++k) {
        v2[k] = ld4(a.dy2 + off + jc[i0 + k]);
        gv2[k] = raw4<S>(g2 + jc[i0 + k]);
      }
    }
    if (a.dacc && !a.dacc_overwrite) {
#pragma unroll
      for (int k = 0; k < G; ++k) vacc[k] = ld4(a.dacc + off + jc[i0 + k]);
    }
#pragma unroll
    for (int k = 0; k < G; ++k) {
      const int i = i0 + k;
      const int j = 4 * (lane + FAL_WAVE * i);
      xh[i] = (xh[i] - f4(mean)) * f4(rstd);
      dxh[i] = f4(0.f);
      if (j < d) {
        float4 t = f4(0.f);
        if (a.dy1) t = t + v1[k] * val4(gv1[k]);
        if (a.dy2) {
          t = t + v2[k] * val4(gv2[k]);
          if (a.dacc) st4(a.dacc + off + j, a.dacc_overwrite ? v2[k] : vacc[k] + v2[k]);
          if (a.dxhatF_acc) {
            const float4 c = ld4s<S>(gF + j) * v2[k];
            st4(a.dxhatF_acc + off + j, a.dxhatF_overwrite ? c : ld4(a.dxhatF_acc + off + j) + c);
          }
        }
        dxh[i] = t;
        s1 += hsum(t);
        s2 += hsum(t * xh[i]);
      }
    }
  }
  s1 = wave_sum(s1) / d;
  s2 = wave_sum(s2) / d;
  S* lp = static_cast<S*>(a.dx_lp);
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int j = 4 * (lane + FAL_WAVE * i);
    if (j >= d) break;
    float4 dx = f4(rstd) * (dxh[i] - f4(s1) - xh[i] * f4(s2));
    if (a.dres) dx = dx + (PRE ? res[PRE ? i : 0] : ld4(a.dres + off + j));
    st4(a.dx + off + j, dx);
    if (lp) st4s<S>(lp + off + j, dx);
  }
}

template <typename S, int NC>
__global__ __launch_bounds__(256) void norm_bwd_v4(const float* A, const float* mean, const float* rstd,
                                                  const float* dxhat, int M, int d, const float* dres, float* da,
                                                  S* lp) {
  const int row = blockIdx.x * kRowsPerBlock + threadIdx.x / FAL_WAVE;
  const int lane = threadIdx.x % FAL_WAVE;
  if (row >= M) return;
  const int64_t off = (int64_t)row * d;
  const float mu = mean[row], rs = rstd[row];
  // every input of the row requested before any is used (a lane past the
  // row's end reads the row's first chunk and discards it); past 4 chunks
  // per lane the residual gradient is read after the reductions
  constexpr bool PRE = NC <= 4;
  float4 xh[NC], g[NC], res[PRE ? NC : 1];
  int jc[NC];
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int j = 4 * (lane + FAL_WAVE * i);
    jc[i] = j < d ? j : 0;
    xh[i] = ld4(A + off + jc[i]);
    g[i] = ld4(dxhat + off + jc[i]);
  }
  if (PRE && dres) {
#pragma unroll
    for (int i = 0; i < NC; ++i) res[PRE ? i : 0] = ld4(dres + off + jc[i]);
  }
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int j = 4 * (lane + FAL_WAVE * i);
    if (j < d) {
      xh[i] = (xh[i] - f4(mu)) * f4(rs);
      s1 += hsum(g[i]);
      s2 += hsum(g[i] * xh[i]);
    }
  }
  s1 = wave_sum(s1) / d;
  s2 = wave_sum(s2) / d;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int j = 4 * (lane + FAL_WAVE * i);
    if (j >= d) break;
    float4 v = f4(rs) * (g[i] - f4(s1) - xh[i] * f4(s2));
    if (dres) v = v + (PRE ? res[PRE ? i : 0] : ld4(dres + off + j));
    st4(da + off + j, v);
    if (lp) st4s<S>(lp + off + j, v);
  }
}

// LayerNorm backward in one pass for widths that are a multiple of 256 (up
// to 4096): a workgroup walks `rows` consecutive rows with all 256 threads
// on one row (NCH 4-element chunks each), combines the four wavefronts' row
// sums through LDS in a fixed order (one barrier per row, double-buffered),
// and keeps the parameter-gradient sums of its rows in registers, written
// once as partial rows [blk][6][d] (rows 0..3: dg1, db1, dg2, db2) for
// col_reduce_multi.  This replaces the separate partial-sum pass and its
// second read of X, dY1 and dY2.  The gains are read once per workgroup and
// every input of a row is requested before any of it is used, so a row
// waits for one memory round trip.  (The FAL+ first-attention terms go to
// the two-kernel path.)
template <typename S, int NCH, bool TAIL>
__global__ __launch_bounds__(256) void ln_bwd_fused(LnBwdArgs a, int rows) {
  __shared__ float red[2][4][2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = a.d;
  S* lp = static_cast<S*>(a.dx_lp);
  // chunk c of this thread holds columns j = 4 (tid + 256 c).  TAIL: d is
  // not a multiple of 1024, so the last chunk of some wavefronts (whole
  // ones, d being a multiple of 256) lies past the row's end; they read the
  // row's first chunk instead and store nothing.
  bool inc[NCH];
  int jc[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int j = 4 * (tid + 256 * c);
    inc[c] = !TAIL || c < NCH - 1 || j < d;
    jc[c] = inc[c] ? j : 0;
  }
  Raw4<S> gv1[NCH], gv2[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    if (a.dy1) gv1[c] = raw4<S>(static_cast<const S*>(a.g1) + jc[c]);
    if (a.dy2) gv2[c] = raw4<S>(static_cast<const S*>(a.g2) + jc[c]);
  }
  float4 q[4][NCH];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int c = 0; c < NCH; ++c) q[k][c] = f4(0.f);
  const int r0 = blockIdx.x * rows, r1 = min(a.M, r0 + rows);
  for (int r = r0; r < r1; ++r) {
    const int64_t off = (int64_t)r * d;
    const float mean = a.mean[r], rstd = a.rstd[r];
    float4 xh[NCH], t[NCH], res[NCH], v1[NCH], v2[NCH], vacc[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) xh[c] = ld4(a.x + off + jc[c]);
    if (a.dy1) {
#pragma unroll
      for (int c = 0; c < NCH; ++c) v1[c] = ld4(a.dy1 + off + jc[c]);
    }
    if (a.dy2) {
#pragma unroll
      for (int c = 0; c < NCH; ++c) v2[c] = ld4(a.dy2 + off + jc[c]);
    }
    if (a.dres) {
#pragma unroll
      for (int c = 0; c < NCH; ++c) res[c] = ld4(a.dres + off + jc[c]);
    }
    if (a.dacc && !a.dacc_overwrite) {
#pragma unroll
      for (int c = 0; c < NCH; ++c) vacc[c] = ld4(a.dacc + off + jc[c]);
    }
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int j = 4 * (tid + 256 * c);
      xh[c] = (xh[c] - f4(mean)) * f4(rstd);
      t[c] = f4(0.f);
      if (!inc[c]) continue;
      float4 tt = f4(0.f);
      if (a.dy1) {
        const float4 v = v1[c];
        tt = tt + v * val4(gv1[c]);
        q[0][c] = q[0][c] + v * xh[c];
        q[1][c] = q[1][c] + v;
      }
      if (a.dy2) {
        const float4 v = v2[c];
        tt = tt + v * val4(gv2[c]);
        q[2][c] = q[2][c] + v * xh[c];
        q[3][c] = q[3][c] + v;
        if (a.dacc) st4(a.dacc + off + j, a.dacc_overwrite ? v : vacc[c] + v);
      }
      t[c] = tt;
      s1 += hsum(tt);
      s2 += hsum(tt * xh[c]);
    }
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    const int b = (r - r0) & 1;
    if (lane == 0) {
      red[b][wave][0] = s1;
      red[b][wave][1] = s2;
    }
    __syncthreads();
    s1 = (((red[b][0][0] + red[b][1][0]) + red[b][2][0]) + red[b][3][0]) / d;
    s2 = (((red[b][0][1] + red[b][1][1]) + red[b][2][1]) + red[b][3][1]) / d;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int j = 4 * (tid + 256 * c);
      if (!inc[c]) continue;
      float4 dx = f4(rstd) * (t[c] - f4(s1) - xh[c] * f4(s2));
      if (a.dres) dx = dx + res[c];
      st4(a.dx + off + j, dx);
      if (lp) st4s<S>(lp + off + j, dx);
    }
  }
  float* p = a.partials + (int64_t)blockIdx.x * 6 * d;
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int c = 0; c < NCH; ++c)
      if (inc[c]) st4(p + (int64_t)k * d + 4 * (tid + 256 * c), q[k][c]);
}

// Chunks of 4 per lane for width d (a multiple of 4), 0 if too wide.
template <typename F>
static hipError_t dispatch_nc(int d, F&& f) {
  if (d <= 256) return f(std::integral_constant<int, 1>{});
  if (d <= 512) return f(std::integral_constant<int, 2>{});
  if (d <= 768) return f(std::integral_constant<int, 3>{});
  if (d <= 1024) return f(std::integral_constant<int, 4>{});
  if (d <= 2048) return f(std::integral_constant<int, 8>{});
  if (d <= 4096) return f(std::integral_constant<int, 16>{});
  return hipErrorInvalidValue;
}
static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }
static bool al8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7) == 0; }
// fp32 row pointers 16-byte aligned, dtype ones 8-byte (4 bf16) or 16-byte (4 fp32); NULL passes
static bool vec_ok(DType dt, int d, std::initializer_list<const void*> f32, std::initializer_list<const void*> lp) {
  if (d % 4) return false;
  for (const void* p : f32)
    if (p && !al16(p)) return false;
  for (const void* p : lp)
    if (p && !(dt == BF16 ? al8(p) : al16(p))) return false;
  return true;
}

template <typename F>
static hipError_t dispatch_vpt(int d, F&& f) {
  if (d <= 64) return f(std::integral_constant<int, 1>{});
  if (d <= 128) return f(std::integral_constant<int, 2>{});
  if (d <= 256) return f(std::integral_constant<int, 4>{});
  if (d <= 512) return f(std::integral_constant<int, 8>{});
  if (d <= 1024) return f(std::integral_constant<int, 16>{});
  if (d <= 2048) return f(std::integral_constant<int, 32>{});
  if (d <= 4096) return f(std::integral_constant<int, 64>{});
  return hipErrorInvalidValue;
}

hipError_t ln_fwd(DType dt, const LnFwdArgs& a, hipStream_t s) {
  const dim3 grid(cdiv(a.M, kRowsPerBlock)), block(256);
  if (vec_ok(dt, a.d, {a.x}, {a.g1, a.b1, a.y1, a.g2, a.b2, a.y2, a.add2, a.xhatF, a.gF, a.bF, a.xhat_out}))
    return dispatch_nc(a.d, [&](auto nc) {
      constexpr int C = decltype(nc)::value;
      if (dt == BF16) hipLaunchKernelGGL((ln_fwd_v4<bf16, C>), grid, block, 0, s, a);
      else hipLaunchKernelGGL((ln_fwd_v4<float, C>), grid, block, 0, s, a);
      return hipGetLastError();
    });
  return dispatch_vpt(a.d, [&](auto vpt) {
    constexpr int V = decltype(vpt)::value;
    if (dt == BF16) hipLaunchKernelGGL((ln_fwd_kernel<bf16, V>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((ln_fwd_kernel<float, V>), grid, block, 0, s, a);
    return hipGetLastError();
  });
}

// Rows per workgroup of the fused pass: as many workgroups as fit on the
// chip at once (256 CUs times the workgroups per CU the kernel's registers
// allow: 4, 4, 2, 2 for d = 1024 .. 4096), so that every CU walks rows with
// several workgroups from the start, and no more, since each workgroup
// writes 4 d partial sums.  Measured against 8 and 16 fixed rows at
// (M, d) = (8192, 2048), (4096, 4096) and (16384, 1024).
static int fused_rows(int M, int d) {
  static const int per_cu[4] = {4, 4, 2, 2};
  const int nch = std::min(4, std::max(1, cdiv(d, 1024)));
  return std::max(1, cdiv(M, 256 * per_cu[nch - 1]));
}

// FAL+ side pass over a group of N blocks: each thread owns 4 columns of a
// block of kSideRows rows, reads the row's xhatF and accumulator once and
// every block's dy2, updates the accumulator in place (block order) and
// writes its column partials of dy2[k] * xhatF as [blk][N][d];
// col_reduce_multi sums the blocks in a fixed order.  No barriers.
constexpr int kSideRows = 32;
struct SideArgs {
  const float* dy2[kSideGroup];
  const void* gF[kSideGroup];
  const void* xF;
  float* acc;
  int ow, M, d;
  float* part;
};
template <typename S, int N>
__global__ __launch_bounds__(256) void falplus_side_kernel(SideArgs a) {
  const int d = a.d;
  const int j = 4 * (blockIdx.x * 256 + threadIdx.x);
  if (j >= d) return;
  const int r0 = blockIdx.y * kSideRows, r1 = min(a.M, r0 + kSideRows);
  const S* xF = static_cast<const S*>(a.xF);
  float4 g[N], q[N];
#pragma unroll
  for (int k = 0; k < N; ++k) {
    g[k] = ld4s<S>(static_cast<const S*>(a.gF[k]) + j);
    q[k] = f4(0.f);
  }
  for (int r = r0; r < r1; ++r) {
    const int64_t off = (int64_t)r * d + j;
    float4 v[N];
#pragma unroll
    for (int k = 0; k < N; ++k) v[k] = ld4(a.dy2[k] + off);
    const float4 x = ld4s<S>(xF + off);
    float4 w = a.ow ? g[0] * v[0] : ld4(a.acc + off) + g[0] * v[0];
#pragma unroll
    for (int k = 1; k < N; ++k) w = w + g[k] * v[k];
    st4(a.acc + off, w);
#pragma unroll
    for (int k = 0; k < N; ++k) q[k] = q[k] + v[k] * x;
  }
  float* p = a.part + (int64_t)blockIdx.y * N * d + j;
#pragma unroll
  for (int k = 0; k < N; ++k) st4(p + (int64_t)k * d, q[k]);
}

bool falplus_side_ok(DType dt, int d, const float* dy2, const void* xhatF, const void* gF, const float* acc) {
  return vec_ok(dt, d, {dy2, acc}, {xhatF, gF}) && dy2 && xhatF && gF && acc;
}

int64_t falplus_side_scratch(int M, int d) { return (int64_t)kSideGroup * cdiv(M, kSideRows) * d; }

template <typename S, int N>
static void side_launch(const SideArgs& a, dim3 grid, hipStream_t s) {
  hipLaunchKernelGGL((falplus_side_kernel<S, N>), grid, dim3(256), 0, s, a);
}
static_assert(kSideGroup == 4, "side_dispatch instantiates groups of 1 to 4 blocks");
template <typename S>
static hipError_t side_dispatch(int n, const SideArgs& a, dim3 grid, hipStream_t s) {
  switch (n) {
    case 1: side_launch<S, 1>(a, grid, s); break;
    case 2: side_launch<S, 2>(a, grid, s); break;
    case 3: side_launch<S, 3>(a, grid, s); break;
    case 4: side_launch<S, 4>(a, grid, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t falplus_side(DType dt, const FalPlusSide& g, const void* xhatF, float* dxhatF_acc, int overwrite, int M,
                        int d, float* scratch, hipStream_t s) {
  if (M < 1 || g.n < 1 || g.n > kSideGroup || !scratch) return hipErrorInvalidValue;
  SideArgs a{};
  for (int k = 0; k < g.n; ++k) {
    if (!falplus_side_ok(dt, d, g.dy2[k], xhatF, g.gF[k], dxhatF_acc) || !g.dgF[k]) return hipErrorInvalidValue;
    a.dy2[k] = g.dy2[k];
    a.gF[k] = g.gF[k];
  }
  a.xF = xhatF; a.acc = dxhatF_acc; a.ow = overwrite ? 1 : 0; a.M = M; a.d = d; a.part = scratch;
  const dim3 grid(cdiv(d / 4, 256), cdiv(M, kSideRows));
  hipError_t e = dt == BF16 ? side_dispatch<bf16>(g.n, a, grid, s) : side_dispatch<float>(g.n, a, grid, s);
  if (e != hipSuccess) return e;
  // the block partial sums, in order, six outputs per launch
  for (int k0 = 0; k0 < g.n; k0 += 6) {
    ColReduceArgs r{};
    r.part = scratch; r.nblk = cdiv(M, kSideRows); r.stride = (int64_t)g.n * d; r.d = d;
    const int nk = std::min(6, g.n - k0);
    for (int k = 0; k < nk; ++k) { r.out[k] = g.dgF[k0 + k]; r.src[k] = k0 + k; }
    hipLaunchKernelGGL(col_reduce_multi, dim3(cdiv(d, 64), nk), dim3(64 * kRedWaves), 0, s, r);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

int64_t ln_bwd_scratch(int M, int d) {
  return (int64_t)std::max(cdiv(M, kPartRows), cdiv(M, fused_rows(M, d))) * 6 * d;
}

hipError_t ln_bwd(DType dt, const LnBwdArgs& a, hipStream_t s) {
  const dim3 grid(cdiv(a.M, kRowsPerBlock)), block(256);
  hipError_t e;
  const bool any = a.dg1 || a.db1 || a.dg2 || a.db2 || a.dgF || a.dbF;
  if (any && a.d % 256 == 0 && a.d <= 4096 && a.partials && !a.xhatF && !a.dxhatF_acc && !a.dgF &&
      vec_ok(dt, a.d, {a.x, a.dy1, a.dy2, a.dres, a.dx, a.dacc, a.dxhatF_acc, a.partials},
             {a.g1, a.g2, a.gF, a.dx_lp, a.xhatF})) {
    const int rows = fused_rows(a.M, a.d);
    const int nblk = cdiv(a.M, rows);
    const bool tail = a.d % 1024 != 0;
    auto launch = [&](auto nc) {
      constexpr int C = decltype(nc)::value;
      if (dt == BF16) {
        if (tail) hipLaunchKernelGGL((ln_bwd_fused<bf16, C, true>), dim3(nblk), block, 0, s, a, rows);
        else hipLaunchKernelGGL((ln_bwd_fused<bf16, C, false>), dim3(nblk), block, 0, s, a, rows);
      } else {
        if (tail) hipLaunchKernelGGL((ln_bwd_fused<float, C, true>), dim3(nblk), block, 0, s, a, rows);
        else hipLaunchKernelGGL((ln_bwd_fused<float, C, false>), dim3(nblk), block, 0, s, a, rows);
      }
    };
    switch (cdiv(a.d, 1024)) {
      case 1: launch(std::integral_constant<int, 1>{}); break;
      case 2: launch(std::integral_constant<int, 2>{}); break;
      case 3: launch(std::integral_constant<int, 3>{}); break;
      default: launch(std::integral_constant<int, 4>{}); break;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    ColReduceArgs r{};
    r.part = a.partials; r.nblk = nblk; r.stride = (int64_t)6 * a.d; r.d = a.d;
    float* outs[6] = {a.dg1, a.db1, a.dg2, a.db2, a.dgF, a.dbF};
    const int src[6] = {0, 1, 2, 3, 3, 3};  // dbF == db2 == sum dy2 (dgF is NULL here)
    for (int k = 0; k < 6; ++k) { r.out[k] = outs[k]; r.src[k] = src[k]; }
    hipLaunchKernelGGL(col_reduce_multi, dim3(cdiv(a.d, 64), 6), dim3(64 * kRedWaves), 0, s, r);
    return hipGetLastError();
  }
  if (vec_ok(dt, a.d, {a.x, a.dy1, a.dy2, a.dres, a.dx, a.dacc, a.dxhatF_acc}, {a.g1, a.g2, a.gF, a.dx_lp}))
    e = dispatch_nc(a.d, [&](auto nc) {
      constexpr int C = decltype(nc)::value;
      if (dt == BF16) hipLaunchKernelGGL((ln_bwd_v4<bf16, C>), grid, block, 0, s, a);
      else hipLaunchKernelGGL((ln_bwd_v4<float, C>), grid, block, 0, s, a);
      return hipGetLastError();
    });
  else
    e = dispatch_vpt(a.d, [&](auto vpt) {
      constexpr int V = decltype(vpt)::value;
      if (dt == BF16) hipLaunchKernelGGL((ln_bwd_rows<bf16, V>), grid, block, 0, s, a);
      else hipLaunchKernelGGL((ln_bwd_rows<float, V>), grid, block, 0, s, a);
      return hipGetLastError();
    });
  if (e != hipSuccess) return e;
  if (!any) return hipSuccess;
  if (a.d % 4) return hipErrorInvalidValue;
  const int nblk = cdiv(a.M, kPartRows);
  const dim3 pgrid(cdiv(a.d, 256), nblk);
  if (dt == BF16) hipLaunchKernelGGL((ln_param_partials<bf16>), pgrid, block, 0, s, a);
  else hipLaunchKernelGGL((ln_param_partials<float>), pgrid, block, 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  ColReduceArgs r{};
  r.part = a.partials; r.nblk = nblk; r.stride = (int64_t)6 * a.d; r.d = a.d;
  float* outs[6] = {a.dg1, a.db1, a.dg2, a.db2, a.dgF, a.dbF};
  const int src[6] = {0, 1, 2, 3, 4, 3};  // dbF == db2 == sum dy2
  for (int k = 0; k < 6; ++k) { r.out[k] = outs[k]; r.src[k] = src[k]; }
  hipLaunchKernelGGL(col_reduce_multi, dim3(cdiv(a.d, 64), 6), dim3(64 * kRedWaves), 0, s, r);
  return hipGetLastError();
}

hipError_t norm_bwd(DType dt, const float* A, const float* mean, const float* rstd, const float* dxhat, int M,
                    int d, const float* dres, float* da, void* da_lp, hipStream_t s) {
  const dim3 grid(cdiv(M, kRowsPerBlock)), block(256);
  auto run = [&](auto tag) {
    using S = decltype(tag);
    S* lp = static_cast<S*>(da_lp);
    if (vec_ok(dt, d, {A, dxhat, dres, da}, {da_lp}))
      return dispatch_nc(d, [&](auto nc) {
        constexpr int C = decltype(nc)::value;
        hipLaunchKernelGGL((norm_bwd_v4<S, C>), grid, block, 0, s, A, mean, rstd, dxhat, M, d, dres, da, lp);
        return hipGetLastError();
      });
    return dispatch_vpt(d, [&](auto vpt) {
      constexpr int V = decltype(vpt)::value;
      hipLaunchKernelGGL((norm_bwd_kernel<S, V>), grid, block, 0, s, A, mean, rstd, dxhat, M, d, dres, da, lp);
      return hipGetLastError();
    });
  };
  return dt == BF16 ? run(bf16{}) : run(float{});
}

// ------------------------------------------------------------- col_sum --
// Bias gradients: column sums in row blocks of kColRows (256 columns x 4
// row groups per workgroup, rows in order, groups combined in fixed order),
// then the fixed-order block reduce.  32-row blocks measured slower here
// (0.35 -> 0.38 ms per GPT-2-small step): the inputs are 4 to 12 times wider.
constexpr int kColRows = 64;

// One partial launch over every input (grid z = input)
// writing packed partial rows [block][W], W = sum of the widths, and one
// reduce over the packed columns that scatters each segment to its outputs.
struct ColSumPacked {
  ColSumInput in[kColSumMax];
  int off[kColSumMax + 1];  // packed column offset of each input; off[n] = W
  int n, M;
  float* part;
};

// Field by field with constant indices: any dynamic index into the by-value
// kernel argument (or a select between whole structs) copies it to scratch.
#define FAL_PICK(b, k, f) \
  ((k) == 0 ? (b).in[0].f : (k) == 1 ? (b).in[1].f : (k) == 2 ? (b).in[2].f : (b).in[3].f)

template <typename S>
__global__ __launch_bounds__(256) void col_sum_batch_partials(ColSumPacked b) {
  __shared__ float red[3][256];
  static_assert(kColSumMax == 4, "update FAL_PICK");
  const int k = blockIdx.z;
  ColSumInput in;
  in.x = FAL_PICK(b, k, x);
  in.ld = FAL_PICK(b, k, ld);
  in.N = FAL_PICK(b, k, N);
  in.f32 = FAL_PICK(b, k, f32);
  const int off = k == 0 ? b.off[0] : k == 1 ? b.off[1] : k == 2 ? b.off[2] : b.off[3];
  const int W = b.n == 1 ? b.off[1] : b.n == 2 ? b.off[2] : b.n == 3 ? b.off[3] : b.off[4];
  const int cl = threadIdx.x & 63, rg = threadIdx.x >> 6;
  const int j = blockIdx.x * 256 + cl * 4;
  if (blockIdx.x * 256 >= in.N) return;  // uniform: this input is narrower
  float s[4] = {0.f, 0.f, 0.f, 0.f};
  constexpr int RG = kColRows / 4;  // rows per thread
  const int r0 = blockIdx.y * kColRows + rg * RG, r1 = min(b.M, r0 + RG);
  if (j < in.N && r1 - r0 == RG) {
    // a whole row group: every row's load in flight before the first add
    if (in.f32) {
      const float* x = static_cast<const float*>(in.x) + (int64_t)r0 * in.ld + j;
      float4 v[RG];
#pragma unroll
      for (int r = 0; r < RG; ++r) v[r] = *reinterpret_cast<const float4*>(x + (int64_t)r * in.ld);
#pragma unroll
      for (int r = 0; r < RG; ++r) {
        s[0] += v[r].x; s[1] += v[r].y; s[2] += v[r].z; s[3] += v[r].w;
      }
    } else {
      const S* x = static_cast<const S*>(in.x) + (int64_t)r0 * in.ld + j;
      Raw4<S> v[RG];
#pragma unroll
      for (int r = 0; r < RG; ++r) v[r] = raw4<S>(x + (int64_t)r * in.ld);
#pragma unroll
      for (int r = 0; r < RG; ++r) {
        const float4 w = val4(v[r]);
        s[0] += w.x; s[1] += w.y; s[2] += w.z; s[3] += w.w;
      }
    }
  } else if (j < in.N) {
    // 4-column vector loads, several rows in flight
    if (in.f32) {
      const float* x = static_cast<const float*>(in.x);
#pragma unroll 4
      for (int r = r0; r < r1; ++r) {
        const float4 v = *reinterpret_cast<const float4*>(x + (int64_t)r * in.ld + j);
        s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
      }
    } else {
      const S* x = static_cast<const S*>(in.x);
#pragma unroll 4
      for (int r = r0; r < r1; ++r) {
        const float4 v = ld4s<S>(x + (int64_t)r * in.ld + j);
        s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
      }
    }
  }
  if (rg > 0) {
#pragma unroll
    for (int c = 0; c < 4; ++c) red[rg - 1][cl * 4 + c] = s[c];
  }
  __syncthreads();
  if (rg == 0 && j < in.N) {
    float v[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = ((s[c] + red[0][cl * 4 + c]) + red[1][cl * 4 + c]) + red[2][cl * 4 + c];
    *reinterpret_cast<float4*>(b.part + (int64_t)blockIdx.y * W + off + j) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

__global__ __launch_bounds__(64 * kRedWaves) void col_reduce_batch(ColSumPacked b, int nblk) {
  __shared__ float red[kRedWaves][64];
  const int W = b.n == 1 ? b.off[1] : b.n == 2 ? b.off[2] : b.n == 3 ? b.off[3] : b.off[4];
  const int col = blockIdx.x * 64 + (threadIdx.x & 63);
  const int q = threadIdx.x >> 6;
  float s = 0.f;
  if (col < W) {
#pragma unroll 8
    for (int blk = q; blk < nblk; blk += kRedWaves) s += b.part[(int64_t)blk * W + col];
  }
  red[q][threadIdx.x & 63] = s;
  __syncthreads();
  if (q == 0 && col < W) {
    const float v = tree_sum(red, threadIdx.x & 63);
#pragma unroll
    for (int k = 0; k < kColSumMax; ++k) {
      if (k < b.n && col >= b.off[k] && col < b.off[k + 1]) {
        float* o = b.in[k].out;
        float* o2 = b.in[k].out2;
        o[col - b.off[k]] = v;
        if (o2) o2[col - b.off[k]] = v;
      }
    }
  }
}

int64_t col_sum_batch_scratch(int M, int W) { return (int64_t)cdiv(M, kColRows) * W; }

hipError_t col_sum_batch(DType dt, const ColSumBatch& b, float* scratch, hipStream_t s) {
  if (b.n < 1 || b.n > kColSumMax || !scratch) return hipErrorInvalidValue;
  ColSumPacked p{};
  p.n = b.n;
  p.M = b.M;
  p.part = scratch;
  int w = 0, maxn = 0;
  for (int k = 0; k < b.n; ++k) {
    const ColSumInput& in = b.in[k];
    if (!in.x || !in.out || in.N % 4 || in.ld % 4 || in.N < 1) return hipErrorInvalidValue;
    // rows are read 4 columns at a time
    if (reinterpret_cast<uintptr_t>(in.x) % ((in.f32 || dt == F32) ? 16 : 8)) return hipErrorInvalidValue;
    p.in[k] = in;
    p.off[k] = w;
    w += in.N;
    maxn = std::max(maxn, in.N);
  }
  p.off[b.n] = w;
  const int nblk = cdiv(b.M, kColRows);
  const dim3 grid(cdiv(maxn, 256), nblk, b.n), block(256);
  if (dt == F32)
    hipLaunchKernelGGL((col_sum_batch_partials<float>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((col_sum_batch_partials<bf16>), grid, block, 0, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(col_reduce_batch, dim3(cdiv(w, 64)), dim3(64 * kRedWaves), 0, s, p, nblk);
  return hipGetLastError();
}

}  // namespace fal
