// LayerNorm kernels of the block (Eq. 1, Eq. 2 and the FAL+ equation):
//  * ln_fwd: one wavefront per row.  One pass over the fp32 residual row
//    gives mean and rstd and up to two normalised outputs with different
//    affine parameters.  FAL uses both outputs, since its MHA and MLP
//    LayerNorms read the same X_i (H1 = LN1(X_i), H2 = LN2(X_i) + F); FAL+
//    adds the per-block LayerNorm of the shared first-attention
//    normalisation to its MLP input in the same pass.
//  * ln_bwd: row kernel for the input gradient (both LayerNorms of one input
//    at once), plus a column kernel for gamma/beta gradients with a fixed
//    reduction order.
//  * norm_bwd: backward of the affine-free normalisation of A_1 (FAL+).
//  * col_sum: bias gradients.
// All of these are HBM-bound; rows are read with 64 consecutive elements
// per wavefront instruction.
#include "common.h"
#include "kernels.h"

namespace fal {

constexpr int kRowsPerBlock = 4;  // 4 wavefronts per 256-thread workgroup

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

// Column partial sums for the LayerNorm parameter gradients: workgroup
// (column chunk of 256, row block of kPartRows).  partials: [nblk][6][d].
constexpr int kPartRows = 64;

template <typename S>
__global__ __launch_bounds__(256) void ln_param_partials(LnBwdArgs a) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  const int rb = blockIdx.y;
  const int d = a.d;
  if (j >= d) return;
  const int r0 = rb * kPartRows, r1 = min(a.M, r0 + kPartRows);
  const S* xF = static_cast<const S*>(a.xhatF);
  float q[6] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int r = r0; r < r1; ++r) {
    const int64_t o = (int64_t)r * d + j;
    const float xh = (a.x[o] - a.mean[r]) * a.rstd[r];
    if (a.dy1) {
      const float dy = a.dy1[o];
      q[0] += dy * xh;
      q[1] += dy;
    }
    if (a.dy2) {
      const float dy = a.dy2[o];
      q[2] += dy * xh;
      q[3] += dy;
      if (xF) q[4] += dy * to_f(xF[o]);
    }
  }
  float* p = a.partials + (int64_t)rb * 6 * d;
#pragma unroll
  for (int k = 0; k < 6; ++k) p[(int64_t)k * d + j] = q[k];
}

// out[j] = sum_b part[b * stride + j], fixed order.
__global__ __launch_bounds__(256) void col_reduce_kernel(const float* part, int nblk, int64_t stride,
                                                         int d, float* out) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= d) return;
  float s = 0.f;
  for (int b = 0; b < nblk; ++b) s += part[(int64_t)b * stride + j];
  out[j] = s;
}

hipError_t col_reduce(const float* part, int nblk, int64_t stride, int d, float* out, hipStream_t s) {
  hipLaunchKernelGGL(col_reduce_kernel, dim3(cdiv(d, 256)), dim3(256), 0, s, part, nblk, stride, d, out);
  return hipGetLastError();
}

template <int VPT>
__global__ __launch_bounds__(256) void norm_bwd_kernel(const float* A, const float* mean,
                                                       const float* rstd, const float* dxhat, int M,
                                                       int d, float* da, int accumulate) {
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
    const float v = rs * (g[i] - s1 - xh[i] * s2);
    da[off + j] = accumulate ? da[off + j] + v : v;
  }
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
  return dispatch_vpt(a.d, [&](auto vpt) {
    constexpr int V = decltype(vpt)::value;
    if (dt == BF16) hipLaunchKernelGGL((ln_fwd_kernel<bf16, V>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((ln_fwd_kernel<float, V>), grid, block, 0, s, a);
    return hipGetLastError();
  });
}

int64_t ln_bwd_scratch(int M, int d) { return (int64_t)cdiv(M, kPartRows) * 6 * d; }

hipError_t ln_bwd(DType dt, const LnBwdArgs& a, hipStream_t s) {
  const dim3 grid(cdiv(a.M, kRowsPerBlock)), block(256);
  hipError_t e = dispatch_vpt(a.d, [&](auto vpt) {
    constexpr int V = decltype(vpt)::value;
    if (dt == BF16) hipLaunchKernelGGL((ln_bwd_rows<bf16, V>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((ln_bwd_rows<float, V>), grid, block, 0, s, a);
    return hipGetLastError();
  });
  if (e != hipSuccess) return e;
  const bool any = a.dg1 || a.db1 || a.dg2 || a.db2 || a.dgF || a.dbF;
  if (!any) return hipSuccess;
  const int nblk = cdiv(a.M, kPartRows);
  const dim3 pgrid(cdiv(a.d, 256), nblk);
  if (dt == BF16) hipLaunchKernelGGL((ln_param_partials<bf16>), pgrid, block, 0, s, a);
  else hipLaunchKernelGGL((ln_param_partials<float>), pgrid, block, 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  float* outs[6] = {a.dg1, a.db1, a.dg2, a.db2, a.dgF, a.dbF};
  const int src[6] = {0, 1, 2, 3, 4, 3};  // dbF == db2 == sum dy2
  for (int k = 0; k < 6; ++k) {
    if (!outs[k]) continue;
    e = col_reduce(a.partials + (int64_t)src[k] * a.d, nblk, (int64_t)6 * a.d, a.d, outs[k], s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t norm_bwd(const float* A, const float* mean, const float* rstd, const float* dxhat, int M,
                    int d, float* da, int accumulate, hipStream_t s) {
  const dim3 grid(cdiv(M, kRowsPerBlock)), block(256);
  return dispatch_vpt(d, [&](auto vpt) {
    constexpr int V = decltype(vpt)::value;
    hipLaunchKernelGGL((norm_bwd_kernel<V>), grid, block, 0, s, A, mean, rstd, dxhat, M, d, da, accumulate);
    return hipGetLastError();
  });
}

// ------------------------------------------------------------- col_sum --
constexpr int kColRows = 128;

template <typename S>
__global__ __launch_bounds__(256) void col_sum_partials(const S* x, int64_t ld, int M, int N, float* part) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= N) return;
  const int r0 = blockIdx.y * kColRows, r1 = min(M, r0 + kColRows);
  float s = 0.f;
  for (int r = r0; r < r1; ++r) s += to_f(x[(int64_t)r * ld + j]);
  part[(int64_t)blockIdx.y * N + j] = s;
}

int64_t col_sum_scratch(int M, int N) { return (int64_t)cdiv(M, kColRows) * N; }

hipError_t col_sum(DType dt, int in_f32, const void* x, int64_t ld, int M, int N, float* out,
                   float* scratch, hipStream_t s) {
  const int nblk = cdiv(M, kColRows);
  const dim3 grid(cdiv(N, 256), nblk), block(256);
  if (in_f32 || dt == F32)
    hipLaunchKernelGGL((col_sum_partials<float>), grid, block, 0, s, static_cast<const float*>(x), ld, M, N, scratch);
  else
    hipLaunchKernelGGL((col_sum_partials<bf16>), grid, block, 0, s, static_cast<const bf16*>(x), ld, M, N, scratch);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return col_reduce(scratch, nblk, N, N, out, s);
}

}  // namespace fal
