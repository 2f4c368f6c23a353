// Scaled-dot-product attention per head (the MHA of Sec. 2), causal or (for
// the bidirectional encoder blocks) unmasked, in the blockwise form with an
// online softmax so that the T x T score matrix is never stored
// (FlashAttention, which the paper uses on its GPUs).
//
// This file holds the SIMT kernels: fp32 arithmetic on fp32 or bf16
// storage, any head_dim in {16, 32, 64, 128}.  A workgroup holds 64 query
// (or key) rows with 4 lanes per row, each lane owning head_dim/4 of the
// row; K/V (or Q/dO) tiles of 64 rows are staged in LDS.
//
// Backward is deterministic without atomics: one kernel accumulates dK, dV
// per key block over the query blocks that see it (at or after it when
// causal); a second kernel accumulates dQ per query block over the key
// blocks it sees.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace fal {

constexpr int ABR = 64;  // rows per tile

template <typename S, int HD>
__global__ __launch_bounds__(256) void attn_fwd_simt(const S* qkv, int T, int H, int Hkv, int causal, S* O,
                                                     int64_t ldo, float* lse) {
  constexpr int P = HD / 4;
  __shared__ float Ks[ABR][HD + 1];
  __shared__ float Vs[ABR][HD + 1];
  // grid (H, B, blocks): causal block index slowest (even XCD mix), the
  // longest (latest) query blocks first
  const int qb = gridDim.z - 1 - blockIdx.z;
  const int h = blockIdx.x, b = blockIdx.y;
  const int dA = H * HD, dKV = Hkv * HD;
  const int64_t ld = dA + 2 * (int64_t)dKV;
  const int kcol = dA + (h / (H / Hkv)) * HD, vcol = kcol + dKV;  // the group's key/value head
  const int tid = threadIdx.x, r = tid >> 2, part = tid & 3;
  const int t = qb * ABR + r;
  const bool valid = t < T;
  const float scale = 1.f / sqrtf((float)HD);
  const S* base = qkv + (int64_t)b * T * ld;
  float q[P], o[P];
#pragma unroll
  for (int c = 0; c < P; ++c) {
    q[c] = valid ? to_f(base[(int64_t)t * ld + h * HD + part * P + c]) * scale : 0.f;
    o[c] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int kend = causal ? min(T, qb * ABR + ABR) : T;
  for (int k0 = 0; k0 < kend; k0 += ABR) {
    for (int e = tid; e < ABR * HD; e += 256) {
      const int kr = e / HD, c = e % HD, key = k0 + kr;
      const bool ok = key < T;
      Ks[kr][c] = ok ? to_f(base[(int64_t)key * ld + kcol + c]) : 0.f;
      Vs[kr][c] = ok ? to_f(base[(int64_t)key * ld + vcol + c]) : 0.f;
    }
    __syncthreads();
    float sc[ABR];
    float mt = -INFINITY;
#pragma unroll
    for (int j = 0; j < ABR; ++j) {
      float p = 0.f;
#pragma unroll
      for (int c = 0; c < P; ++c) p = fmaf(q[c], Ks[j][part * P + c], p);
      p += __shfl_xor(p, 1, FAL_WAVE);
      p += __shfl_xor(p, 2, FAL_WAVE);
      const int key = k0 + j;
      sc[j] = ((!causal || key <= t) && key < T) ? p : -INFINITY;
      mt = fmaxf(mt, sc[j]);
    }
    if (mt > -INFINITY) {
      const float mn = fmaxf(m, mt);
      const float corr = expf(m - mn);
      l *= corr;
#pragma unroll
      for (int c = 0; c < P; ++c) o[c] *= corr;
#pragma unroll
      for (int j = 0; j < ABR; ++j) {
        const float p = expf(sc[j] - mn);
        l += p;
#pragma unroll
        for (int c = 0; c < P; ++c) o[c] = fmaf(p, Vs[j][part * P + c], o[c]);
      }
      m = mn;
    }
    __syncthreads();
  }
  if (valid) {
    const float inv = 1.f / l;
    S* orow = O + ((int64_t)b * T + t) * ldo + h * HD + part * P;
#pragma unroll
    for (int c = 0; c < P; ++c) orow[c] = from_f<S>(o[c] * inv);
    if (part == 0) lse[((int64_t)b * H + h) * T + t] = m + logf(l);
  }
}

// D[b, h, t] = sum_c dO[t, h*HD + c] * O[t, h*HD + c]; consecutive threads
// take consecutive heads of one row, reading 8 elements at a time.
template <typename S>
__global__ __launch_bounds__(256) void attn_bwd_dot(const S* O, int64_t ldo, const S* dO, int64_t lddo,
                                                    int B, int T, int H, int HD, float* Dvec) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * H * T) return;
  const int h = i % H;
  const int64_t row = i / H;
  const int t = row % T, b = row / T;
  const S* o = O + row * ldo + h * HD;
  const S* g = dO + row * lddo + h * HD;
  float s = 0.f;
  for (int c = 0; c < HD; c += 8) {
    S a[8], e[8];
    *reinterpret_cast<uint4*>(a) = *reinterpret_cast<const uint4*>(o + c);
    *reinterpret_cast<uint4*>(e) = *reinterpret_cast<const uint4*>(g + c);
    if (sizeof(S) == 4) {
      *reinterpret_cast<uint4*>(a + 4) = *reinterpret_cast<const uint4*>(o + c + 4);
      *reinterpret_cast<uint4*>(e + 4) = *reinterpret_cast<const uint4*>(g + c + 4);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) s += to_f(a[j]) * to_f(e[j]);
  }
  Dvec[((int64_t)b * H + h) * T + t] = s;
}

template <typename S, int HD>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_simt(const S* qkv, const S* dO, int64_t lddo,
                                                          const float* lse, const float* Dvec, int T,
                                                          int H, int Hkv, int causal, S* dqkv) {
  constexpr int P = HD / 4;
  __shared__ float Qs[ABR][HD + 1];
  __shared__ float dOs[ABR][HD + 1];
  __shared__ float Ls[ABR], Ds[ABR];
  // grid (Hkv, B, blocks), causal block index slowest; a key/value head
  // accumulates over the query heads of its group in order
  const int kb = blockIdx.z, kvh = blockIdx.x, b = blockIdx.y, grp = H / Hkv;
  const int dA = H * HD, dKV = Hkv * HD;
  const int64_t ld = dA + 2 * (int64_t)dKV;
  const int kcol = dA + kvh * HD, vcol = kcol + dKV;
  const int tid = threadIdx.x, r = tid >> 2, part = tid & 3;
  const int key = kb * ABR + r;
  const bool valid = key < T;
  const float scale = 1.f / sqrtf((float)HD);
  const S* base = qkv + (int64_t)b * T * ld;
  const S* dObase = dO + (int64_t)b * T * lddo;
  float k[P], v[P], dk[P], dv[P];
#pragma unroll
  for (int c = 0; c < P; ++c) {
    k[c] = valid ? to_f(base[(int64_t)key * ld + kcol + part * P + c]) : 0.f;
    v[c] = valid ? to_f(base[(int64_t)key * ld + vcol + part * P + c]) : 0.f;
    dk[c] = 0.f;
    dv[c] = 0.f;
  }
  for (int h = kvh * grp; h < (kvh + 1) * grp; ++h) {
    const float* lrow = lse + ((int64_t)b * H + h) * T;
    const float* drow = Dvec + ((int64_t)b * H + h) * T;
    for (int q0 = causal ? kb * ABR : 0; q0 < T; q0 += ABR) {
      for (int e = tid; e < ABR * HD; e += 256) {
        const int qr = e / HD, c = e % HD, tq = q0 + qr;
        const bool ok = tq < T;
        Qs[qr][c] = ok ? to_f(base[(int64_t)tq * ld + h * HD + c]) : 0.f;
        dOs[qr][c] = ok ? to_f(dObase[(int64_t)tq * lddo + h * HD + c]) : 0.f;
      }
      if (tid < ABR) {
        const int tq = q0 + tid;
        Ls[tid] = tq < T ? lrow[tq] : 0.f;
        Ds[tid] = tq < T ? drow[tq] : 0.f;
      }
      __syncthreads();
#pragma unroll 4
      for (int j = 0; j < ABR; ++j) {
        const int tq = q0 + j;
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int c = 0; c < P; ++c) {
          s = fmaf(Qs[j][part * P + c], k[c], s);
          dp = fmaf(dOs[j][part * P + c], v[c], dp);
        }
        s += __shfl_xor(s, 1, FAL_WAVE);
        s += __shfl_xor(s, 2, FAL_WAVE);
        dp += __shfl_xor(dp, 1, FAL_WAVE);
        dp += __shfl_xor(dp, 2, FAL_WAVE);
        const float p = (valid && tq < T && (!causal || tq >= key)) ? expf(s * scale - Ls[j]) : 0.f;
        const float ds = p * (dp - Ds[j]) * scale;
#pragma unroll
        for (int c = 0; c < P; ++c) {
          dv[c] = fmaf(p, dOs[j][part * P + c], dv[c]);
          dk[c] = fmaf(ds, Qs[j][part * P + c], dk[c]);
        }
      }
      __syncthreads();
    }
  }
  if (valid) {
    S* row = dqkv + ((int64_t)b * T + key) * ld;
#pragma unroll
    for (int c = 0; c < P; ++c) {
      row[kcol + part * P + c] = from_f<S>(dk[c]);
      row[vcol + part * P + c] = from_f<S>(dv[c]);
    }
  }
}

template <typename S, int HD>
__global__ __launch_bounds__(256) void attn_bwd_dq_simt(const S* qkv, const S* dO, int64_t lddo,
                                                        const float* lse, const float* Dvec, int T,
                                                        int H, int Hkv, int causal, S* dqkv) {
  constexpr int P = HD / 4;
  __shared__ float Ks[ABR][HD + 1];
  __shared__ float Vs[ABR][HD + 1];
  // grid (H, B, blocks): the causal block index varies slowest, so the
  // round-robin dispatch over XCDs gives every XCD the same mix of long and
  // short blocks; the longest (latest) query blocks are dispatched first.
  const int qb = gridDim.z - 1 - blockIdx.z;
  const int h = blockIdx.x, b = blockIdx.y;
  const int dA = H * HD, dKV = Hkv * HD;
  const int64_t ld = dA + 2 * (int64_t)dKV;
  const int kcol = dA + (h / (H / Hkv)) * HD, vcol = kcol + dKV;
  const int tid = threadIdx.x, r = tid >> 2, part = tid & 3;
  const int t = qb * ABR + r;
  const bool valid = t < T;
  const float scale = 1.f / sqrtf((float)HD);
  const S* base = qkv + (int64_t)b * T * ld;
  float q[P], g[P], dq[P];
#pragma unroll
  for (int c = 0; c < P; ++c) {
    q[c] = valid ? to_f(base[(int64_t)t * ld + h * HD + part * P + c]) : 0.f;
    g[c] = valid ? to_f(dO[((int64_t)b * T + t) * lddo + h * HD + part * P + c]) : 0.f;
    dq[c] = 0.f;
  }
  const float L = valid ? lse[((int64_t)b * H + h) * T + t] : 0.f;
  const float Dt = valid ? Dvec[((int64_t)b * H + h) * T + t] : 0.f;
  const int kend = causal ? min(T, qb * ABR + ABR) : T;
  for (int k0 = 0; k0 < kend; k0 += ABR) {
    for (int e = tid; e < ABR * HD; e += 256) {
      const int kr = e / HD, c = e % HD, key = k0 + kr;
      const bool ok = key < T;
      Ks[kr][c] = ok ? to_f(base[(int64_t)key * ld + kcol + c]) : 0.f;
      Vs[kr][c] = ok ? to_f(base[(int64_t)key * ld + vcol + c]) : 0.f;
    }
    __syncthreads();
#pragma unroll 4
    for (int j = 0; j < ABR; ++j) {
      const int key = k0 + j;
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int c = 0; c < P; ++c) {
        s = fmaf(q[c], Ks[j][part * P + c], s);
        dp = fmaf(g[c], Vs[j][part * P + c], dp);
      }
      s += __shfl_xor(s, 1, FAL_WAVE);
      s += __shfl_xor(s, 2, FAL_WAVE);
      dp += __shfl_xor(dp, 1, FAL_WAVE);
      dp += __shfl_xor(dp, 2, FAL_WAVE);
      const float p = (valid && (!causal || key <= t) && key < T) ? expf(s * scale - L) : 0.f;
      const float ds = p * (dp - Dt) * scale;
#pragma unroll
      for (int c = 0; c < P; ++c) dq[c] = fmaf(ds, Ks[j][part * P + c], dq[c]);
    }
    __syncthreads();
  }
  if (valid) {
    S* row = dqkv + ((int64_t)b * T + t) * ld + h * HD + part * P;
#pragma unroll
    for (int c = 0; c < P; ++c) row[c] = from_f<S>(dq[c]);
  }
}

template <typename F>
static hipError_t dispatch_hd(int hd, F&& f) {
  switch (hd) {
    case 16: return f(std::integral_constant<int, 16>{});
    case 32: return f(std::integral_constant<int, 32>{});
    case 64: return f(std::integral_constant<int, 64>{});
    case 128: return f(std::integral_constant<int, 128>{});
  }
  return hipErrorInvalidValue;
}

bool attn_mfma_supported(int hd);
hipError_t attn_fwd_mfma_launch(const void* qkv, int B, int T, int H, int Hkv, int hd, int causal, void* O,
                                int64_t ldo, float* lse, hipStream_t s);
hipError_t attn_bwd_mfma_launch(const void* qkv, const void* O, int64_t ldo, const void* dO, int64_t lddo,
                                const float* lse, float* Dvec, int B, int T, int H, int Hkv, int hd, int causal,
                                void* dqkv, hipStream_t s);

hipError_t attn_fwd(DType dt, const void* qkv, int B, int T, int H, int Hkv, int hd, int causal, void* O,
                    int64_t ldo, float* lse, hipStream_t s) {
  if (Hkv < 1 || H % Hkv) return hipErrorInvalidValue;
  if (dt == BF16 && attn_mfma_supported(hd))
    return attn_fwd_mfma_launch(qkv, B, T, H, Hkv, hd, causal, O, ldo, lse, s);
  const dim3 grid(H, B, cdiv(T, ABR)), block(256);
  return dispatch_hd(hd, [&](auto c) {
    constexpr int HD = decltype(c)::value;
    if (dt == BF16)
      hipLaunchKernelGGL((attn_fwd_simt<bf16, HD>), grid, block, 0, s, static_cast<const bf16*>(qkv), T, H,
                         Hkv, causal, static_cast<bf16*>(O), ldo, lse);
    else
      hipLaunchKernelGGL((attn_fwd_simt<float, HD>), grid, block, 0, s, static_cast<const float*>(qkv), T,
                         H, Hkv, causal, static_cast<float*>(O), ldo, lse);
    return hipGetLastError();
  });
}

hipError_t attn_bwd(DType dt, const void* qkv, const void* O, int64_t ldo, const void* dO,
                    int64_t lddo, const float* lse, int B, int T, int H, int Hkv, int hd, int causal, void* dqkv,
                    float* Dvec, float* dq_acc, hipStream_t s) {
  (void)dq_acc;
  if (Hkv < 1 || H % Hkv) return hipErrorInvalidValue;
  // the matrix-core dQ kernel computes D itself
  if (dt == BF16 && attn_mfma_supported(hd))
    return attn_bwd_mfma_launch(qkv, O, ldo, dO, lddo, lse, Dvec, B, T, H, Hkv, hd, causal, dqkv, s);
  const int64_t nrows = (int64_t)B * H * T;
  if (dt == BF16)
    hipLaunchKernelGGL((attn_bwd_dot<bf16>), dim3(cdiv(nrows, 256)), dim3(256), 0, s,
                       static_cast<const bf16*>(O), ldo, static_cast<const bf16*>(dO), lddo, B, T, H, hd, Dvec);
  else
    hipLaunchKernelGGL((attn_bwd_dot<float>), dim3(cdiv(nrows, 256)), dim3(256), 0, s,
                       static_cast<const float*>(O), ldo, static_cast<const float*>(dO), lddo, B, T, H, hd, Dvec);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 grid(H, B, cdiv(T, ABR)), gkv(Hkv, B, cdiv(T, ABR)), block(256);
  return dispatch_hd(hd, [&](auto c) {
    constexpr int HD = decltype(c)::value;
    if (dt == BF16) {
      hipLaunchKernelGGL((attn_bwd_dkdv_simt<bf16, HD>), gkv, block, 0, s, static_cast<const bf16*>(qkv),
                         static_cast<const bf16*>(dO), lddo, lse, Dvec, T, H, Hkv, causal, static_cast<bf16*>(dqkv));
      hipLaunchKernelGGL((attn_bwd_dq_simt<bf16, HD>), grid, block, 0, s, static_cast<const bf16*>(qkv),
                         static_cast<const bf16*>(dO), lddo, lse, Dvec, T, H, Hkv, causal, static_cast<bf16*>(dqkv));
    } else {
      hipLaunchKernelGGL((attn_bwd_dkdv_simt<float, HD>), gkv, block, 0, s, static_cast<const float*>(qkv),
                         static_cast<const float*>(dO), lddo, lse, Dvec, T, H, Hkv, causal, static_cast<float*>(dqkv));
      hipLaunchKernelGGL((attn_bwd_dq_simt<float, HD>), grid, block, 0, s, static_cast<const float*>(qkv),
                         static_cast<const float*>(dO), lddo, lse, Dvec, T, H, Hkv, causal, static_cast<float*>(dqkv));
    }
    return hipGetLastError();
  });
}

}  // namespace fal
