// Dense GEMMs of the training step: the four linear layers of a block
// (QKV, output projection, FFN up, FFN down; Sec. 2), their data- and
// weight-gradient products, and the tied LM head.
//
// Two kernels share one problem descriptor (kernels.h):
//  * gemm_bf16_mfma: bf16 operands, fp32 accumulation on the gfx950 matrix
//    cores (v_mfma_f32_16x16x32_bf16).  128x128 output tile per 256-thread
//    workgroup, 2x2 wavefronts of 64x64, K staged through LDS 64 at a time
//    in k-contiguous rows.  Operands whose contraction dimension is strided
//    (the weight of a forward layer, both operands of a weight gradient) are
//    transposed in registers on their way into LDS.
//  * gemm_simt: fp32 FMA kernel (fp32 parity mode).
// Both launch every problem of a group in one grid, so the independent
// GEMMs of FAL's two branches can share a launch.
#include "common.h"
#include "kernels.h"

namespace fal {

template <typename S>
__device__ __forceinline__ void epilogue(const GemmProblem& P, int m, int n, float v, int gelu_tanh) {
  if (m >= P.M || n >= P.N) return;
  if (P.bias) v += to_f(static_cast<const S*>(P.bias)[n]);
  if (P.bias2) v += to_f(static_cast<const S*>(P.bias2)[n]);
  switch (P.epi) {
    case EPI_STORE:
      if (P.out_f32)
        static_cast<float*>(P.out)[(int64_t)m * P.ldo + n] = v;
      else
        static_cast<S*>(P.out)[(int64_t)m * P.ldo + n] = from_f<S>(v);
      break;
    case EPI_GELU:
      static_cast<S*>(P.out2)[(int64_t)m * P.ldo2 + n] = from_f<S>(v);
      static_cast<S*>(P.out)[(int64_t)m * P.ldo + n] = from_f<S>(gelu_f(v, gelu_tanh));
      break;
    case EPI_RESID: {
      float* o = static_cast<float*>(P.out) + (int64_t)m * P.ldo + n;
      *o = P.resid[(int64_t)m * P.ldr + n] + v;
      break;
    }
    case EPI_GELU_BWD: {
      const float pre = to_f(static_cast<const S*>(P.aux)[(int64_t)m * P.ldaux + n]);
      static_cast<S*>(P.out)[(int64_t)m * P.ldo + n] = from_f<S>(v * gelu_grad_f(pre, gelu_tanh));
      break;
    }
  }
}

// The problem owning workgroup `tile`, selected with constant indices so the
// descriptor stays in scalar registers (a dynamic index into the by-value
// array would copy it to scratch).
__device__ __forceinline__ GemmProblem find_problem(const GemmGroup& g, int tile) {
  static_assert(kMaxGroup == 4, "update find_problem");
  if (g.n > 3 && tile >= g.p[3].tile_start) return g.p[3];
  if (g.n > 2 && tile >= g.p[2].tile_start) return g.p[2];
  if (g.n > 1 && tile >= g.p[1].tile_start) return g.p[1];
  return g.p[0];
}

// ------------------------------------------------------------ SIMT (fp32) --
constexpr int ST = 64, SK = 16;

template <typename S, int AK, int BKM>
__global__ __launch_bounds__(256) void gemm_simt(GemmGroup g, int gelu_tanh) {
  __shared__ float As[SK][ST + 4];
  __shared__ float Bs[SK][ST + 4];
  const GemmProblem P = find_problem(g, blockIdx.x);
  const int local = blockIdx.x - P.tile_start;
  const int m0 = (local / P.tiles_n) * ST, n0 = (local % P.tiles_n) * ST;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  float acc[4][4] = {};
  for (int seg = 0; seg < 2; ++seg) {
    const S* A = static_cast<const S*>(seg ? P.A2 : P.A);
    const S* B = static_cast<const S*>(seg ? P.B2 : P.B);
    const int64_t lda = seg ? P.lda2 : P.lda, ldb = seg ? P.ldb2 : P.ldb;
    const int K = seg ? P.K2 : P.K;
    for (int k0 = 0; k0 < K; k0 += SK) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = tid + 256 * i;
        int mm, kk;
        if (AK) { mm = e / SK; kk = e % SK; } else { kk = e / ST; mm = e % ST; }
        const int m = m0 + mm, k = k0 + kk;
        float v = 0.f;
        if (m < P.M && k < K) v = to_f(A[AK ? (int64_t)m * lda + k : (int64_t)k * lda + m]);
        As[kk][mm] = v;
        int nn;
        if (BKM) { nn = e / SK; kk = e % SK; } else { kk = e / ST; nn = e % ST; }
        const int n = n0 + nn, k2 = k0 + kk;
        float w = 0.f;
        if (n < P.N && k2 < K) w = to_f(B[BKM ? (int64_t)n * ldb + k2 : (int64_t)k2 * ldb + n]);
        Bs[kk][nn] = w;
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < SK; ++kk) {
        float a[4], b[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) { a[i] = As[kk][ty * 4 + i]; b[i] = Bs[kk][tx * 4 + i]; }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
      }
      __syncthreads();
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) epilogue<S>(P, m0 + ty * 4 + i, n0 + tx * 4 + j, acc[i][j], gelu_tanh);
}

// ----------------------------------------------------------- MFMA (bf16) --
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int MT = 128, NT = 128, KT = 64, LDK = KT + 8;  // LDS row: 72 bf16 = 144 B

// Rows r0.. of a k-contiguous operand: 128 rows x 64 k = 1024 16-byte chunks,
// 4 per thread.  Chunks past K are zero-filled element-wise.
__device__ __forceinline__ void load_kmaj(uint4 (&r)[4], const bf16* X, int64_t ld, int r0, int R,
                                          int k0, int K, int tid) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i, row = c >> 3, kc = (c & 7) * 8;
    const int gr = r0 + row, gk = k0 + kc;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (gr < R && gk < K) {
      v = *reinterpret_cast<const uint4*>(X + (int64_t)gr * ld + gk);
      if (gk + 8 > K) {
        uint16_t* e = reinterpret_cast<uint16_t*>(&v);
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (gk + q >= K) e[q] = 0;
      }
    }
    r[i] = v;
  }
}

__device__ __forceinline__ void store_kmaj(const uint4 (&r)[4], bf16* s, int tid) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i, row = c >> 3, kc = (c & 7) * 8;
    *reinterpret_cast<uint4*>(s + row * LDK + kc) = r[i];
  }
}

// Rows r0.. of an operand whose rows are contiguous along m (or n): 64 k
// rows x 128 columns.  Thread: 4 consecutive k x 8 consecutive columns.
__device__ __forceinline__ void load_mnmaj(uint4 (&r)[4], const bf16* X, int64_t ld, int r0, int R,
                                           int k0, int K, int tid) {
  const int kg = (tid & 15) * 4, mc = (tid >> 4) * 8;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int gk = k0 + kg + j, gr = r0 + mc;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (gk < K && gr < R) v = *reinterpret_cast<const uint4*>(X + (int64_t)gk * ld + gr);
    r[j] = v;
  }
}

// Transpose the 4 (k) x 8 (column) block in registers and store it as 8
// k-contiguous LDS rows of 4 elements.
__device__ __forceinline__ void store_mnmaj(const uint4 (&r)[4], bf16* s, int tid) {
  const int kg = (tid & 15) * 4, mc = (tid >> 4) * 8;
  const uint32_t* w0 = reinterpret_cast<const uint32_t*>(&r[0]);
  const uint32_t* w1 = reinterpret_cast<const uint32_t*>(&r[1]);
  const uint32_t* w2 = reinterpret_cast<const uint32_t*>(&r[2]);
  const uint32_t* w3 = reinterpret_cast<const uint32_t*>(&r[3]);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    // columns 2q (low halves) and 2q+1 (high halves)
    uint2 lo, hi;
    lo.x = (w0[q] & 0xFFFFu) | (w1[q] << 16);
    lo.y = (w2[q] & 0xFFFFu) | (w3[q] << 16);
    hi.x = (w0[q] >> 16) | (w1[q] & 0xFFFF0000u);
    hi.y = (w2[q] >> 16) | (w3[q] & 0xFFFF0000u);
    *reinterpret_cast<uint2*>(s + (mc + 2 * q) * LDK + kg) = lo;
    *reinterpret_cast<uint2*>(s + (mc + 2 * q + 1) * LDK + kg) = hi;
  }
}

// Epilogue of one wavefront's 64x64 accumulator block; one instantiation per
// epilogue kind keeps every accumulator index a compile-time constant.
template <int EPI, int F32OUT>
__device__ __forceinline__ void store_tiles(const GemmProblem& P, const f32x4_t (&acc)[4][4], int mb, int nb,
                                            int gelu_tanh) {
  const bf16* bias = static_cast<const bf16*>(P.bias);
  const bf16* bias2 = static_cast<const bf16*>(P.bias2);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = nb + j * 16;
    if (n >= P.N) continue;
    float bn = 0.f;
    if (bias) bn += to_f(bias[n]);
    if (bias2) bn += to_f(bias2[n]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb + i * 16 + r;
        if (m >= P.M) continue;
        const float v = acc[i][j][r] + bn;
        const int64_t o = (int64_t)m * P.ldo + n;
        if (EPI == EPI_STORE) {
          if (F32OUT) static_cast<float*>(P.out)[o] = v;
          else static_cast<bf16*>(P.out)[o] = from_f<bf16>(v);
        } else if (EPI == EPI_GELU) {
          static_cast<bf16*>(P.out2)[(int64_t)m * P.ldo2 + n] = from_f<bf16>(v);
          static_cast<bf16*>(P.out)[o] = from_f<bf16>(gelu_f(v, gelu_tanh));
        } else if (EPI == EPI_RESID) {
          static_cast<float*>(P.out)[o] = P.resid[(int64_t)m * P.ldr + n] + v;
        } else {
          const float pre = to_f(static_cast<const bf16*>(P.aux)[(int64_t)m * P.ldaux + n]);
          static_cast<bf16*>(P.out)[o] = from_f<bf16>(v * gelu_grad_f(pre, gelu_tanh));
        }
      }
  }
}

template <int AK, int BKM>
__global__ __launch_bounds__(256, 2) void gemm_bf16_mfma(GemmGroup g, int gelu_tanh) {
  __shared__ __attribute__((aligned(16))) bf16 sA[MT * LDK];
  __shared__ __attribute__((aligned(16))) bf16 sB[NT * LDK];
  const GemmProblem P = find_problem(g, blockIdx.x);
  const int local = blockIdx.x - P.tile_start;
  const int m0 = (local / P.tiles_n) * MT, n0 = (local % P.tiles_n) * NT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nt1 = (P.K + KT - 1) / KT;
  const int nt = nt1 + (P.K2 > 0 ? (P.K2 + KT - 1) / KT : 0);
  uint4 ra[4], rb[4];

  auto fetch = [&](int t) {
    const int seg = t >= nt1;
    const bf16* A = static_cast<const bf16*>(seg ? P.A2 : P.A);
    const bf16* B = static_cast<const bf16*>(seg ? P.B2 : P.B);
    const int64_t lda = seg ? P.lda2 : P.lda, ldb = seg ? P.ldb2 : P.ldb;
    const int K = seg ? P.K2 : P.K;
    const int k0 = (seg ? t - nt1 : t) * KT;
    if (AK) load_kmaj(ra, A, lda, m0, P.M, k0, K, tid);
    else load_mnmaj(ra, A, lda, m0, P.M, k0, K, tid);
    if (BKM) load_kmaj(rb, B, ldb, n0, P.N, k0, K, tid);
    else load_mnmaj(rb, B, ldb, n0, P.N, k0, K, tid);
  };

  fetch(0);
  for (int t = 0; t < nt; ++t) {
    if (AK) store_kmaj(ra, sA, tid); else store_mnmaj(ra, sA, tid);
    if (BKM) store_kmaj(rb, sB, tid); else store_mnmaj(rb, sB, tid);
    __syncthreads();
    if (t + 1 < nt) fetch(t + 1);
#pragma unroll
    for (int ks = 0; ks < KT / 32; ++ks) {
      bf16x8_t a[4], b[4];
      const int koff = ks * 32 + (lane >> 4) * 8;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        a[i] = *reinterpret_cast<const bf16x8_t*>(sA + (wm * 64 + i * 16 + (lane & 15)) * LDK + koff);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        b[j] = *reinterpret_cast<const bf16x8_t*>(sB + (wn * 64 + j * 16 + (lane & 15)) * LDK + koff);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }

  // acc[i][j][r] holds C[row 4*(lane/16) + r][col lane%16] of 16x16 tile (i, j).
  const int mb = m0 + wm * 64 + (lane >> 4) * 4, nb = n0 + wn * 64 + (lane & 15);
  switch (P.epi) {
    case EPI_STORE:
      if (P.out_f32) store_tiles<EPI_STORE, 1>(P, acc, mb, nb, gelu_tanh);
      else store_tiles<EPI_STORE, 0>(P, acc, mb, nb, gelu_tanh);
      break;
    case EPI_GELU: store_tiles<EPI_GELU, 0>(P, acc, mb, nb, gelu_tanh); break;
    case EPI_RESID: store_tiles<EPI_RESID, 1>(P, acc, mb, nb, gelu_tanh); break;
    case EPI_GELU_BWD: store_tiles<EPI_GELU_BWD, 0>(P, acc, mb, nb, gelu_tanh); break;
  }
}

// ------------------------------------------------------------- launcher --
static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

static const char* check_vec_operand(const void* X, int64_t ld, int kmaj, int rows, int K) {
  if (!X) return "GEMM operand is NULL";
  if (!aligned16(X)) return "GEMM operand not 16-byte aligned";
  if (ld % 8) return "GEMM leading dimension not a multiple of 8";
  if (kmaj) {
    if (ld < ((K + 7) / 8) * 8) return "GEMM k-contiguous leading dimension too small";
  } else {
    if (ld < ((rows + 7) / 8) * 8) return "GEMM row-contiguous leading dimension too small";
  }
  return nullptr;
}

hipError_t gemm(DType dt, int a_kmaj, int b_kmaj, GemmGroup& g, int gelu_tanh, hipStream_t s,
                const char** why) {
  *why = nullptr;
  if (g.n < 1 || g.n > kMaxGroup) { *why = "bad GEMM group size"; return hipErrorInvalidValue; }
  const int tm = dt == BF16 ? MT : ST, tn = dt == BF16 ? NT : ST;
  int total = 0;
  for (int i = 0; i < g.n; ++i) {
    GemmProblem& P = g.p[i];
    if (P.M <= 0 || P.N <= 0 || P.K <= 0 || P.K2 < 0) { *why = "bad GEMM shape"; return hipErrorInvalidValue; }
    if (dt == BF16) {
      const char* e = check_vec_operand(P.A, P.lda, a_kmaj, P.M, P.K);
      if (!e) e = check_vec_operand(P.B, P.ldb, b_kmaj, P.N, P.K);
      if (!e && P.K2 > 0) e = check_vec_operand(P.A2, P.lda2, a_kmaj, P.M, P.K2);
      if (!e && P.K2 > 0) e = check_vec_operand(P.B2, P.ldb2, b_kmaj, P.N, P.K2);
      if (e) { *why = e; return hipErrorInvalidValue; }
    }
    P.tiles_m = (P.M + tm - 1) / tm;
    P.tiles_n = (P.N + tn - 1) / tn;
    P.tile_start = total;
    total += P.tiles_m * P.tiles_n;
  }
  g.total_tiles = total;
  const dim3 grid(total), block(256);
#define FAL_GEMM_LAUNCH(KERNEL)                                                              \
  if (a_kmaj && b_kmaj) hipLaunchKernelGGL((KERNEL<1, 1>), grid, block, 0, s, g, gelu_tanh); \
  else if (a_kmaj) hipLaunchKernelGGL((KERNEL<1, 0>), grid, block, 0, s, g, gelu_tanh);      \
  else if (b_kmaj) hipLaunchKernelGGL((KERNEL<0, 1>), grid, block, 0, s, g, gelu_tanh);      \
  else hipLaunchKernelGGL((KERNEL<0, 0>), grid, block, 0, s, g, gelu_tanh);
  if (dt == BF16) {
    FAL_GEMM_LAUNCH(gemm_bf16_mfma)
  } else {
    if (a_kmaj && b_kmaj) hipLaunchKernelGGL((gemm_simt<float, 1, 1>), grid, block, 0, s, g, gelu_tanh);
    else if (a_kmaj) hipLaunchKernelGGL((gemm_simt<float, 1, 0>), grid, block, 0, s, g, gelu_tanh);
    else if (b_kmaj) hipLaunchKernelGGL((gemm_simt<float, 0, 1>), grid, block, 0, s, g, gelu_tanh);
    else hipLaunchKernelGGL((gemm_simt<float, 0, 0>), grid, block, 0, s, g, gelu_tanh);
  }
#undef FAL_GEMM_LAUNCH
  return hipGetLastError();
}

}  // namespace fal
