// Dense GEMMs of the training step: the four linear layers of a block
// (QKV, output projection, FFN up, FFN down; Sec. 2), their data- and
// weight-gradient products, and the tied LM head.
//
// All kernels share one problem descriptor (kernels.h):
//  * gemm_bf16_dbl / gemm_bf16_pipe: bf16 operands, fp32 accumulation on the
//    gfx950 matrix cores (v_mfma_f32_16x16x32_bf16), operand slices copied
//    from global memory straight into LDS; operands whose contraction
//    dimension is strided (the weight of a forward layer, both operands of a
//    weight gradient) are read back with LDS transpose loads.  The epilogue
//    (bias, GELU and its derivative, residual add, GELU-derivative product)
//    runs on row segments staged through LDS so every global access covers
//    whole wavefront-tile rows.  Operands are addressed with 32-bit buffer
//    offsets: every operand must span less than 2 GiB (the library's config
//    check guarantees it; the launcher rejects anything else).
//  * gemm_simt: fp32 FMA kernel (fp32 parity mode).
// Every kernel launches all problems of a group in one grid, so the
// independent GEMMs of FAL's two branches can share a launch.
#include <algorithm>

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
    case EPI_GELU: {
      float gv, dg;
      gelu_and_grad(v, gelu_tanh, gv, dg);
      if (P.out2) static_cast<S*>(P.out2)[(int64_t)m * P.ldo2 + n] = from_f<S>(dg);
      static_cast<S*>(P.out)[(int64_t)m * P.ldo + n] = from_f<S>(gv);
      break;
    }
    case EPI_RESID: {
      float* o = static_cast<float*>(P.out) + (int64_t)m * P.ldo + n;
      *o = P.resid[(int64_t)m * P.ldr + n] + v;
      break;
    }
    case EPI_MUL_AUX: {
      const float a = to_f(static_cast<const S*>(P.aux)[(int64_t)m * P.ldaux + n]);
      static_cast<S*>(P.out)[(int64_t)m * P.ldo + n] = from_f<S>(v * a);
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

constexpr int kRsrcWord3 = 0x00020000;  // gfx9-family buffer descriptor word 3

// An operand whose contraction dimension is strided (MN-major: the weight of
// a forward layer, both operands of a weight gradient) is staged as loaded,
// [k][row], and read back with the gfx950 LDS transpose load.
// ds_read_b64_tr_b16 gives lane i of each 16-lane group element i % 4 of the
// 8-byte chunks addressed by lanes 4j + i / 4 (j = 0..3); lane L therefore
// addresses k-row kb + L / 4, rows 4 (L % 4)..+3 of the fragment, and two
// reads (kb, kb + 4) return the eight consecutive k a 16x16x32 operand lane
// holds.
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

__device__ __forceinline__ i16x4_t lds_read_tr(const bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_i16x4_t*)((__attribute__((address_space(3))) char*)(const_cast<bf16*>(p))));
}

__device__ __forceinline__ void ld4(const bf16* p, float (&v)[4]) {
  const uint2 w = *reinterpret_cast<const uint2*>(p);
  v[0] = __uint_as_float(w.x << 16); v[1] = __uint_as_float(w.x & 0xFFFF0000u);
  v[2] = __uint_as_float(w.y << 16); v[3] = __uint_as_float(w.y & 0xFFFF0000u);
}
__device__ __forceinline__ void st4(bf16* p, const float (&v)[4]) {
  union { bf16 h[4]; uint2 w; } u;
#pragma unroll
  for (int c = 0; c < 4; ++c) u.h[c] = from_f<bf16>(v[c]);
  *reinterpret_cast<uint2*>(p) = u.w;
}

// Epilogue of one row segment of four columns: v = accumulator (+ bias),
// row m, columns n..n+3 (those < N).  full: all four in range and the rows
// allow vector access.
template <int EPI, int F32OUT>
__device__ __forceinline__ void apply4(const GemmProblem& P, int m, int n, float (&v)[4], bool full, int gelu_tanh) {
  const int64_t o = (int64_t)m * P.ldo + n;
  if (full) {
    if (EPI == EPI_STORE) {
      if (F32OUT) *reinterpret_cast<float4*>(static_cast<float*>(P.out) + o) = make_float4(v[0], v[1], v[2], v[3]);
      else st4(static_cast<bf16*>(P.out) + o, v);
    } else if (EPI == EPI_GELU) {
      float g[4], dg[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) gelu_and_grad(v[c], gelu_tanh, g[c], dg[c]);
      if (P.out2) st4(static_cast<bf16*>(P.out2) + (int64_t)m * P.ldo2 + n, dg);
      st4(static_cast<bf16*>(P.out) + o, g);
    } else if (EPI == EPI_RESID) {
      const float4 r = *reinterpret_cast<const float4*>(P.resid + (int64_t)m * P.ldr + n);
      *reinterpret_cast<float4*>(static_cast<float*>(P.out) + o) =
          make_float4(r.x + v[0], r.y + v[1], r.z + v[2], r.w + v[3]);
    } else {
      float a[4];
      ld4(static_cast<const bf16*>(P.aux) + (int64_t)m * P.ldaux + n, a);
#pragma unroll
      for (int c = 0; c < 4; ++c) v[c] *= a[c];
      st4(static_cast<bf16*>(P.out) + o, v);
    }
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (n + c >= P.N) continue;
      const int64_t oc = o + c;
      if (EPI == EPI_STORE) {
        if (F32OUT) static_cast<float*>(P.out)[oc] = v[c];
        else static_cast<bf16*>(P.out)[oc] = from_f<bf16>(v[c]);
      } else if (EPI == EPI_GELU) {
        float g, dg;
        gelu_and_grad(v[c], gelu_tanh, g, dg);
        if (P.out2) static_cast<bf16*>(P.out2)[(int64_t)m * P.ldo2 + n + c] = from_f<bf16>(dg);
        static_cast<bf16*>(P.out)[oc] = from_f<bf16>(g);
      } else if (EPI == EPI_RESID) {
        static_cast<float*>(P.out)[oc] = P.resid[(int64_t)m * P.ldr + n + c] + v[c];
      } else {
        const float a = to_f(static_cast<const bf16*>(P.aux)[(int64_t)m * P.ldaux + n + c]);
        static_cast<bf16*>(P.out)[oc] = from_f<bf16>(v[c] * a);
      }
    }
  }
}

__device__ __forceinline__ void bias4(const GemmProblem& P, int n, bool full, float (&bn)[4]) {
  const bf16* bias = static_cast<const bf16*>(P.bias);
  const bf16* bias2 = static_cast<const bf16*>(P.bias2);
#pragma unroll
  for (int c = 0; c < 4; ++c) bn[c] = 0.f;
  if (full) {
    float t[4];
    if (bias) { ld4(bias + n, t); for (int c = 0; c < 4; ++c) bn[c] += t[c]; }
    if (bias2) { ld4(bias2 + n, t); for (int c = 0; c < 4; ++c) bn[c] += t[c]; }
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (n + c < P.N) bn[c] = (bias ? to_f(bias[n + c]) : 0.f) + (bias2 ? to_f(bias2[n + c]) : 0.f);
  }
}

// Orders this wavefront's LDS writes before its later reads (and reads
// before later writes) without a workgroup barrier: LDS executes one
// wavefront's instructions in order, so only compiler motion must be stopped.
__device__ __forceinline__ void wave_lds_order() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Epilogue through a wavefront-private LDS strip.  One 16-row strip of the
// wavefront tile at a time is written from the accumulators and read back
// with consecutive lanes on consecutive columns, so every global access
// (output, residual, GELU derivative) covers whole row segments of the
// wavefront tile (256 B of bf16 for a 128-column tile).  The accumulators
// are transposed blocks (the MFMA ran as B^T A^T): lane 16g+c of block
// (i, j) holds row 16i + c, columns 16j + 4g .. +3, written to the strip as
// one 16-byte store.
//
// A wavefront tile that lies wholly inside the output takes the fast path
// (plain stores, residual add, GELU-derivative product): each strip's
// read-back passes are issued together, and the rows an epilogue reads (the
// residual, the GELU derivative) for strip i + 1 are loaded while strip i
// is computed and stored, so their memory latency is paid about once per
// tile instead of once per pass.  Edge tiles and the GELU epilogue take the
// per-pass path with bounds checks.
template <int EPI, int F32OUT, int FM, int FN>
__device__ __forceinline__ void store_staged(const GemmProblem& P, const f32x4_t (&acc)[FM][FN], float* stage,
                                             int mw, int nw, int lane, int gelu_tanh) {
  constexpr int WTN = FN * 16, PITCH = WTN + 4;
  constexpr int LPR = WTN / 4, RPI = 64 / LPR;    // lanes per row, rows per access
  constexpr int NPASS = 16 / RPI;                 // accesses per 16-row strip
  static_assert(RPI * LPR == 64 && NPASS * RPI == 16, "strip shape");
  const int rr = lane / LPR, cc = (lane % LPR) * 4;  // read-back position
  const int n = nw + cc;
  const bool full = P.vec_out && n + 4 <= P.N;
  float bn[4];
  bias4(P, n, full, bn);
  auto write_strip = [&](int i) {
#pragma unroll
    for (int j = 0; j < FN; ++j)
      *reinterpret_cast<float4*>(stage + (lane & 15) * PITCH + 16 * j + 4 * (lane >> 4)) =
          make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
  };
  // GELU tiles keep the per-pass path: there the batched passes measured
  // slower (the GELU arithmetic, not memory latency, sets the pace)
  const bool inside = EPI != EPI_GELU && P.vec_out && mw + 16 * FM <= P.M && nw + WTN <= P.N;
  if (inside) {
    // operand rows the epilogue reads, one strip ahead
    constexpr int NA = EPI == EPI_MUL_AUX ? NPASS : 1;
    constexpr int NR = EPI == EPI_RESID ? NPASS : 1;
    uint2 aux[2][NA];
    float4 res[2][NR];
    auto prefetch = [&](int i, int buf) {
#pragma unroll
      for (int k = 0; k < NPASS; ++k) {
        const int64_t m = mw + 16 * i + k * RPI + rr;
        if (EPI == EPI_MUL_AUX)
          aux[buf][k] = *reinterpret_cast<const uint2*>(static_cast<const bf16*>(P.aux) + m * P.ldaux + n);
        if (EPI == EPI_RESID) res[buf][k] = *reinterpret_cast<const float4*>(P.resid + m * P.ldr + n);
      }
    };
    if (EPI == EPI_MUL_AUX || EPI == EPI_RESID) prefetch(0, 0);
    // fully unrolled whatever the body size: a rolled loop would index the
    // accumulators dynamically and move them to scratch
#pragma clang loop unroll(full)
    for (int i = 0; i < FM; ++i) {
      const int cur = i & 1;
      write_strip(i);
      wave_lds_order();
      float4 t[NPASS];
#pragma unroll
      for (int k = 0; k < NPASS; ++k) t[k] = *reinterpret_cast<const float4*>(stage + (k * RPI + rr) * PITCH + cc);
      wave_lds_order();
      if ((EPI == EPI_MUL_AUX || EPI == EPI_RESID) && i + 1 < FM) prefetch(i + 1, cur ^ 1);
#pragma unroll
      for (int k = 0; k < NPASS; ++k) {
        const int64_t m = mw + 16 * i + k * RPI + rr;
        const int64_t o = m * P.ldo + n;
        float v[4] = {t[k].x + bn[0], t[k].y + bn[1], t[k].z + bn[2], t[k].w + bn[3]};
        if (EPI == EPI_STORE) {
          if (F32OUT) *reinterpret_cast<float4*>(static_cast<float*>(P.out) + o) = make_float4(v[0], v[1], v[2], v[3]);
          else st4(static_cast<bf16*>(P.out) + o, v);
        } else if (EPI == EPI_RESID) {
          const float4 r = res[cur][k];
          *reinterpret_cast<float4*>(static_cast<float*>(P.out) + o) =
              make_float4(r.x + v[0], r.y + v[1], r.z + v[2], r.w + v[3]);
        } else {
          const uint2 w = aux[cur][k];
          const float a[4] = {__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xFFFF0000u),
                              __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xFFFF0000u)};
#pragma unroll
          for (int c = 0; c < 4; ++c) v[c] *= a[c];
          st4(static_cast<bf16*>(P.out) + o, v);
        }
      }
    }
    return;
  }
#pragma clang loop unroll(full)
  for (int i = 0; i < FM; ++i) {
    write_strip(i);
    wave_lds_order();
    // kept rolled: the edge path runs on few tiles, and unrolling it
    // multiplies its code (one copy per output kind)
#pragma unroll 1
    for (int k = 0; k < NPASS; ++k) {
      const int r = k * RPI + rr;
      const float4 t = *reinterpret_cast<const float4*>(stage + r * PITCH + cc);
      const int m = mw + 16 * i + r;
      if (m < P.M && n < P.N) {
        float v[4] = {t.x + bn[0], t.y + bn[1], t.z + bn[2], t.w + bn[3]};
        apply4<EPI, F32OUT>(P, m, n, v, full, gelu_tanh);
      }
    }
    wave_lds_order();
  }
}

#ifndef FAL_NS11
#define FAL_NS11 4
#endif
#ifndef FAL_NS10
#define FAL_NS10 4
#endif
#ifndef FAL_NS01
#define FAL_NS01 4
#endif
#ifndef FAL_NS00
#define FAL_NS00 5
#endif
#ifndef FAL_LATE_B
#define FAL_LATE_B 1
#endif
#ifndef FAL_GEMM_DBL
#define FAL_GEMM_DBL 1
#endif
#ifndef FAL_GEMM_REMAP
#define FAL_GEMM_REMAP 1
#endif
#ifndef FAL_OCC3_KMAX
#define FAL_OCC3_KMAX 1024  // longest K (both segments) sent to the three-workgroup kernel
#endif
#ifndef FAL_GEMM_GROUP_M
#define FAL_GEMM_GROUP_M 4
#endif
constexpr int kXcds = 8, kGroupM = FAL_GEMM_GROUP_M;
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  const int q = total / kXcds, r = total % kXcds;
  const int xcd = bid % kXcds, slot = bid / kXcds;
  return xcd < r ? xcd * (q + 1) + slot : r * (q + 1) + (xcd - r) * q + slot;
}
__device__ __forceinline__ void grouped_tile(int t, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int band = kGroupM * tiles_n;
  const int first = (t / band) * kGroupM;
  const int gs = min(kGroupM, tiles_m - first);
  const int in = t % band;
  tm = first + in % gs;
  tn = in / gs;
}

// ------------------------------------- MFMA (bf16), direct-to-LDS pipeline --
// Four wavefronts (one per SIMD) own a BM x BN output tile as 2 x 2
// wavefront tiles of (BM/2) x (BN/2).  K advances in slices of 32 (one
// 16x16x32 MFMA step).  Each slice of both operands is copied from global
// memory straight into one of four LDS stages by buffer loads with the LDS
// destination (no registers, no LDS store instructions), three slices ahead
// of the slice being multiplied; the fragments of slice s + 1 are read while
// the MFMAs of slice s run.  One workgroup barrier per slice.
//
// LDS layout of one operand in one stage (R rows of the output dimension):
//  * k-contiguous operand: R rows of 32 k (64 B), 16-byte chunk c of row r
//    stored at chunk c ^ ((r >> 2) & 3): the 16 rows of a fragment read
//    (one chunk each) fall in 16 different 16-byte bank groups.
//  * MN-major operand: 32 k-rows of R elements, 32-byte segment q of k-row k
//    stored at segment q ^ g(k), g(k) = (k & 3) | ((k >> 3) & 1) << 2: the
//    16 k-rows touched by one transposing read hit each 32-byte bank group
//    exactly twice (the minimum for 512 bytes).
// A buffer load writes lane l's 16 bytes at LDS offset 16 l of its 1 KiB
// block, so the swizzle is applied by choosing which global chunk each lane
// fetches.  Rows past M / N and k past K read outside the buffer's range and
// land as zeros; k past K inside a k-contiguous row is pointed out of range.
namespace pipe {
constexpr int KS = 32;
constexpr uint32_t kOob = 0x80000000u;      // offset beyond any buffer range (ranges are < 2^31)

__device__ __forceinline__ int mn_g(int k) { return (k & 3) | (((k >> 3) & 1) << 2); }

typedef __attribute__((address_space(3))) void lds_void_t;
__device__ __forceinline__ lds_void_t* lds_ptr(const void* p) {
  return (lds_void_t*)((__attribute__((address_space(3))) char*)(const_cast<void*>(p)));
}

// One operand's loader (both K segments) for slices W wide in K (32 or
// 64).  Load block i of this wavefront is block 4 i + wave of the stage
// region; its global offset is a per-lane part (which repeats with period
// NV in i) plus a wave-uniform step per i.
//  * k-contiguous: a block holds RPI = 1024 / 2W rows of W k; the 16-byte
//    chunk c of row r sits at c ^ kswz(r), kswz(r) = (r >> 2) & 3 for
//    64-byte rows and (r >> 1) & 7 for 128-byte rows.
//  * MN-major: a block holds 1024 / 2R k-rows of R elements, 32-byte
//    segment q of k-row k at q ^ g(k).
template <int W>
__device__ __forceinline__ int kswz(int r) { return W == 32 ? (r >> 2) & 3 : (r >> 1) & 7; }

template <int R, int KMAJ, int W = KS>
struct Src {
  static constexpr int BYTES = R * W * 2;                  // one stage region
  static constexpr int NINS = BYTES / 1024;                // 1 KiB load blocks per slice
  static constexpr int IPW = NINS / 4;                     // per wavefront
  static constexpr int CPR = R / 8;                        // MN-major: 16-byte chunks per k-row
  static constexpr int CPRK = W / 8;                       // k-contiguous: 16-byte chunks per row
  static constexpr int RPI = KMAJ ? 1024 / (2 * W) : 1024 / (2 * R);  // rows / k-rows per block
  // MN-major: the swizzle g(k) of a lane's k-row repeats every 16 k-rows
  static constexpr int NV = KMAJ ? 1 : ((4 * RPI) % 16 == 0 ? 1 : 16 / (4 * RPI));
  static_assert(NINS % 4 == 0 && IPW % NV == 0, "tile too small for four wavefronts");
  uint32_t voff[2][NV];    // per segment
  uint32_t istep[2];       // bytes from block i to block i + 1 of this wavefront
  int kof;                 // k-contiguous: k offset of this lane's chunk within the slice
  uint64_t base[2];
  int nbytes[2];
  uint32_t kstep[2];       // bytes per k (k-contiguous: 2; MN-major: 2 ld)

  __device__ __forceinline__ void init(int seg, const bf16* X, int64_t ld, int r0, int Rmax, int Kseg, int wave,
                                       int lane) {
    base[seg] = reinterpret_cast<uint64_t>(KMAJ ? X + (int64_t)r0 * ld : X + r0);
    const int64_t ext = KMAJ ? (int64_t)(Rmax - r0) * ld * 2 : ((int64_t)Kseg * ld - r0) * 2;
    nbytes[seg] = (int)min<int64_t>(ext, 0x7fffffff);
    kstep[seg] = KMAJ ? 2u : (uint32_t)(ld * 2);
    istep[seg] = (uint32_t)(4 * RPI * ld * 2);
    if (KMAJ) {
      // kswz(row) does not depend on the block index i (rows advance by 4 RPI)
      const int row = wave * RPI + lane / CPRK;
      const int gc = (lane % CPRK) ^ kswz<W>(row);
      voff[seg][0] = (uint32_t)(((int64_t)row * ld + gc * 8) * 2);
      kof = gc * 8;
    } else {
      kof = 0;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int k = (4 * v + wave) * RPI + lane / CPR;
        const int gc = (lane % CPR) ^ (2 * mn_g(k));
        voff[seg][v] = (uint32_t)(((int64_t)k * ld + gc * 8) * 2);
      }
    }
  }
  __device__ __forceinline__ void clear(int seg) {
    base[seg] = base[0];
    nbytes[seg] = 0;
    kstep[seg] = istep[seg] = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v) voff[seg][v] = kOob;
  }

  // Load state: the slice the next load() fetches.
  uint32_t rlo, rhi;
  int rn;
  uint32_t so, is, ks;
  uint32_t vo[NV];
  // Point the state at the slice at k0 of segment seg; chunks at slice
  // offset >= lim are pointed out of range (lim: 0 for a slice past the
  // end, K - k0 in a k-contiguous tail slice, W otherwise).
  __device__ __forceinline__ void set(int seg, int k0, int lim) {
    const uint64_t b = seg ? base[1] : base[0];
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    rlo = lo;
    rhi = hi;
    rn = __builtin_amdgcn_readfirstlane(seg ? nbytes[1] : nbytes[0]);
    ks = __builtin_amdgcn_readfirstlane(seg ? kstep[1] : kstep[0]);
    so = (uint32_t)k0 * ks;
    is = __builtin_amdgcn_readfirstlane(seg ? istep[1] : istep[0]);
    const bool bad = kof >= lim;
#pragma unroll
    for (int v = 0; v < NV; ++v) vo[v] = bad ? kOob : (seg ? voff[1][v] : voff[0][v]);
  }
  // Next slice of the same segment (full and live).
  __device__ __forceinline__ void advance() { so += W * ks; }
  // Issue this wavefront's loads of the current slice into the region at dst.
  __device__ __forceinline__ void load(char* dst, int wave) const {
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(((uint64_t)rhi << 32) | rlo), (short)0, rn, kRsrcWord3);
    // (the offsets go through locals: with member expressions as builtin
    // arguments the host pass drops the kernel's launch stubs)
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
      const uint32_t v = vo[i % NV];
      const uint32_t o = so + (uint32_t)(i - i % NV) * is;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds_ptr(dst + (i * 4 + wave) * 1024), 16, v, o, 0, 0);
    }
  }
};

// Fragment reads from one stage region (byte addresses precomputed per
// lane); fragment f of MFMA k-step kk (0 .. W/32 - 1).
template <int R, int KMAJ, int NF, int W = KS>
struct Frag {
  static constexpr int NKK = W / 32;
  uint32_t off[KMAJ ? NKK : NF];
  // row0: first row of fragment 0 within the region (the wavefront tile's base)
  __device__ __forceinline__ void init(int row0, int lane) {
    if (KMAJ) {
      const int row = row0 + (lane & 15);
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk)
        off[kk] = (uint32_t)(row * 2 * W + ((((4 * kk + (lane >> 4)) ^ kswz<W>(row))) << 4));
    } else {
      const int k = 8 * (lane >> 4) + ((lane & 15) >> 2);
      const int g2 = 2 * mn_g(k);
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        const int mn0 = row0 + 16 * f;
        off[f] = (uint32_t)(k * 2 * R + (((((mn0 >> 3) ^ g2) + ((lane & 3) >> 1))) << 4) + 8 * (lane & 1));
      }
    }
  }
  __device__ __forceinline__ bf16x8_t read(const char* region, int f, int kk = 0) const {
    if (KMAJ) return *reinterpret_cast<const bf16x8_t*>(region + off[kk] + f * 16 * 2 * W);
    const bf16* p = reinterpret_cast<const bf16*>(region + off[f]) + kk * 32 * R;
    const i16x4_t lo = lds_read_tr(p), hi = lds_read_tr(p + 4 * R);
    const i16x4_t v8[2] = {lo, hi};
    return *reinterpret_cast<const bf16x8_t*>(v8);
  }
};

// s_waitcnt with vmcnt(v) and lgkmcnt(l) (gfx9 encoding; expcnt not waited)
#define FAL_WAITCNT(v, l) __builtin_amdgcn_s_waitcnt(((v) & 15) | (((v) >> 4) << 14) | (7 << 4) | ((l) << 8))
__device__ __forceinline__ void bar() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
}  // namespace pipe

template <int AK, int BKM, int BM, int BN, int OCC, int NS>
__global__ __launch_bounds__(256, OCC) void gemm_bf16_pipe(GemmGroup g, int gelu_tanh) {
  using namespace pipe;
  static_assert(NS >= 3 && NS <= 8, "stage count");
  constexpr int WTM = BM / 2, WTN = BN / 2;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  typedef Src<BM, AK> SA;
  typedef Src<BN, BKM> SB;
  constexpr int SBYTES = SA::BYTES + SB::BYTES;
  constexpr int L = SA::IPW + SB::IPW;  // loads per wavefront per slice
  static_assert(L * (NS - 2) <= 63, "vmcnt range");
  // one array per stage: the compiler tracks buffer-to-LDS loads per array
  // (arrays past NS are 16-byte placeholders)
  constexpr int SB4 = NS > 4 ? SBYTES : 16, SB5 = NS > 5 ? SBYTES : 16, SB6 = NS > 6 ? SBYTES : 16,
                SB7 = NS > 7 ? SBYTES : 16;
  __shared__ __attribute__((aligned(1024))) char st0[SBYTES], st1[SBYTES], st2[SBYTES], st3[SBYTES], st4[SB4],
      st5[SB5], st6[SB6], st7[SB7];
  auto stage_ptr = [&](int k) -> char* {
    switch (k) {
      case 0: return st0;
      case 1: return st1;
      case 2: return st2;
      case 3: return st3;
      case 4: return st4;
      case 5: return st5;
      case 6: return st6;
      default: return st7;
    }
  };

#if FAL_GEMM_REMAP
  const int bid = xcd_remap(blockIdx.x, g.total_tiles);
#else
  const int bid = blockIdx.x;
#endif
  const GemmProblem P = find_problem(g, bid);
  const int per_split = P.tiles_m * P.tiles_n;
  const int local = (bid - P.tile_start) % per_split;
  const int split = (bid - P.tile_start) / per_split;
  int tmi, tni;
  grouped_tile(local, P.tiles_m, P.tiles_n, tmi, tni);
  const int m0 = tmi * BM, n0 = tni * BN;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // slices: segment 0 is [0, nt1), segment 1 is [nt1, nt)
  const int nt1 = (P.K + KS - 1) / KS;
  int sbeg = 0, send = nt1 + (P.K2 > 0 ? (P.K2 + KS - 1) / KS : 0);
  if (P.splits > 1) {
    const int per = (nt1 + P.splits - 1) / P.splits;
    sbeg = min(nt1, split * per);
    send = min(nt1, sbeg + per);
  }
  const int n = send - sbeg;

  SA sa;
  SB sb;
  sa.init(0, static_cast<const bf16*>(P.A), P.lda, m0, P.M, P.K, wave, lane);
  sb.init(0, static_cast<const bf16*>(P.B), P.ldb, n0, P.N, P.K, wave, lane);
  if (P.K2 > 0) {
    sa.init(1, static_cast<const bf16*>(P.A2), P.lda2, m0, P.M, P.K2, wave, lane);
    sb.init(1, static_cast<const bf16*>(P.B2), P.ldb2, n0, P.N, P.K2, wave, lane);
  } else {  // never selected; an empty range all the same
    sa.clear(1);
    sb.clear(1);
  }
  // Slices s with f_lo < s < f_hi are full, live and in the segment of the
  // current load state: the loader only advances.  Others (segment start,
  // k tail, past the end) recompute the state.
  int f_lo = 0, f_hi = 0;
  const int full0 = P.K / KS, full1 = nt1 + P.K2 / KS;
  auto issue = [&](char* stage, int s) {
    if (s > f_lo && s < f_hi) {
      sa.advance();
      sb.advance();
    } else {
      const bool live = s < send;
      const int seg = live && s >= nt1 ? 1 : 0;
      const int k0 = live ? (seg ? s - nt1 : s) * KS : 0;
      const int Kseg = seg ? P.K2 : P.K;
      // k-contiguous operands read whole 8-element chunks up to Kpad
      const int Kpad = P.kpad ? (Kseg + 7) / 8 * 8 : Kseg;
      const int lim = !live ? 0 : k0 + KS > Kpad ? Kpad - k0 : KS;
      sa.set(seg, k0, AK ? lim : (live ? KS : 0));
      sb.set(seg, k0, BKM ? lim : (live ? KS : 0));
      f_lo = s;
      f_hi = live && k0 + KS <= Kseg ? min(send, seg ? full1 : full0) : s;
    }
    sa.load(stage, wave);
    sb.load(stage + SA::BYTES, wave);
  };

  Frag<BM, AK, FM> fa;
  Frag<BN, BKM, FN> fb;
  fa.init(wm * WTM, lane);
  fb.init(wn * WTN, lane);

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  bf16x8_t ra[2][FM], rb[2][FN];

  // B's fragments of the next slice: all at the start of a step (two slices
  // live at once), or each right after its last use in the step's final row
  constexpr bool LATE_B = FAL_LATE_B;
  auto read = [&](const char* stage, int buf) {
#pragma unroll
    for (int i = 0; i < FM; ++i) ra[buf][i] = fa.read(stage, i);
#pragma unroll
    for (int j = 0; j < FN; ++j) rb[buf][j] = fb.read(stage + SA::BYTES, j);
  };
  // MFMAs of the slice in buffer `cur` with the fragment reads of the next
  // slice (from `stage`) into buffer cur ^ 1: B's fragments first, spread
  // over the first MFMAs; A's fragment i right after the last MFMA that uses
  // A's current fragment i, so the two can share registers.
  auto step = [&](const char* stage, int cur) {
    const int nxt = cur ^ 1;
    if (!LATE_B) {
#pragma unroll
      for (int j = 0; j < FN; ++j) rb[nxt][j] = fb.read(stage + SA::BYTES, j);
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rb[cur][j], ra[cur][i], acc[i][j], 0, 0, 0);
        if (LATE_B && i == FM - 1) rb[nxt][j] = fb.read(stage + SA::BYTES, j);
      }
      ra[nxt][i] = fa.read(stage, i);
    }
  };
  // Issue order inside a step (scheduling groups, in order): per MFMA of
  // slice s, then B's reads of slice s + 1 one per MFMA, A's read i after
  // MFMA row i, and the loads of slice s + 3 spread evenly.
  constexpr int NRB = BKM ? FN : 2 * FN;  // LDS read instructions for B
  constexpr int RA = AK ? 1 : 2;          // per A fragment
  constexpr int NMF = FM * FN;
  constexpr int DMA_EVERY = NMF / L > 0 ? NMF / L : 1;
  static_assert(NRB <= NMF, "more B reads than MFMAs");
  constexpr int RBJ = NRB / FN;           // LDS read instructions per B fragment
  auto interleave = [&]() {
    int dma = 0;
#pragma unroll
    for (int q = 0; q < NMF; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      if (LATE_B) {
        if (q >= NMF - FN) {
#pragma unroll
          for (int r = 0; r < RBJ; ++r) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read (B)
        }
      } else if (q < NRB) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read (B)
      }
      if ((q + 1) % FN == 0) {
#pragma unroll
        for (int r = 0; r < RA; ++r) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read (A)
      }
      if (q % DMA_EVERY == 0 && dma < L) {
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // buffer load to LDS
        ++dma;
      }
    }
  };
  // The reads issued by a step (the last A reads, and with LATE_B all of
  // B's) may still be in flight at the next step's barrier; reads of the
  // slice before (whose stage is refilled after the barrier) are older and
  // complete.  The counter field holds at most 15.
  constexpr int LGK_N = FM * RA + (LATE_B ? NRB : 0);
  constexpr int LGK = LGK_N < 15 ? LGK_N : 15;

  if (n > 0) {
    // prologue: slices sbeg .. sbeg+NS-2 into stages 0..NS-2; slice sbeg's fragments
#pragma unroll
    for (int k = 0; k < NS - 1; ++k) issue(stage_ptr(k), sbeg + k);
    FAL_WAITCNT(L * (NS - 2), 0);
    bar();
    read(st0, 0);
    // step s: wait for own loads of slice s + 1 and own reads of slice s - 1,
    // barrier (slice s + 1 complete in LDS; slice s - 1's stage free), load
    // slice s + NS - 1 into that stage, MFMAs of slice s with slice s + 1's
    // reads.  Unrolled over a whole number of stage cycles and register
    // buffer pairs, so every stage and buffer index is a constant.
    constexpr int UNR = NS % 2 ? 2 * NS : NS;
    // The slice count is rounded up to whole unrolled groups: slices past
    // the end load zeros in both operands and add nothing.
    const int tend = sbeg + ((n + UNR - 1) / UNR) * UNR;
    for (int t = sbeg; t < tend; t += UNR) {
#pragma unroll
      for (int U = 0; U < UNR; ++U) {
        const int s = t + U;
        FAL_WAITCNT(L * (NS - 3), LGK);
        bar();
        __builtin_amdgcn_sched_barrier(0);
        issue(stage_ptr((U + NS - 1) % NS), s + NS - 1);
        step(stage_ptr((U + 1) % NS), U & 1);
        interleave();
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  // every load (including those past the end) has landed and every
  // wavefront is done with the stages before they are reused for staging
  FAL_WAITCNT(0, 0);
  bar();

  float* stage = reinterpret_cast<float*>(wm ? st1 : st0) + wn * 16 * (WTN + 4);
  static_assert(2 * 16 * (WTN + 4) * 4 <= SBYTES, "epilogue staging exceeds a stage");
  const int mw = m0 + wm * WTM, nw = n0 + wn * WTN;
  if (P.splits > 1) {
    GemmProblem Q = P;
    Q.out = P.part + (int64_t)split * P.M * P.N;
    Q.ldo = P.N;
    Q.bias = Q.bias2 = nullptr;
    Q.vec_out = (P.N & 3) == 0;
    store_staged<EPI_STORE, 1, FM, FN>(Q, acc, stage, mw, nw, lane, gelu_tanh);
    return;
  }
  switch (P.epi) {
    case EPI_STORE:
      if (P.out_f32) store_staged<EPI_STORE, 1, FM, FN>(P, acc, stage, mw, nw, lane, gelu_tanh);
      else store_staged<EPI_STORE, 0, FM, FN>(P, acc, stage, mw, nw, lane, gelu_tanh);
      break;
    case EPI_GELU: store_staged<EPI_GELU, 0, FM, FN>(P, acc, stage, mw, nw, lane, gelu_tanh); break;
    case EPI_RESID: store_staged<EPI_RESID, 1, FM, FN>(P, acc, stage, mw, nw, lane, gelu_tanh); break;
    case EPI_MUL_AUX: store_staged<EPI_MUL_AUX, 0, FM, FN>(P, acc, stage, mw, nw, lane, gelu_tanh); break;
  }
}

// The same tile shapes with 64-wide K slices in two LDS stages.  A
// k-contiguous operand then arrives as whole 128-byte lines per row (a
// 32-wide slice takes half a line from twice as many rows per load, which
// measured slow with operands coming from HBM).  Step s: wait for own
// loads of slice s + 1 and own fragment reads of slice s, barrier, refill
// slice s's stage with slice s + 2, then the MFMAs of slice s with every
// fragment read of slice s + 1 issued among the first of them.  The load
// lead is one step (two MFMA k-steps), the same time as the three-slice
// lead of the four-stage kernel.
template <int AK, int BKM, int BM, int BN, int OCC>
__global__ __launch_bounds__(256, OCC) void gemm_bf16_dbl(GemmGroup g, int gelu_tanh) {
  using namespace pipe;
  constexpr int W = 64, NKK = W / 32;
  constexpr int WTM = BM / 2, WTN = BN / 2;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  typedef Src<BM, AK, W> SA;
  typedef Src<BN, BKM, W> SB;
  constexpr int SBYTES = SA::BYTES + SB::BYTES;
  constexpr int L = SA::IPW + SB::IPW;  // loads per wavefront per slice
  static_assert(L <= 63, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) char st0[SBYTES], st1[SBYTES];

#if FAL_GEMM_REMAP
  const int bid = xcd_remap(blockIdx.x, g.total_tiles);
#else
  const int bid = blockIdx.x;
#endif
  const GemmProblem P = find_problem(g, bid);
  const int per_split = P.tiles_m * P.tiles_n;
  const int local = (bid - P.tile_start) % per_split;
  const int split = (bid - P.tile_start) / per_split;
  int tmi, tni;
  grouped_tile(local, P.tiles_m, P.tiles_n, tmi, tni);
  const int m0 = tmi * BM, n0 = tni * BN;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // slices of W: segment 0 is [0, nt1), segment 1 is [nt1, nt)
  const int nt1 = (P.K + W - 1) / W;
  int sbeg = 0, send = nt1 + (P.K2 > 0 ? (P.K2 + W - 1) / W : 0);
  if (P.splits > 1) {
    const int per = (nt1 + P.splits - 1) / P.splits;
    sbeg = min(nt1, split * per);
    send = min(nt1, sbeg + per);
  }
  const int n = send - sbeg;

  SA sa;
  SB sb;
  sa.init(0, static_cast<const bf16*>(P.A), P.lda, m0, P.M, P.K, wave, lane);
  sb.init(0, static_cast<const bf16*>(P.B), P.ldb, n0, P.N, P.K, wave, lane);
  if (P.K2 > 0) {
    sa.init(1, static_cast<const bf16*>(P.A2), P.lda2, m0, P.M, P.K2, wave, lane);
    sb.init(1, static_cast<const bf16*>(P.B2), P.ldb2, n0, P.N, P.K2, wave, lane);
  } else {  // never selected; an empty range all the same
    sa.clear(1);
    sb.clear(1);
  }
  int f_lo = 0, f_hi = 0;
  const int full0 = P.K / W, full1 = nt1 + P.K2 / W;
  auto issue = [&](char* stage, int s) {
    if (s > f_lo && s < f_hi) {
      sa.advance();
      sb.advance();
    } else {
      // slices past the end use segment 0 at k 0 with every chunk out of range
      const bool live = s < send;
      const int seg = live && s >= nt1 ? 1 : 0;
      const int k0 = live ? (seg ? s - nt1 : s) * W : 0;
      const int Kseg = seg ? P.K2 : P.K;
      // k-contiguous operands read whole 8-element chunks up to Kpad
      const int Kpad = P.kpad ? (Kseg + 7) / 8 * 8 : Kseg;
      const int lim = !live ? 0 : k0 + W > Kpad ? Kpad - k0 : W;
      sa.set(seg, k0, AK ? lim : (live ? W : 0));
      sb.set(seg, k0, BKM ? lim : (live ? W : 0));
      f_lo = s;
      f_hi = live && k0 + W <= Kseg ? min(send, seg ? full1 : full0) : s;
    }
    sa.load(stage, wave);
    sb.load(stage + SA::BYTES, wave);
  };

  Frag<BM, AK, FM, W> fa;
  Frag<BN, BKM, FN, W> fb;
  fa.init(wm * WTM, lane);
  fb.init(wn * WTN, lane);

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  bf16x8_t ra[2][NKK][FM], rb[2][NKK][FN];
  auto read = [&](const char* stage, int buf) {
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
#pragma unroll
      for (int j = 0; j < FN; ++j) rb[buf][kk][j] = fb.read(stage + SA::BYTES, j, kk);
#pragma unroll
      for (int i = 0; i < FM; ++i) ra[buf][kk][i] = fa.read(stage, i, kk);
    }
  };
  auto mma = [&](int buf) {
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rb[buf][kk][j], ra[buf][kk][i], acc[i][j], 0, 0, 0);
  };
  // Issue order inside a step: one fragment read after each of the first
  // MFMAs, the loads spread over the rest.
  constexpr int NRD = NKK * ((AK ? FM : 2 * FM) + (BKM ? FN : 2 * FN));
  constexpr int NMF = NKK * FM * FN;
  constexpr int DMA_EVERY = (NMF - NRD) / L > 0 ? (NMF - NRD) / L : 1;
  static_assert(NRD <= NMF, "more fragment reads than MFMAs");
  auto interleave = [&]() {
    int dma = 0;
#pragma unroll
    for (int q = 0; q < NMF; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      if (q < NRD) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
      else if ((q - NRD) % DMA_EVERY == 0 && dma < L) {
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // buffer load to LDS
        ++dma;
      }
    }
  };

  if (n > 0) {
    issue(st0, sbeg);
    issue(st1, sbeg + 1);
    FAL_WAITCNT(L, 0);
    bar();
    read(st0, 0);
    // The slice count is rounded up to whole pairs: slices past the end
    // load zeros in both operands and add nothing.
    const int tend = sbeg + ((n + 1) / 2) * 2;
    for (int t = sbeg; t < tend; t += 2) {
      FAL_WAITCNT(0, 0);
      bar();
      __builtin_amdgcn_sched_barrier(0);
      issue(st0, t + 2);
      read(st1, 1);
      mma(0);
      interleave();
      __builtin_amdgcn_sched_barrier(0);
      FAL_WAITCNT(0, 0);
      bar();
      __builtin_amdgcn_sched_barrier(0);
      issue(st1, t + 3);
      read(st0, 0);
      mma(1);
      interleave();
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // every load (including those past the end) has landed and every
  // wavefront is done with the stages before they are reused for staging
  FAL_WAITCNT(0, 0);
  bar();

  float* stage = reinterpret_cast<float*>(wm ? st1 : st0) + wn * 16 * (WTN + 4);
  static_assert(2 * 16 * (WTN + 4) * 4 <= SBYTES, "epilogue staging exceeds a stage");
  const int mw = m0 + wm * WTM, nw = n0 + wn * WTN;
  if (P.splits > 1) {
    GemmProblem Q = P;
    Q.out = P.part + (int64_t)split * P.M * P.N;
    Q.ldo = P.N;
    Q.bias = Q.bias2 = nullptr;
    Q.vec_out = (P.N & 3) == 0;
    store_staged<EPI_STORE, 1, FM, FN>(Q, acc, stage, mw, nw, lane, gelu_tanh);
    return;
  }
  switch (P.epi) {
    case EPI_STORE:
      if (P.out_f32) store_staged<EPI_STORE, 1, FM, FN>(P, acc, stage, mw, nw, lane, gelu_tanh);
      else store_staged<EPI_STORE, 0, FM, FN>(P, acc, stage, mw, nw, lane, gelu_tanh);
      break;
    case EPI_GELU: store_staged<EPI_GELU, 0, FM, FN>(P, acc, stage, mw, nw, lane, gelu_tanh); break;
    case EPI_RESID: store_staged<EPI_RESID, 1, FM, FN>(P, acc, stage, mw, nw, lane, gelu_tanh); break;
    case EPI_MUL_AUX: store_staged<EPI_MUL_AUX, 0, FM, FN>(P, acc, stage, mw, nw, lane, gelu_tanh); break;
  }
}

// out[m, n] = sum_s part[s, m, n] (+ bias), s in order.
__global__ __launch_bounds__(256) void splitk_reduce(const float* part, int splits, int M, int N, const bf16* bias,
                                                     const bf16* bias2, float* out, int64_t ldo) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)M * N) return;
  const int m = i / N, n = i % N;
  const int64_t MN = (int64_t)M * N;
  float v = 0.f;
  for (int s = 0; s < splits; ++s) v += part[s * MN + i];
  if (bias) v += to_f(bias[n]);
  if (bias2) v += to_f(bias2[n]);
  out[(int64_t)m * ldo + n] = v;
}

// The same four columns at a time (N and ldo multiples of 4, out 16-byte
// aligned): one 16-byte load per slice, the slices summed in order.
__global__ __launch_bounds__(256) void splitk_reduce4(const float* part, int splits, int M, int N, const bf16* bias,
                                                      const bf16* bias2, float* out, int64_t ldo) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i >= (int64_t)M * N) return;
  const int m = i / N, n = i % N;
  const int64_t MN = (int64_t)M * N;
  float4 v = *reinterpret_cast<const float4*>(part + i);
#pragma unroll 4
  for (int s = 1; s < splits; ++s) {
    const float4 p = *reinterpret_cast<const float4*>(part + s * MN + i);
    v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
  }
  if (bias) { v.x += to_f(bias[n]); v.y += to_f(bias[n + 1]); v.z += to_f(bias[n + 2]); v.w += to_f(bias[n + 3]); }
  if (bias2) { v.x += to_f(bias2[n]); v.y += to_f(bias2[n + 1]); v.z += to_f(bias2[n + 2]); v.w += to_f(bias2[n + 3]); }
  *reinterpret_cast<float4*>(out + (int64_t)m * ldo + n) = v;
}

constexpr int kCUs = 256;
constexpr int kMaxSplits = 16;

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

// Pipelined kernel shapes (gemm_bf16_pipe): four wavefronts of (BM/2) x
// (BN/2); per_cu resident workgroups per CU (LDS: 4 stages of (BM + BN) x
// 64 bytes).  Launch time model, fitted to measurements on MI355X
// (GPT-2-sized problems, 8192^3): a k-slice of one tile costs t1 us when
// the tile has its CU alone and t2 us when per_cu tiles share it; each
// round of tiles adds ovh us (prologue, epilogue, launch ramp).  The
// 128 x 128 t1 comes from a lone round of weight-gradient tiles at the 1.3B
// shape (2048 x 2048 x 8192: 0.39 us per slice; with 0.30 the model kept
// that GEMM unsplit, 99.9 us, against 70.4 us split in two).
struct PipeShape { int bm, bn, per_cu; double t1, t2, ovh; };
enum { PIPE_256x256 = 0, PIPE_256x128 = 1, PIPE_128x256 = 2, PIPE_128x128 = 3, kPipeShapes = 4 };
constexpr PipeShape kPipe[kPipeShapes] = {{256, 256, 1, 0.85, 0.85, 10.0},
                                          {256, 128, 1, 0.56, 0.56, 5.0},
                                          {128, 256, 1, 0.56, 0.56, 5.0},
                                          {128, 128, 2, 0.39, 0.54, 3.0}};
constexpr int kPipeKS = 32;
constexpr double kHbmBytesPerUs = 5.0e6;       // sustained HBM rate for operand re-reads
constexpr double kPartialBytesPerUs = 8.0e6;   // split-K partials (written and re-read while cached)
constexpr double kLaunchUs = 5.0;              // the split-K reduce launch
constexpr double kCachedBytes = 128.0 * (1 << 20);  // operands below this are fetched from HBM once

static int64_t count_tiles_shape(const GemmGroup& g, int bm, int bn) {
  int64_t t = 0;
  for (int i = 0; i < g.n; ++i) t += (int64_t)((g.p[i].M + bm - 1) / bm) * ((g.p[i].N + bn - 1) / bn);
  return t;
}

// Estimated time (us) of the launch on shape c with K split sp ways.
static double pipe_estimate(const GemmGroup& g, int c, int sp) {
  const PipeShape& t = kPipe[c];
  const int64_t tiles = count_tiles_shape(g, t.bm, t.bn) * sp;
  int slices = 0;
  double reread = 0.0;
  for (int i = 0; i < g.n; ++i) {
    const GemmProblem& P = g.p[i];
    const int ns = (P.K + kPipeKS - 1) / kPipeKS + (P.K2 + kPipeKS - 1) / kPipeKS;
    slices = std::max(slices, (ns + sp - 1) / sp);
    const double a_bytes = 2.0 * P.M * (P.K + P.K2), b_bytes = 2.0 * P.N * (P.K + P.K2);
    if (a_bytes > kCachedBytes) reread += a_bytes * ((P.N + t.bn - 1) / t.bn - 1);
    if (b_bytes > kCachedBytes) reread += b_bytes * ((P.M + t.bm - 1) / t.bm - 1);
  }
  const int64_t slots = (int64_t)t.per_cu * kCUs;
  const int64_t full = tiles / slots, rem = tiles % slots;
  double us = (double)full * (t.ovh + slices * t.t2);
  if (rem > 0) us += t.ovh + slices * (rem > kCUs ? t.t2 : t.t1);
  us += reread / kHbmBytesPerUs;
  if (sp > 1) us += (2.0 * sp + 1.0) * 4.0 * g.p[0].M * g.p[0].N / kPartialBytesPerUs + kLaunchUs;
  return us;
}

// Shape (and split count for a splittable single problem) with the smallest
// estimated time.
static void choose_pipe(const GemmGroup& g, bool splittable, int64_t scratch_floats, int& shape, int& splits) {
  double best = 0.0;
  shape = PIPE_256x256;
  splits = 1;
  const int ns = (g.p[0].K + kPipeKS - 1) / kPipeKS;
  for (int c = 0; c < kPipeShapes; ++c) {
    const int maxsp = splittable ? kMaxSplits : 1;
    for (int sp = 1; sp <= maxsp; ++sp) {
      if (sp > 1 && (ns / sp < 8 || (int64_t)sp * g.p[0].M * g.p[0].N > scratch_floats)) break;
      const double us = pipe_estimate(g, c, sp);
      if ((c == 0 && sp == 1) || us < best) { best = us; shape = c; splits = sp; }
    }
  }
}

// The pipelined kernel reads whole 8-element chunks along K from
// k-contiguous operands (K a multiple of 8, or zero-padded storage with an
// MN-major partner) and addresses operands with 32-bit offsets.
static bool pipe_ok(const GemmGroup& g, int a_kmaj, int b_kmaj) {
  auto ext_ok = [](int64_t rows, int64_t ld, int64_t K, int kmaj) {
    const int64_t bytes = kmaj ? rows * ld * 2 : (K + 2 * kPipeKS * 4) * ld * 2;
    return bytes < ((int64_t)1 << 31) - (int64_t)(1 << 20);
  };
  for (int i = 0; i < g.n; ++i) {
    const GemmProblem& P = g.p[i];
    if ((a_kmaj || b_kmaj) && (P.K % 8 || P.K2 % 8)) {
      if (!P.kpad || (a_kmaj && b_kmaj) || P.K2 > 0) return false;
      const int64_t lda = a_kmaj ? P.lda : P.ldb;  // the k-contiguous operand's row pitch
      if (lda < (P.K + 7) / 8 * 8) return false;
    }
    if (!ext_ok(P.M, P.lda, P.K, a_kmaj) || !ext_ok(P.N, P.ldb, P.K, b_kmaj)) return false;
    if (P.K2 > 0 && (!ext_ok(P.M, P.lda2, P.K2, a_kmaj) || !ext_ok(P.N, P.ldb2, P.K2, b_kmaj))) return false;
  }
  return true;
}

double gemm_last_round_fill(DType dt, int a_kmaj, int b_kmaj, const GemmGroup& g, int64_t splitk_floats) {
  if (dt != BF16 || g.n < 1 || g.n > kMaxGroup || !pipe_ok(g, a_kmaj, b_kmaj)) return 1.0;
  const GemmProblem& P0 = g.p[0];
  const bool splittable = splitk_floats > 0 && g.n == 1 && P0.K2 == 0 && P0.epi == EPI_STORE && P0.out_f32;
  int shape, sp;
  choose_pipe(g, splittable, splitk_floats, shape, sp);
  const PipeShape& t = kPipe[shape];
  int kmax = 0;
  for (int i = 0; i < g.n; ++i) kmax = std::max(kmax, g.p[i].K + g.p[i].K2);
  const bool occ3 = shape == PIPE_128x128 && a_kmaj && !b_kmaj && sp == 1 && kmax <= FAL_OCC3_KMAX;
  const int64_t slots = (int64_t)(occ3 ? 3 : t.per_cu) * kCUs;
  const int64_t tiles = count_tiles_shape(g, t.bm, t.bn) * sp;
  const int64_t rem = tiles % slots;
  return rem == 0 ? 1.0 : (double)rem / (double)slots;
}

hipError_t gemm(DType dt, int a_kmaj, int b_kmaj, GemmGroup& g, int gelu_tanh, hipStream_t s,
                const char** why, float* splitk_scratch, int64_t splitk_floats) {
  *why = nullptr;
  if (g.n < 1 || g.n > kMaxGroup) { *why = "bad GEMM group size"; return hipErrorInvalidValue; }
  const GemmProblem& P0 = g.p[0];
  const bool splittable = dt == BF16 && splitk_scratch && g.n == 1 && P0.K2 == 0 && P0.epi == EPI_STORE &&
                          P0.out_f32;
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
    P.splits = 1;
    P.part = nullptr;
    {
      // The epilogue moves 4 consecutive columns at a time (8 bytes of bf16,
      // 16 of fp32): every row it touches, and the bias, must be aligned to that.
      auto al = [](const void* p, int bytes) { return (reinterpret_cast<uintptr_t>(p) & (bytes - 1)) == 0; };
      const int el = (P.epi == EPI_RESID || (P.epi == EPI_STORE && P.out_f32)) ? 4 : 2;
      bool ok = P.out && al(P.out, 4 * el) && P.ldo % 4 == 0;
      if (P.bias) ok = ok && al(P.bias, 8);
      if (P.bias2) ok = ok && al(P.bias2, 8);
      if (P.epi == EPI_RESID) ok = ok && al(P.resid, 16) && P.ldr % 4 == 0;
      if (P.epi == EPI_GELU && P.out2) ok = ok && al(P.out2, 8) && P.ldo2 % 4 == 0;
      if (P.epi == EPI_MUL_AUX) ok = ok && P.aux && al(P.aux, 8) && P.ldaux % 4 == 0;
      P.vec_out = ok ? 1 : 0;
    }
  }
  auto set_tiles = [&](int tm, int tn) {
    int total = 0;
    for (int i = 0; i < g.n; ++i) {
      GemmProblem& P = g.p[i];
      P.tiles_m = (P.M + tm - 1) / tm;
      P.tiles_n = (P.N + tn - 1) / tn;
      P.tile_start = total;
      total += P.tiles_m * P.tiles_n;
    }
    return total;
  };
  auto launch_reduce = [&]() -> hipError_t {
    const GemmProblem& P = g.p[0];
    if (g.n == 1 && P.splits > 1) {
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      const bool v4 = P.N % 4 == 0 && P.ldo % 4 == 0 && reinterpret_cast<uintptr_t>(P.out) % 16 == 0;
      if (v4)
        hipLaunchKernelGGL(splitk_reduce4, dim3(cdiv((int64_t)P.M * P.N / 4, 256)), dim3(256), 0, s, P.part,
                           P.splits, P.M, P.N, static_cast<const bf16*>(P.bias), static_cast<const bf16*>(P.bias2),
                           static_cast<float*>(P.out), P.ldo);
      else
        hipLaunchKernelGGL(splitk_reduce, dim3(cdiv((int64_t)P.M * P.N, 256)), dim3(256), 0, s, P.part, P.splits,
                           P.M, P.N, static_cast<const bf16*>(P.bias), static_cast<const bf16*>(P.bias2),
                           static_cast<float*>(P.out), P.ldo);
    }
    return hipGetLastError();
  };

  if (dt == BF16 && pipe_ok(g, a_kmaj, b_kmaj)) {
    int shape, sp;
    choose_pipe(g, splittable, splitk_floats, shape, sp);
    int total = set_tiles(kPipe[shape].bm, kPipe[shape].bn);
    if (sp > 1) {
      g.p[0].splits = sp;
      g.p[0].part = splitk_scratch;
      total *= sp;
    }
    g.total_tiles = total;
    const dim3 grid(total), block(256);
#define FAL_PIPE_LAUNCH(BM, BN, OCC, NS)                                                                           \
  if (a_kmaj && b_kmaj) hipLaunchKernelGGL((gemm_bf16_pipe<1, 1, BM, BN, OCC, NS>), grid, block, 0, s, g, gelu_tanh); \
  else if (a_kmaj) hipLaunchKernelGGL((gemm_bf16_pipe<1, 0, BM, BN, OCC, NS>), grid, block, 0, s, g, gelu_tanh);      \
  else if (b_kmaj) hipLaunchKernelGGL((gemm_bf16_pipe<0, 1, BM, BN, OCC, NS>), grid, block, 0, s, g, gelu_tanh);      \
  else hipLaunchKernelGGL((gemm_bf16_pipe<0, 0, BM, BN, OCC, NS>), grid, block, 0, s, g, gelu_tanh);
    // Four LDS stages (a three-slice load lead).  Deeper rings (five stages
    // at 128 x 128, six at 256 x 128) measured no faster with operands
    // coming from HBM and slightly slower with them in cache.
#define FAL_DBL_LAUNCH(BM, BN, OCC)                                                                           \
  if (a_kmaj && b_kmaj) hipLaunchKernelGGL((gemm_bf16_dbl<1, 1, BM, BN, OCC>), grid, block, 0, s, g, gelu_tanh); \
  else if (a_kmaj) hipLaunchKernelGGL((gemm_bf16_dbl<1, 0, BM, BN, OCC>), grid, block, 0, s, g, gelu_tanh);      \
  else if (b_kmaj) hipLaunchKernelGGL((gemm_bf16_dbl<0, 1, BM, BN, OCC>), grid, block, 0, s, g, gelu_tanh);      \
  else hipLaunchKernelGGL((gemm_bf16_dbl<0, 0, BM, BN, OCC>), grid, block, 0, s, g, gelu_tanh);
    // 128 x 128 tiles of a k-contiguous A and an n-contiguous B with a short
    // K (the forward projections): three workgroups per CU on three 32-deep
    // LDS stages hide more latency than two on the 64-deep double buffer
    // (measured 8-14% faster for the QKV and FFN-up shapes); the other
    // orientations and long K keep the double buffer.
    int kmax = 0;
    for (int i = 0; i < g.n; ++i) kmax = std::max(kmax, g.p[i].K + g.p[i].K2);
    const bool occ3 = shape == PIPE_128x128 && a_kmaj && !b_kmaj && sp == 1 && kmax <= FAL_OCC3_KMAX;
    if (occ3) {
      hipLaunchKernelGGL((gemm_bf16_pipe<1, 0, 128, 128, 3, 3>), grid, block, 0, s, g, gelu_tanh);
    } else if (FAL_GEMM_DBL && shape != PIPE_256x256) {
      switch (shape) {
        case PIPE_256x128: FAL_DBL_LAUNCH(256, 128, 1) break;
        case PIPE_128x256: FAL_DBL_LAUNCH(128, 256, 1) break;
        default: FAL_DBL_LAUNCH(128, 128, 2) break;
      }
    } else {
      switch (shape) {
        case PIPE_256x256:
          // stage count per orientation: the ones with which the register
          // allocator keeps every accumulator in place across the unrolled
          // main loop (no accumulator copies between iterations)
          if (a_kmaj && b_kmaj) hipLaunchKernelGGL((gemm_bf16_pipe<1, 1, 256, 256, 1, FAL_NS11>), grid, block, 0, s, g, gelu_tanh);
          else if (a_kmaj) hipLaunchKernelGGL((gemm_bf16_pipe<1, 0, 256, 256, 1, FAL_NS10>), grid, block, 0, s, g, gelu_tanh);
          else if (b_kmaj) hipLaunchKernelGGL((gemm_bf16_pipe<0, 1, 256, 256, 1, FAL_NS01>), grid, block, 0, s, g, gelu_tanh);
          else hipLaunchKernelGGL((gemm_bf16_pipe<0, 0, 256, 256, 1, FAL_NS00>), grid, block, 0, s, g, gelu_tanh);
          break;
        case PIPE_256x128: FAL_PIPE_LAUNCH(256, 128, 1, 4) break;
        case PIPE_128x256: FAL_PIPE_LAUNCH(128, 256, 1, 4) break;
        default: FAL_PIPE_LAUNCH(128, 128, 2, 4) break;
      }
    }
#undef FAL_DBL_LAUNCH
#undef FAL_PIPE_LAUNCH
    return launch_reduce();
  }

  if (dt == BF16) {
    // the config check keeps every operand inside the kernels' 32-bit range
    // and every k-contiguous K a multiple of 8 (or zero-padded)
    *why = "bf16 GEMM operand outside the pipelined kernels' range (>= 2 GiB, or K not a multiple of 8 without "
           "zero padding)";
    return hipErrorInvalidValue;
  }
  const int total = set_tiles(ST, ST);
  g.total_tiles = total;
  const dim3 grid(total), block(256);
  if (a_kmaj && b_kmaj) hipLaunchKernelGGL((gemm_simt<float, 1, 1>), grid, block, 0, s, g, gelu_tanh);
  else if (a_kmaj) hipLaunchKernelGGL((gemm_simt<float, 1, 0>), grid, block, 0, s, g, gelu_tanh);
  else if (b_kmaj) hipLaunchKernelGGL((gemm_simt<float, 0, 1>), grid, block, 0, s, g, gelu_tanh);
  else hipLaunchKernelGGL((gemm_simt<float, 0, 0>), grid, block, 0, s, g, gelu_tanh);
  return hipGetLastError();
}

}  // namespace fal
