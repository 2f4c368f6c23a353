// Dense GEMMs of the training step: the four linear layers of a block
// (QKV, output projection, FFN up, FFN down; Sec. 2), their data- and
// weight-gradient products, and the tied LM head.
//
// Two kernels share one problem descriptor (kernels.h):
//  * gemm_bf16_mfma: bf16 operands, fp32 accumulation on the gfx950 matrix
//    cores (v_mfma_f32_16x16x32_bf16).  128x128 output tile per 256-thread
//    workgroup (2x2 wavefronts of 64x64) or 256x256 per 512-thread
//    workgroup (4x2 wavefronts of 64x128), K staged through LDS 64 at a time
//    in k-contiguous rows.  Operands whose contraction dimension is strided
//    (the weight of a forward layer, both operands of a weight gradient) are
//    transposed in registers on their way into LDS.  The epilogue (bias,
//    GELU, residual add, GELU derivative) runs on row segments staged
//    through LDS so every global access is a whole wavefront-tile row.
//  * gemm_simt: fp32 FMA kernel (fp32 parity mode).
// Both launch every problem of a group in one grid, so the independent
// GEMMs of FAL's two branches can share a launch.
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
      static_cast<S*>(P.out2)[(int64_t)m * P.ldo2 + n] = from_f<S>(dg);
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

#ifndef FAL_LDS_SWZ
#define FAL_LDS_SWZ 2
#endif
#ifndef FAL_LDS_PAD
#define FAL_LDS_PAD 8
#endif
constexpr int KT = 64;
// LDS operand tiles are k-contiguous rows of KT elements.  Either padded
// rows (FAL_LDS_SWZ 0) or unpadded rows whose 16-byte chunks are permuted
// by an XOR of the row index (FAL_LDS_SWZ 1: row & 7, 2: (row >> 1) & 7).
constexpr int LDK = FAL_LDS_SWZ ? KT : KT + FAL_LDS_PAD;
__device__ __forceinline__ int lds_off(int row, int k) {
  if (FAL_LDS_SWZ == 0) return row * LDK + k;
  const int f = FAL_LDS_SWZ == 1 ? (row & 7) : ((row >> 1) & 7);
  return row * LDK + ((((k >> 3) ^ f)) << 3) + (k & 7);
}

// Operand staging through buffer loads.  Each thread's chunk offsets (32-bit,
// bytes from the tile's first row or column) are computed once per K
// segment; the k-tile advance goes into the scalar offset, so the steady
// state issues loads with no per-load address arithmetic.  Rows past the
// matrix are clamped to an in-bounds row when the offsets are built and
// zeroed when written to LDS (edge tiles only); k past the segment is
// checked only in the tail tile.  The resource's range is the operand's
// extent, so even a clamped offset cannot leave the buffer.
constexpr int kRsrcWord3 = 0x00020000;  // gfx9-family buffer descriptor word 3

// An operand whose contraction dimension is strided (MN-major: the weight of
// a forward layer, both operands of a weight gradient) is staged as loaded,
// [k][row], and read back with the gfx950 LDS transpose load.
// ds_read_b64_tr_b16 gives lane i of each 16-lane group element i % 4 of the
// 8-byte chunks addressed by lanes 4j + i / 4 (j = 0..3); lane L therefore
// addresses k-row kb + L / 4, rows 4 (L % 4)..+3 of the fragment, and two
// reads (kb, kb + 4) return the eight consecutive k a 16x16x32 operand lane
// holds.  One such read spans the k-rows {kb + 8G + j} (G, j = 0..3).  Rows
// are padded by 16 elements (the k-rows then start 32 bytes apart modulo
// 256) and stored in the order sigma(k) = k ^ (((k >> 3) & 1) << 2): the 16
// k-rows of a read then hit every 32-byte bank group exactly twice, the
// minimum for 512 bytes, while each fragment's offset stays an immediate.
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

__device__ __forceinline__ i16x4_t lds_read_tr(const bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_i16x4_t*)((__attribute__((address_space(3))) char*)(const_cast<bf16*>(p))));
}

template <int R, int KMAJ, int NTH>
struct BStage {
  static constexpr int CPR = R / 8;                         // 16-byte chunks per MN-major k-row
  static constexpr int TP = R + 16;                         // MN-major LDS row pitch (elements)
  static constexpr int ELEMS = KMAJ ? R * KT : KT * TP;     // one LDS stage
  __device__ __forceinline__ static int mn_row(int k) { return k ^ (((k >> 3) & 1) << 2); }
  __device__ __forceinline__ static int mn_off(int k, int r) { return mn_row(k) * TP + r; }
  static constexpr int NC = R * KT / 8 / NTH;               // 16-byte chunks per thread
  static_assert(NC > 0 && NC <= 32, "tile / thread count mismatch");
  uint4 v[NC];
  uint32_t voff[NC];
  uint32_t rowbad;
  int kpart[NC];
  uint64_t base;   // byte address of the tile's first row / column
  int nbytes;      // extent of the operand from base
  uint32_t kstep;

  // chunk i of this thread: k-contiguous rows (row, k) or MN-major (k, row)
  __device__ __forceinline__ static void chunk(int i, int tid, int& row, int& k) {
    const int c = tid + NTH * i;
    if (KMAJ) { row = c >> 3; k = (c & 7) * 8; }
    else { k = c / CPR; row = (c % CPR) * 8; }
  }

  __device__ __forceinline__ void init(const bf16* X, int64_t ld, int r0, int Rmax, int Kseg, int tid) {
    base = reinterpret_cast<uint64_t>(KMAJ ? X + (int64_t)r0 * ld : X + r0);
    const int64_t ext = KMAJ ? (int64_t)(Rmax - r0) * ld * 2 : ((int64_t)Kseg * ld - r0) * 2;
    nbytes = (int)min<int64_t>(ext, 0x7fffffff);
    rowbad = 0;
    kstep = KMAJ ? 2 : (uint32_t)(ld * 2);
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      int row, k;
      chunk(i, tid, row, k);
      if (KMAJ) {
        int rr = row;
        if (r0 + row >= Rmax) { rowbad |= 1u << i; rr = Rmax - 1 - r0; }
        voff[i] = (uint32_t)(((int64_t)rr * ld + k) * 2);
      } else {
        // 8 consecutive rows per chunk; a chunk starting past the matrix is
        // clamped (and zeroed in LDS).  Rows past the matrix inside a valid
        // chunk only reach outputs that are never stored.
        int cc = row;
        if (r0 + row >= Rmax) { rowbad |= 1u << i; cc = ((Rmax - r0 - 1) / 8) * 8; }
        voff[i] = (uint32_t)(((int64_t)k * ld + cc) * 2);
      }
    }
  }

  // The descriptor is wave-uniform: rebuild it from readfirstlane'd scalars at
  // the load so it lives in scalar registers (no waterfall loops).
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc() const {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)base);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(base >> 32));
    const int n = __builtin_amdgcn_readfirstlane(nbytes);
    return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(((uint64_t)hi << 32) | lo), (short)0, n,
                                             kRsrcWord3);
  }
  __device__ __forceinline__ uint4 ld16(__amdgpu_buffer_rsrc_t rs, uint32_t off, uint32_t soff) const {
    typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
    const u32x4v r = __builtin_amdgcn_raw_buffer_load_b128(rs, off, soff, 0);
    return make_uint4(r[0], r[1], r[2], r[3]);
  }

  __device__ __forceinline__ uint32_t soff(int k0) const {
    return __builtin_amdgcn_readfirstlane((uint32_t)k0 * kstep);
  }
  // Full tile at k0 (relative to the segment).
  __device__ __forceinline__ void load_full(__amdgpu_buffer_rsrc_t rs, uint32_t so) {
#pragma unroll
    for (int i = 0; i < NC; ++i) v[i] = ld16(rs, voff[i], so);
  }
  // Tail tile: chunks past K are not read.
  __device__ __forceinline__ void load_tail(__amdgpu_buffer_rsrc_t rs, uint32_t so, int k0, int K, int tid) {
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      int row, k;
      chunk(i, tid, row, k);
      const int kk = k0 + k;
      kpart[i] = KMAJ ? max(0, min(8, K - kk)) : (kk < K ? 8 : 0);
      v[i] = kpart[i] > 0 ? ld16(rs, voff[i], so) : make_uint4(0, 0, 0, 0);
    }
  }

  __device__ __forceinline__ uint4 masked(int i, bool tail) const {
    uint4 w = v[i];
    if (rowbad & (1u << i)) return make_uint4(0, 0, 0, 0);
    if (tail && kpart[i] < 8) {
      uint16_t* e = reinterpret_cast<uint16_t*>(&w);
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (q >= kpart[i]) e[q] = 0;
    }
    return w;
  }

  // check: edge tile or tail tile (uniform); otherwise stores go straight in.
  __device__ __forceinline__ void store(bf16* s, int tid, bool check, bool tail) const {
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      int row, k;
      chunk(i, tid, row, k);
      const int off = KMAJ ? lds_off(row, k) : mn_off(k, row);
      *reinterpret_cast<uint4*>(s + off) = check ? masked(i, tail) : v[i];
    }
  }

  // Operand fragment of a 16x16x32 MFMA: rows row0 + lane % 16, k
  // 32 ks + 8 (lane / 16) .. +7.
  __device__ __forceinline__ static bf16x8_t frag(const bf16* s, int row0, int ks, int lane) {
    if (KMAJ)
      return *reinterpret_cast<const bf16x8_t*>(s + lds_off(row0 + (lane & 15), ks * 32 + (lane >> 4) * 8));
    const int L = lane & 15;
    const int k = ks * 32 + (lane >> 4) * 8 + (L >> 2);
    const bf16* p = s + row0 + 4 * (L & 3);
    const i16x4_t lo = lds_read_tr(p + mn_row(k) * TP), hi = lds_read_tr(p + mn_row(k + 4) * TP);
    const i16x4_t v8[2] = {lo, hi};
    return *reinterpret_cast<const bf16x8_t*>(v8);
  }
};

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
      st4(static_cast<bf16*>(P.out2) + (int64_t)m * P.ldo2 + n, dg);
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
        static_cast<bf16*>(P.out2)[(int64_t)m * P.ldo2 + n + c] = from_f<bf16>(dg);
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
// with consecutive lanes on consecutive columns, so every
// global access (output, residual, pre-activation) covers whole row segments
// of the wavefront tile (128 B of bf16 for a 64-column tile).
template <int EPI, int F32OUT, int FM, int FN>
__device__ __forceinline__ void store_staged(const GemmProblem& P, const f32x4_t (&acc)[FM][FN], float* stage,
                                             int mw, int nw, int lane, int gelu_tanh) {
  constexpr int WTN = FN * 16, PITCH = WTN + 4;
  constexpr int LPR = WTN / 4, RPI = 64 / LPR;    // lanes per row, rows per access
  constexpr int NPASS = (16 + RPI - 1) / RPI;     // accesses per 16-row strip
  const int rr = lane / LPR, cc = (lane % LPR) * 4;  // read-back position (rr >= RPI: idle)
  const int n = nw + cc;
  const bool full = P.vec_out && n + 4 <= P.N;
  float bn[4];
  bias4(P, n, full, bn);
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    // straight from the MFMA layout: lane 16g+c holds rows 4g..4g+3 of
    // column c (with the 4-float pad, 64 different banks per store)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) stage[((lane >> 4) * 4 + r) * PITCH + 16 * j + (lane & 15)] = acc[i][j][r];
    wave_lds_order();
    // kept rolled: unrolling it multiplies the epilogue code (one copy per
    // output kind) several-fold, and the once-per-tile epilogue then runs
    // out of the instruction cache
#pragma unroll 1
    for (int k = 0; k < NPASS; ++k) {
      const int r = k * RPI + rr;
      if (rr >= RPI || r >= 16) continue;
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



#ifndef FAL_GEMM_REMAP
#define FAL_GEMM_REMAP 1
#endif
#ifndef FAL_GEMM_GROUP_M
#define FAL_GEMM_GROUP_M 8
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

// BM x BN output tile per workgroup of WGM x WGN wavefronts, each owning a
// (BM/WGM) x (BN/WGN) block; K staged through two LDS buffers 64 at a time.
template <int AK, int BKM, int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_bf16_mfma(GemmGroup g, int gelu_tanh) {
  constexpr int NTH = 64 * WGM * WGN;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;  // wavefront tile
  constexpr int FM = WTM / 16, FN = WTN / 16;    // 16x16 fragments per wavefront
  typedef BStage<BM, AK, NTH> StA;
  typedef BStage<BN, BKM, NTH> StB;
  // one LDS block: two stages of A, two of B; reused for the epilogue
  __shared__ __attribute__((aligned(16))) bf16 smem[2 * (StA::ELEMS + StB::ELEMS)];
  auto sA = [&](int st) { return smem + st * StA::ELEMS; };
  auto sB = [&](int st) { return smem + 2 * StA::ELEMS + st * StB::ELEMS; };
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
#if FAL_GEMM_REMAP
  grouped_tile(local, P.tiles_m, P.tiles_n, tmi, tni);
#else
  tmi = local / P.tiles_n;
  tni = local % P.tiles_n;
#endif
  const int m0 = tmi * BM, n0 = tni * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nt1 = (P.K + KT - 1) / KT;
  int nt = nt1 + (P.K2 > 0 ? (P.K2 + KT - 1) / KT : 0);
  int tbeg = 0;
  if (P.splits > 1) {  // single K segment: this slice covers k-tiles [tbeg, tbeg + nt)
    const int per = (nt1 + P.splits - 1) / P.splits;
    tbeg = split * per;
    nt = max(0, min(nt1, tbeg + per) - tbeg);
  }
  auto compute = [&](const bf16* a_s, const bf16* b_s) {
#pragma unroll
    for (int ks = 0; ks < KT / 32; ++ks) {
      bf16x8_t a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) a[i] = StA::frag(a_s, wm * WTM + i * 16, ks, lane);
#pragma unroll
      for (int j = 0; j < FN; ++j) b[j] = StB::frag(b_s, wn * WTN + j * 16, ks, lane);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };
  const bool edge = (m0 + BM > P.M) || (n0 + BN > P.N);
  StA sa;
  StB sb;
  int fk = 0, fK = P.K;
  auto seg_init = [&](int seg, int k0) {
    fK = seg ? P.K2 : P.K;
    fk = k0;
    sa.init(static_cast<const bf16*>(seg ? P.A2 : P.A), seg ? P.lda2 : P.lda, m0, P.M, fK, tid);
    sb.init(static_cast<const bf16*>(seg ? P.B2 : P.B), seg ? P.ldb2 : P.ldb, n0, P.N, fK, tid);
  };
  // Issues every load of the next tile of both operands (one branch, so no
  // wait is forced between them); returns whether it is a tail tile.
  auto fetch_next = [&]() {
    if (fk >= fK) seg_init(1, 0);
    const bool tail = fk + KT > fK;
    const __amdgpu_buffer_rsrc_t ra = sa.rsrc(), rb = sb.rsrc();
    const uint32_t oa = sa.soff(fk), ob = sb.soff(fk);
    if (!tail) {
      sa.load_full(ra, oa);
      sb.load_full(rb, ob);
    } else {
      sa.load_tail(ra, oa, fk, fK, tid);
      sb.load_tail(rb, ob, fk, fK, tid);
    }
    fk += KT;
    return tail;
  };
  bool tail_next = false;
  if (nt > 0) {
    seg_init(tbeg >= nt1 ? 1 : 0, (tbeg >= nt1 ? tbeg - nt1 : tbeg) * KT);
    const bool tail = fetch_next();
    sa.store(sA(0), tid, edge || tail, tail);
    sb.store(sB(0), tid, edge || tail, tail);
  }
  __syncthreads();
  for (int t = 0; t < nt; ++t) {
    const int cur = t & 1;
    if (t + 1 < nt) tail_next = fetch_next();
    compute(sA(cur), sB(cur));
    if (t + 1 < nt) {
      sa.store(sA(cur ^ 1), tid, edge || tail_next, tail_next);
      sb.store(sB(cur ^ 1), tid, edge || tail_next, tail_next);
    }
    __syncthreads();
  }

  // acc[i][j][r] holds C[row 4*(lane/16) + r][col lane%16] of 16x16 tile (i, j).
  // The main loop ended with a barrier, so the LDS tiles are free: each
  // wavefront stages its strips in a private slice.
  float* stage = reinterpret_cast<float*>(smem) + wave * 16 * (WTN + 4);
  static_assert(WGM * WGN * 16 * (WTN + 4) * 4 <= (int)sizeof(smem), "epilogue staging exceeds LDS");
  const int mw = m0 + wm * WTM, nw = n0 + wn * WTN;
  if (P.splits > 1) {  // raw fp32 partial of this K slice, row pitch N
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

// ------------------------------------------------------------- launcher --
// Block shapes.  128x128 (2x2 wavefronts of 64x64) and 128x96 (2x2 of 64x48)
// run two workgroups per CU; 256x256 (4x2 wavefronts of 64x128) runs one and
// moves half the global traffic and a quarter less LDS traffic per MFMA.
// Their throughput per CU differs (rate, relative to 128x128) and so does
// how finely they quantise a launch into waves; the launcher picks the shape
// with the smallest estimated time.  The 128x96 shape fills the chip exactly
// for 768-wide outputs (8192 x 768 = 512 tiles).
constexpr int kCUs = 256;
struct TileShape { int bm, bn, per_cu; double rate; };
enum { TILE_SQ = 0, TILE_NARROW = 1, TILE_BIG = 2, kTileShapes = 3 };
constexpr TileShape kTile[kTileShapes] = {{128, 128, 2, 1.0}, {128, 96, 2, 0.92}, {256, 256, 1, 1.25}};

static int64_t count_tiles(const GemmGroup& g, int bm, int bn) {
  int64_t t = 0;
  for (int i = 0; i < g.n; ++i) t += (int64_t)((g.p[i].M + bm - 1) / bm) * ((g.p[i].N + bn - 1) / bn);
  return t;
}

static int choose_tile(const GemmGroup& g) {
  int best = TILE_SQ;
  double tbest = 0.0;
  for (int c = 0; c < kTileShapes; ++c) {
    const TileShape& t = kTile[c];
    const int64_t slots = (int64_t)t.per_cu * kCUs;
    const int64_t rounds = (count_tiles(g, t.bm, t.bn) + slots - 1) / slots;
    // time in units of one 128x128 tile on a whole CU
    const double time = (double)rounds * t.per_cu * (t.bm * t.bn) / (128.0 * 128.0) / t.rate;
    if (c == 0 || time < tbest) { tbest = time; best = c; }
  }
  return best;
}

constexpr int kSlots = 2 * kCUs;    // resident 128x128 workgroups
constexpr int kMaxSplits = 16;
// Partials' write and re-read per split, in k-tile rounds per 128 tiles
// (measured: 3 slices beat 7 for the 768 x 3072 x 8192 weight gradient).
constexpr double kSplitBeta = 3.0;

// Split-K factor for a launch of `tiles` 128x128 tiles over nt k-tiles:
// minimises (rounds of all workgroup slots) x (k-tiles per slice) plus the
// partials' extra write and read (kSplitBeta k-tile rounds per split for
// every 128 tiles).  1 = no split.
static int choose_splits(int tiles, int nt, int64_t MN, int64_t scratch_floats) {
  auto cost = [&](int sp) {
    const double rounds = (double)((tiles * sp + kSlots - 1) / kSlots);
    return rounds * ((nt + sp - 1) / sp) + (sp > 1 ? kSplitBeta * sp * tiles / 128.0 : 0.0);
  };
  int best = 1;
  double cbest = cost(1);
  for (int sp = 2; sp <= kMaxSplits && nt / sp >= 4 && (int64_t)sp * MN <= scratch_floats; ++sp) {
    const double c = cost(sp);
    if (c < cbest) { cbest = c; best = sp; }
  }
  return best;
}
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
                const char** why, float* splitk_scratch, int64_t splitk_floats) {
  *why = nullptr;
  if (g.n < 1 || g.n > kMaxGroup) { *why = "bad GEMM group size"; return hipErrorInvalidValue; }
  // Weight gradients (one fp32 plain output, few 128x128 tiles) split K on
  // 128x128 tiles; everything else picks its tile shape.
  const GemmProblem& P0 = g.p[0];
  const bool splittable = dt == BF16 && splitk_scratch && g.n == 1 && P0.K2 == 0 && P0.epi == EPI_STORE &&
                          P0.out_f32 && count_tiles(g, 128, 128) <= kCUs;
  const int shape = dt != BF16 ? TILE_SQ : splittable ? TILE_SQ : choose_tile(g);
  const int tm = dt == BF16 ? kTile[shape].bm : ST, tn = dt == BF16 ? kTile[shape].bn : ST;
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
      if (P.epi == EPI_GELU) ok = ok && P.out2 && al(P.out2, 8) && P.ldo2 % 4 == 0;
      if (P.epi == EPI_MUL_AUX) ok = ok && P.aux && al(P.aux, 8) && P.ldaux % 4 == 0;
      P.vec_out = ok ? 1 : 0;
    }
    total += P.tiles_m * P.tiles_n;
  }
  // Split K for launches that would leave compute units idle (fewer tiles
  // than CUs); fp32 plain outputs only (the weight gradients).
  if (splittable) {
    GemmProblem& P = g.p[0];
    const int tiles = P.tiles_m * P.tiles_n;
    const int sp = choose_splits(tiles, (P.K + KT - 1) / KT, (int64_t)P.M * P.N, splitk_floats);
    if (sp > 1) {
      P.splits = sp;
      P.part = splitk_scratch;
      total = tiles * sp;
    }
  }
  g.total_tiles = total;
  const dim3 grid(total), block(dt == BF16 && shape == TILE_BIG ? 512 : 256);
  if (dt == BF16) {
#define FAL_GEMM_LAUNCH(BM, BN, WGM, WGN)                                                                      \
  if (a_kmaj && b_kmaj) hipLaunchKernelGGL((gemm_bf16_mfma<1, 1, BM, BN, WGM, WGN>), grid, block, 0, s, g, gelu_tanh); \
  else if (a_kmaj) hipLaunchKernelGGL((gemm_bf16_mfma<1, 0, BM, BN, WGM, WGN>), grid, block, 0, s, g, gelu_tanh);      \
  else if (b_kmaj) hipLaunchKernelGGL((gemm_bf16_mfma<0, 1, BM, BN, WGM, WGN>), grid, block, 0, s, g, gelu_tanh);      \
  else hipLaunchKernelGGL((gemm_bf16_mfma<0, 0, BM, BN, WGM, WGN>), grid, block, 0, s, g, gelu_tanh);
    if (shape == TILE_BIG) {
      FAL_GEMM_LAUNCH(256, 256, 4, 2)
    } else if (shape == TILE_NARROW) {
      FAL_GEMM_LAUNCH(128, 96, 2, 2)
    } else {
      FAL_GEMM_LAUNCH(128, 128, 2, 2)
    }
#undef FAL_GEMM_LAUNCH
    const GemmProblem& P = g.p[0];
    if (g.n == 1 && P.splits > 1) {
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(splitk_reduce, dim3(cdiv((int64_t)P.M * P.N, 256)), dim3(256), 0, s, P.part, P.splits,
                         P.M, P.N, static_cast<const bf16*>(P.bias), static_cast<const bf16*>(P.bias2),
                         static_cast<float*>(P.out), P.ldo);
    }
  } else {
    if (a_kmaj && b_kmaj) hipLaunchKernelGGL((gemm_simt<float, 1, 1>), grid, block, 0, s, g, gelu_tanh);
    else if (a_kmaj) hipLaunchKernelGGL((gemm_simt<float, 1, 0>), grid, block, 0, s, g, gelu_tanh);
    else if (b_kmaj) hipLaunchKernelGGL((gemm_simt<float, 0, 1>), grid, block, 0, s, g, gelu_tanh);
    else hipLaunchKernelGGL((gemm_simt<float, 0, 0>), grid, block, 0, s, g, gelu_tanh);
  }
  return hipGetLastError();
}

}  // namespace fal
