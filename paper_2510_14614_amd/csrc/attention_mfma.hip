// Attention on the gfx950 matrix cores (bf16 in, fp32 accumulate), head_dim
// 64 or 128, with the causal mask (CAUSAL = true) or without it (the
// bidirectional encoder blocks: every query sees every key of its sequence).  Same mathematics as the SIMT kernels in
// attention.hip (blockwise, online softmax, deterministic backward), laid
// out for v_mfma_f32_32x32x16_bf16:
//
//  * A wavefront owns 32 rows of the "outer" sequence dimension (queries in
//    the forward and dQ kernels, keys in the dK/dV kernel); a workgroup of
//    four wavefronts owns 128.  The other dimension streams through LDS in
//    tiles of 64 rows.
//  * Forward computes S^T = K Q^T, so each lane holds 16 scores of one query
//    and the row max/sum need one cross-lane exchange (lane ^ 32).  The
//    accumulator registers of S^T are exactly the B operand of O^T = V^T P^T
//    (the contraction index order of A and B only has to agree), so P never
//    leaves registers.
//  * dK/dV kernel computes S = Q K^T and dP = dO V^T per key block; P^T and
//    dS^T feed dV += P^T dO and dK += dS^T Q straight from registers.
//  * dQ kernel computes S^T and dP^T per query block and accumulates
//    dQ^T += K^T dS^T.
//  * Every tile sits in LDS row-major, as loaded.  Operands that contract
//    over a tile's rows (V, dO, Q, K in the second products) are read with
//    the gfx950 LDS transpose load (ds_read_b64_tr_b16), so no transposed
//    copy is ever written.
// Accumulator layout of one 32x32 tile: lane l, register r holds
// C[8*(r/4) + 4*(l/32) + r%4][l%32].
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace fal {

typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4v __attribute__((ext_vector_type(4)));
typedef float f32x16v __attribute__((ext_vector_type(16)));

constexpr int AT = 64;        // rows per LDS tile of the streamed dimension
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ f32x16v mfma32(bf16x8v a, bf16x8v b, f32x16v c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16v zero16() {
  f32x16v z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// 8 bf16 made of two runs of 4 (each 8 bytes, 8-byte aligned)
__device__ __forceinline__ bf16x8v ld_2x4(const bf16* p0, const bf16* p1) {
  const bf16x4v a = *reinterpret_cast<const bf16x4v*>(p0);
  const bf16x4v b = *reinterpret_cast<const bf16x4v*>(p1);
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

__device__ __forceinline__ bf16x8v pack8(const f32x16v& v, int base) {
  bf16x8v o;
#pragma unroll
  for (int j = 0; j < 8; ++j) o[j] = static_cast<bf16>(v[base + j]);
  return o;
}

// Row r of the 32x32 accumulator tile held by lane group g.
__device__ __forceinline__ int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

// Tiles of AT rows (row0.., zero past T) of a head slice, staged through
// registers: load() issues the global loads (rows past T read a clamped
// row), store() writes LDS (zeroing rows past T).  Loading the next tile
// before computing on the current one keeps its memory latency behind the
// MFMA work.
//
// LDS tiles hold rows of HD contiguous elements, 16 rows to a group of
// 16 (HD + 8) elements; inside a group, row r sits in slot m(r) at a stride
// of HD + 8 elements.  Measured with the SQ LDS counters, a wavefront's
// 16-byte read occupies the LDS 4 cycles and an 8-byte transposing read 2
// when free of bank conflicts, a 16-byte write 8; for the access patterns
// of these tiles the conflicts follow 16 consecutive lanes (32 for the
// transposing read) per cycle over 256 bytes of banks.  A slot stride of
// HD + 8 elements puts slot j's 16-byte chunk c at bank group
// (j (HD/8 + 1) + c) mod 16, and the slots are permuted so that, with
// s(r) = 8 (r & 1) + 4 ((r >> 1) & 1) + ((r >> 2) & 3) the bank group of
// row r's chunk 0:
//  * row reads (16 consecutive rows, one chunk each) meet 16 values of s;
//  * transposing reads (4 consecutive rows, 4 adjacent chunks each) meet s
//    values 4 apart, so the rows' chunk runs tile the 16 bank groups;
//  * stores (8 lanes: 128 bytes of one row) cover distinct bank groups.
// The counters read no conflicts in any of the kernels below; rows in order
// at the same stride left the transposing reads four-way conflicted at
// head_dim 128 and two-way at 64.  m(r) = s(r) at HD = 128 (stride 17
// chunks, 17 = 1 mod 16) and 9 s(r) mod 16 at HD = 64 (stride 9,
// 9 * 9 = 1 mod 16).
// trow(a + b) = trow(a) + trow(b) for a a multiple of 16, and trow(r + 8) =
// trow(r) + 2 (HD + 8) for r % 16 < 8: callers split a row into a part known
// at compile time and a per-lane part, so every fragment offset is an
// immediate.
template <int HD>
__device__ __forceinline__ int trow(int r) {
  const int x = r & 15;
  const int s = ((x & 1) << 3) | ((x & 2) << 1) | ((x >> 2) & 3);
  const int m = HD == 128 ? s : (9 * s) & 15;
  return (HD + 8) * (16 * (r >> 4) + m);
}
// elements of an AT-row tile
template <int HD>
constexpr int tile_elems() { return AT * (HD + 8); }

template <int HD>
struct RowTile {
  static constexpr int CH = HD / 8, N = (AT * CH + 255) / 256;
  uint4 v[N];
  __device__ __forceinline__ void load(const bf16* src, int64_t ld, int row0, int T, int tid) {
#pragma unroll
    for (int k = 0; k < N; ++k) {
      const int i = tid + 256 * k;
      const int r = i / CH, c = (i % CH) * 8;
      const int row = min(row0 + r, T - 1);
      if (i < AT * CH) v[k] = *reinterpret_cast<const uint4*>(src + (int64_t)row * ld + c);
    }
  }
  __device__ __forceinline__ void store(bf16* s, int row0, int T, int tid) const {
#pragma unroll
    for (int k = 0; k < N; ++k) {
      const int i = tid + 256 * k;
      if (i >= AT * CH) continue;
      const int r = i / CH, c = i % CH;
      *reinterpret_cast<uint4*>(s + trow<HD>(r) + 8 * c) = row0 + r < T ? v[k] : make_uint4(0, 0, 0, 0);
    }
  }
};

// A or B operand fragment from an LDS tile: row rowbase + r (rowbase a
// multiple of 16), dims 16*kk + 8*g .. +7.
template <int HD>
__device__ __forceinline__ bf16x8v frag_rows(const bf16* s, int rowbase, int r, int kk, int g) {
  return *reinterpret_cast<const bf16x8v*>(s + trow<HD>(rowbase) + trow<HD>(r) + 16 * kk + 8 * g);
}

// Operand fragment for a contraction over the rows of an LDS tile (rowbase
// a multiple of 16): lane (c = lane % 32, g = lane / 32) gets column colbase + c
// of rows rowbase + {4g..4g+3, 8+4g..8+4g+3}, the order in which the
// accumulator registers of a 32x32 tile hold them.  ds_read_b64_tr_b16
// hands lane i of each 16-lane group element i % 4 of the 8-byte chunks
// addressed by lanes 4j + i / 4 (j = 0..3): lane L addresses row
// rowbase + 4g + L / 4 (then + 8), columns 4 (L % 4)..+3 of its group's 16.
typedef short i16x4v __attribute__((ext_vector_type(4)));
template <int HD>
__device__ __forceinline__ bf16x8v frag_tr(const bf16* s, int rowbase, int colbase, int lane) {
  const int L = lane & 15;
  const int col = colbase + 16 * ((lane >> 4) & 1) + 4 * (L & 3);
  const bf16* p = s + trow<HD>(rowbase) + trow<HD>(4 * (lane >> 5) + (L >> 2)) + col;
  typedef __attribute__((address_space(3))) i16x4v lds_i16x4;
  const lds_i16x4* p0 = reinterpret_cast<const lds_i16x4*>((__attribute__((address_space(3))) const char*)p);
  const lds_i16x4* p1 =
      reinterpret_cast<const lds_i16x4*>((__attribute__((address_space(3))) const char*)(p + 2 * (HD + 8)));
  const i16x4v a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_i16x4*>(p0));
  const i16x4v b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_i16x4*>(p1));
  const i16x4v* pa = &a;
  const i16x4v* pb = &b;
  return ld_2x4(reinterpret_cast<const bf16*>(pa), reinterpret_cast<const bf16*>(pb));
}

// Operand fragment straight from global memory (row of a head slice).
template <int HD>
__device__ __forceinline__ bf16x8v frag_global(const bf16* src, int64_t ld, int row, int T, int kk, int g) {
  if (row >= T) {
    bf16x8v z;
#pragma unroll
    for (int j = 0; j < 8; ++j) z[j] = static_cast<bf16>(0.f);
    return z;
  }
  return *reinterpret_cast<const bf16x8v*>(src + (int64_t)row * ld + 16 * kk + 8 * g);
}

// ------------------------------------------------------------- forward --
template <int HD, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void attn_fwd_mfma(const bf16* qkv, int T, int H, int Hkv, bf16* O,
                                                     int64_t ldo, float* lse) {
  constexpr int KK = HD / 16, NT = HD / 32;
  __shared__ __attribute__((aligned(16))) bf16 sK[tile_elems<HD>()];
  __shared__ __attribute__((aligned(16))) bf16 sV[tile_elems<HD>()];
  // grid (H, B, blocks): the causal block index varies slowest, so the
  // round-robin dispatch over XCDs gives every XCD the same mix of long and
  // short blocks; the longest (latest) query blocks are dispatched first.
  const int qb = gridDim.z - 1 - blockIdx.z;
  const int h = blockIdx.x, b = blockIdx.y;
  const int dA = H * HD, dKV = Hkv * HD, kvh = h / (H / Hkv);
  const int64_t ld = dA + 2 * (int64_t)dKV;
  const bf16* Qg = qkv + (int64_t)b * T * ld + h * HD;
  const bf16* Kg = qkv + (int64_t)b * T * ld + dA + kvh * HD;  // shared by the heads of a group
  const bf16* Vg = Kg + dKV;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5, c = lane & 31;
  const int q0 = qb * 128 + wave * 32;
  const int tq = q0 + c;
  const float sl2 = kLog2e / sqrtf((float)HD);

  bf16x8v qf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) qf[kk] = frag_global<HD>(Qg, ld, tq, T, kk, g);
  f32x16v acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = zero16();
  // Online softmax against a reference maximum mref (scaled scores, log2
  // units) that moves only when a row's maximum exceeds it by more than
  // kSlack: probabilities are exp2(s sl2 - mref) <= 2^kSlack, and acc and
  // lsum share mref, so O = acc / lsum is unchanged by where mref sits.
  constexpr float kSlack = 8.f;
  float mref = -INFINITY, lsum = 0.f;

  const int kend = CAUSAL ? min(T, qb * 128 + 128) : T;
  const int wave_kend = CAUSAL ? min(T, q0 + 32) : T;
  RowTile<HD> rk, rv;
  rk.load(Kg, ld, 0, T, tid);
  rv.load(Vg, ld, 0, T, tid);
  for (int k0 = 0; k0 < kend; k0 += AT) {
    __syncthreads();
    rk.store(sK, k0, T, tid);
    rv.store(sV, k0, T, tid);
    __syncthreads();
    if (k0 + AT < kend) {
      rk.load(Kg, ld, k0 + AT, T, tid);
      rv.load(Vg, ld, k0 + AT, T, tid);
    }
#pragma unroll
    for (int sub = 0; sub < AT / 32; ++sub) {
      const int kb = k0 + 32 * sub;
      if (kb >= wave_kend) break;
      f32x16v s = zero16();
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) s = mfma32(frag_rows<HD>(sK, 32 * sub, c, kk, g), qf[kk], s);
      // Causal: only the sub-tile on the diagonal (kb == q0) holds keys
      // after a query or past T; every earlier one is fully visible.
      // Without the mask only the last sub-tile can hold keys past T.
      if (CAUSAL ? kb + 31 > q0 : kb + 31 >= T) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kb + acc_row(r, g);
          if ((CAUSAL && key > tq) || key >= T) s[r] = -INFINITY;
        }
      }
      float mx = s[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * sl2;
      if (__any(mx > mref + kSlack)) {
        // the first sub-tile always lands here (mref = -inf; every row sees key 0)
        const float mn = mx > mref + kSlack ? mx : mref;
        const float alpha = __builtin_amdgcn_exp2f(mref - mn);
        lsum *= alpha;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[t][r] *= alpha;
        mref = mn;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[r], sl2, -mref));
        s[r] = p;
        lsum += p;
      }
      const bf16x8v p0 = pack8(s, 0), p1 = pack8(s, 8);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        acc[t] = mfma32(frag_tr<HD>(sV, 32 * sub, 32 * t, lane), p0, acc[t]);
        acc[t] = mfma32(frag_tr<HD>(sV, 32 * sub + 16, 32 * t, lane), p1, acc[t]);
      }
    }
  }
  const float l = lsum + __shfl_xor(lsum, 32, 64);
  if (tq < T) {
    const float inv = 1.f / l;
    bf16* orow = O + ((int64_t)b * T + tq) * ldo + h * HD;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        bf16x4v o;
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = static_cast<bf16>(acc[t][4 * r4 + j] * inv);
        *reinterpret_cast<bf16x4v*>(orow + 32 * t + 8 * r4 + 4 * g) = o;
      }
    if (g == 0) lse[((int64_t)b * H + h) * T + tq] = (mref + log2f(l)) * 0.6931471805599453f;
  }
}

// Scheduling groups for a run of N MFMAs that take R LDS read instructions
// each: the reads of the next LA MFMAs stay in flight, so a fragment read
// is not waited for right before its MFMA (head_dim 128, where one
// wavefront per SIMD leaves nothing else to cover that wait).  Ends the
// scheduling region.
template <int N, int R, int LA>
__device__ __forceinline__ void lds_ahead() {
  __builtin_amdgcn_sched_group_barrier(0x100, R * LA, 0);  // LDS reads of the first LA MFMAs
#pragma unroll
  for (int q = 0; q < N - LA; ++q) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, R, 0);  // LDS reads of the MFMA LA ahead
  }
  __builtin_amdgcn_sched_group_barrier(0x008, LA, 0);
  __builtin_amdgcn_sched_barrier(0);
}

// ------------------------------------------------------- backward: dK dV --
// dK and dV of a key block in one pass.  head_dim 64: two wavefronts per
// SIMD; head_dim 128: the accumulators take most of the register file, one
// wavefront per SIMD.  (A dV pass and a dK pass, each at two wavefronts per
// SIMD but both recomputing S, ran faster while the LDS tiles had bank
// conflicts and slower since: 467 -> 437 us for the backward at B4 T2048
// H16.)
template <int HD, bool CAUSAL, bool GQA>
__global__ __launch_bounds__(256, HD == 128 ? 1 : 2) void attn_bwd_dkdv_mfma(
    const bf16* qkv, const bf16* dO, int64_t lddo, const float* lse, const float* Dvec, int T, int H, int Hkv,
    bf16* dqkv) {
  constexpr int KK = HD / 16, NT = HD / 32;
  __shared__ __attribute__((aligned(16))) bf16 sQ[tile_elems<HD>()];
  __shared__ __attribute__((aligned(16))) bf16 sdO[tile_elems<HD>()];
  __shared__ float sL[AT], sD[AT];
  // grid (Hkv, B, blocks): causal block index slowest (even XCD mix); the
  // earliest key blocks see the most queries and are dispatched first.  A
  // key/value head accumulates over every query head of its group, in order.
  const int kb0 = blockIdx.z * 128;
  const int kvh = blockIdx.x, b = blockIdx.y, grp = GQA ? H / Hkv : 1;
  const int dA = H * HD, dKV = Hkv * HD;
  const int64_t ld = dA + 2 * (int64_t)dKV;
  const bf16* Qb = qkv + (int64_t)b * T * ld;
  const bf16* Kg = Qb + dA + kvh * HD;
  const bf16* Vg = Kg + dKV;
  const bf16* dOb = dO + (int64_t)b * T * lddo;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5, c = lane & 31;
  const int kw = kb0 + wave * 32;  // this wave's first key
  const int key = kw + c;          // this lane's key (column of S)
  const float sl2 = kLog2e / sqrtf((float)HD);

  bf16x8v kf[KK], vf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    kf[kk] = frag_global<HD>(Kg, ld, key, T, kk, g);
    vf[kk] = frag_global<HD>(Vg, ld, key, T, kk, g);
  }
  f32x16v dk[NT], dv[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    dk[t] = zero16();
    dv[t] = zero16();
  }

  // causal: only the queries at or after this block's keys see them.
  // Iteration it covers query tile it % nq of group head it / nq.
  const int qbeg = CAUSAL ? kb0 : 0;
  const int nq = qbeg < T ? (T - qbeg + AT - 1) / AT : 0;
  const int nit = grp * nq;
  RowTile<HD> rq, ro;
  if (nit > 0) {
    rq.load(Qb + kvh * grp * HD, ld, qbeg, T, tid);
    ro.load(dOb + kvh * grp * HD, lddo, qbeg, T, tid);
  }
  for (int it = 0; it < nit; ++it) {
    // without grouping the iteration is the query tile itself
    const int h = kvh * grp + (GQA ? it / nq : 0);
    const int q0 = qbeg + (GQA ? it % nq : it) * AT;
    const float* Lg = lse + ((int64_t)b * H + h) * T;
    const float* Dg = Dvec + ((int64_t)b * H + h) * T;
    __syncthreads();
    rq.store(sQ, q0, T, tid);
    ro.store(sdO, q0, T, tid);
    if (tid < AT) {
      const int tq = q0 + tid;
      sL[tid] = tq < T ? Lg[tq] * kLog2e : 0.f;
      sD[tid] = tq < T ? Dg[tq] : 0.f;
    }
    __syncthreads();
    if (it + 1 < nit) {
      const int hn = kvh * grp + (GQA ? (it + 1) / nq : 0);
      const int qn = qbeg + (GQA ? (it + 1) % nq : it + 1) * AT;
      rq.load(Qb + hn * HD, ld, qn, T, tid);
      ro.load(dOb + hn * HD, lddo, qn, T, tid);
    }
#pragma unroll
    for (int sub = 0; sub < AT / 32; ++sub) {
      const int qs = q0 + 32 * sub;
      if ((CAUSAL && qs + 31 < kw) || qs >= T) continue;  // whole sub-tile before this wave's keys
      f32x16v s = zero16(), dp = zero16();
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        s = mfma32(frag_rows<HD>(sQ, 32 * sub, c, kk, g), kf[kk], s);
        dp = mfma32(frag_rows<HD>(sdO, 32 * sub, c, kk, g), vf[kk], dp);
      }
      if (HD == 128) lds_ahead<2 * KK, 1, 4>();
      // s[r] = S[query qs + acc_row(r, g)][key].  Queries past T have zero
      // Q and dO rows and zero L and D, so they add nothing; only the
      // diagonal sub-tile (qs == kw) has queries before this wave's keys.
      const bool diag = CAUSAL && qs < kw + 32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qr = 32 * sub + acc_row(r, g);
        float p = __builtin_amdgcn_exp2f(fmaf(s[r], sl2, -sL[qr]));
        if (diag && key > q0 + qr) p = 0.f;
        s[r] = p;
        dp[r] = p * (dp[r] - sD[qr]);
      }
      // head_dim 128: the dV and dK MFMAs in a scheduling region of their
      // own, with the transposing reads of the next four in flight
      if (HD == 128) __builtin_amdgcn_sched_barrier(0);
      {
        const bf16x8v p0 = pack8(s, 0), p1 = pack8(s, 8);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          dv[t] = mfma32(p0, frag_tr<HD>(sdO, 32 * sub, 32 * t, lane), dv[t]);
          dv[t] = mfma32(p1, frag_tr<HD>(sdO, 32 * sub + 16, 32 * t, lane), dv[t]);
        }
      }
      {
        const bf16x8v d0 = pack8(dp, 0), d1 = pack8(dp, 8);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          dk[t] = mfma32(d0, frag_tr<HD>(sQ, 32 * sub, 32 * t, lane), dk[t]);
          dk[t] = mfma32(d1, frag_tr<HD>(sQ, 32 * sub + 16, 32 * t, lane), dk[t]);
        }
      }
      if (HD == 128) lds_ahead<4 * NT, 2, 4>();
    }
  }
  // dk[t][r] = dK[key kw + acc_row(r, g)][dim 32t + c]
  const float scale = 1.f / sqrtf((float)HD);
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int kr = kw + acc_row(r, g);
      if (kr < T) {
        bf16* row = dqkv + ((int64_t)b * T + kr) * ld + dA + kvh * HD + 32 * t + c;
        row[0] = static_cast<bf16>(dk[t][r] * scale);
        row[dKV] = static_cast<bf16>(dv[t][r]);
      }
    }
}

// ----------------------------------------------------------- backward: dQ --
template <int HD, bool CAUSAL>
// Also computes D = rowsum(dO * O) for its queries and writes it to Dvec
// for the dK/dV kernel, which runs after it.
__global__ __launch_bounds__(256, 2) void attn_bwd_dq_mfma(const bf16* qkv, const bf16* O, int64_t ldo,
                                                        const bf16* dO, int64_t lddo, const float* lse,
                                                        float* Dvec, int T, int H, int Hkv, bf16* dqkv) {
  constexpr int KK = HD / 16, NT = HD / 32;
  __shared__ __attribute__((aligned(16))) bf16 sK[tile_elems<HD>()];
  __shared__ __attribute__((aligned(16))) bf16 sV[tile_elems<HD>()];
  // grid (H, B, blocks): the causal block index varies slowest, so the
  // round-robin dispatch over XCDs gives every XCD the same mix of long and
  // short blocks; the longest (latest) query blocks are dispatched first.
  const int qb = gridDim.z - 1 - blockIdx.z;
  const int h = blockIdx.x, b = blockIdx.y;
  const int dA = H * HD, dKV = Hkv * HD, kvh = h / (H / Hkv);
  const int64_t ld = dA + 2 * (int64_t)dKV;
  const bf16* Qg = qkv + (int64_t)b * T * ld + h * HD;
  const bf16* Kg = qkv + (int64_t)b * T * ld + dA + kvh * HD;
  const bf16* Vg = Kg + dKV;
  const bf16* dOg = dO + (int64_t)b * T * lddo + h * HD;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5, c = lane & 31;
  const int q0 = qb * 128 + wave * 32;
  const int tq = q0 + c;
  const float sl2 = kLog2e / sqrtf((float)HD);

  bf16x8v qf[KK], of[KK];
  float dsum = 0.f;  // this lane's half of dO . O for query tq
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    qf[kk] = frag_global<HD>(Qg, ld, tq, T, kk, g);
    of[kk] = frag_global<HD>(dOg, lddo, tq, T, kk, g);
    const bf16x8v o8 = frag_global<HD>(O + (int64_t)b * T * ldo + h * HD, ldo, tq, T, kk, g);
#pragma unroll
    for (int j = 0; j < 8; ++j) dsum += static_cast<float>(of[kk][j]) * static_cast<float>(o8[j]);
  }
  const float L2 = tq < T ? lse[((int64_t)b * H + h) * T + tq] * kLog2e : 0.f;
  const float Dq = tq < T ? dsum + __shfl_xor(dsum, 32, 64) : 0.f;
  if (g == 0 && tq < T) Dvec[((int64_t)b * H + h) * T + tq] = Dq;
  f32x16v dq[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) dq[t] = zero16();

  const int kend = CAUSAL ? min(T, qb * 128 + 128) : T;
  const int wave_kend = CAUSAL ? min(T, q0 + 32) : T;
  RowTile<HD> rk, rv;
  rk.load(Kg, ld, 0, T, tid);
  rv.load(Vg, ld, 0, T, tid);
  for (int k0 = 0; k0 < kend; k0 += AT) {
    __syncthreads();
    rk.store(sK, k0, T, tid);
    rv.store(sV, k0, T, tid);
    __syncthreads();
    if (k0 + AT < kend) {
      rk.load(Kg, ld, k0 + AT, T, tid);
      rv.load(Vg, ld, k0 + AT, T, tid);
    }
#pragma unroll
    for (int sub = 0; sub < AT / 32; ++sub) {
      const int kb = k0 + 32 * sub;
      if (kb >= wave_kend) break;
      f32x16v s = zero16(), dp = zero16();
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        s = mfma32(frag_rows<HD>(sK, 32 * sub, c, kk, g), qf[kk], s);
        dp = mfma32(frag_rows<HD>(sV, 32 * sub, c, kk, g), of[kk], dp);
      }
      if (HD == 128) lds_ahead<2 * KK, 1, 4>();
      // s[r] = S^T[key kb + acc_row(r, g)][query tq].  Keys past T have
      // zero K and V rows (dS there multiplies a zero K row); only the
      // diagonal sub-tile (kb == q0) has keys after a query.
      const bool diag = CAUSAL && kb + 31 > q0;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = __builtin_amdgcn_exp2f(fmaf(s[r], sl2, -L2));
        if (diag && kb + acc_row(r, g) > tq) p = 0.f;
        dp[r] = p * (dp[r] - Dq);
      }
      if (HD == 128) __builtin_amdgcn_sched_barrier(0);
      const bf16x8v d0 = pack8(dp, 0), d1 = pack8(dp, 8);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        dq[t] = mfma32(frag_tr<HD>(sK, 32 * sub, 32 * t, lane), d0, dq[t]);
        dq[t] = mfma32(frag_tr<HD>(sK, 32 * sub + 16, 32 * t, lane), d1, dq[t]);
      }
      if (HD == 128) lds_ahead<2 * NT, 2, 4>();
    }
  }
  if (tq < T) {
    const float scale = 1.f / sqrtf((float)HD);
    bf16* row = dqkv + ((int64_t)b * T + tq) * ld + h * HD;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        bf16x4v o;
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = static_cast<bf16>(dq[t][4 * r4 + j] * scale);
        *reinterpret_cast<bf16x4v*>(row + 32 * t + 8 * r4 + 4 * g) = o;
      }
  }
}

bool attn_mfma_supported(int hd) { return hd == 64 || hd == 128; }


template <int HD, bool CAUSAL>
static void fwd_launch(dim3 grid, hipStream_t s, const bf16* q, int T, int H, int Hkv, bf16* o, int64_t ldo,
                       float* lse) {
  hipLaunchKernelGGL((attn_fwd_mfma<HD, CAUSAL>), grid, dim3(256), 0, s, q, T, H, Hkv, o, ldo, lse);
}

hipError_t attn_fwd_mfma_launch(const void* qkv, int B, int T, int H, int Hkv, int hd, int causal, void* O,
                                int64_t ldo, float* lse, hipStream_t s) {
  const dim3 grid(H, B, cdiv(T, 128));
  const bf16* q = static_cast<const bf16*>(qkv);
  bf16* o = static_cast<bf16*>(O);
  if (hd == 64) {
    if (causal) fwd_launch<64, true>(grid, s, q, T, H, Hkv, o, ldo, lse);
    else fwd_launch<64, false>(grid, s, q, T, H, Hkv, o, ldo, lse);
  } else if (hd == 128) {
    if (causal) fwd_launch<128, true>(grid, s, q, T, H, Hkv, o, ldo, lse);
    else fwd_launch<128, false>(grid, s, q, T, H, Hkv, o, ldo, lse);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// dQ over (query head, sequence, query block); dK / dV over (key/value
// head, sequence, key block).
template <int HD, bool CAUSAL, bool GQA>
static void dkdv_launch(dim3 gk, hipStream_t s, const bf16* q, const bf16* d, int64_t lddo, const float* lse,
                        const float* Dvec, int T, int H, int Hkv, bf16* o) {
  const dim3 block(256);
  hipLaunchKernelGGL((attn_bwd_dkdv_mfma<HD, CAUSAL, GQA>), gk, block, 0, s, q, d, lddo, lse, Dvec, T, H, Hkv, o);
}

template <int HD, bool CAUSAL>
static void bwd_launch(int B, int T, int H, int Hkv, hipStream_t s, const bf16* q, const bf16* ob, int64_t ldo,
                       const bf16* d, int64_t lddo, const float* lse, float* Dvec, bf16* o) {
  const dim3 block(256), gq(H, B, cdiv(T, 128)), gk(Hkv, B, cdiv(T, 128));
  hipLaunchKernelGGL((attn_bwd_dq_mfma<HD, CAUSAL>), gq, block, 0, s, q, ob, ldo, d, lddo, lse, Dvec, T, H, Hkv, o);
  if (Hkv == H) dkdv_launch<HD, CAUSAL, false>(gk, s, q, d, lddo, lse, Dvec, T, H, Hkv, o);
  else dkdv_launch<HD, CAUSAL, true>(gk, s, q, d, lddo, lse, Dvec, T, H, Hkv, o);
}

// dQ first (it also writes D = rowsum(dO * O) into Dvec), then dK / dV.
hipError_t attn_bwd_mfma_launch(const void* qkv, const void* O, int64_t ldo, const void* dO, int64_t lddo,
                                const float* lse, float* Dvec, int B, int T, int H, int Hkv, int hd, int causal,
                                void* dqkv, hipStream_t s) {
  const bf16* q = static_cast<const bf16*>(qkv);
  const bf16* ob = static_cast<const bf16*>(O);
  const bf16* d = static_cast<const bf16*>(dO);
  bf16* o = static_cast<bf16*>(dqkv);
  if (hd == 64) {
    if (causal) bwd_launch<64, true>(B, T, H, Hkv, s, q, ob, ldo, d, lddo, lse, Dvec, o);
    else bwd_launch<64, false>(B, T, H, Hkv, s, q, ob, ldo, d, lddo, lse, Dvec, o);
  } else if (hd == 128) {
    if (causal) bwd_launch<128, true>(B, T, H, Hkv, s, q, ob, ldo, d, lddo, lse, Dvec, o);
    else bwd_launch<128, false>(B, T, H, Hkv, s, q, ob, ldo, d, lddo, lse, Dvec, o);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace fal
