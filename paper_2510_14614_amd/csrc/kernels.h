// Internal launch interface between the host scheduler (api.cpp) and the
// HIP kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fal {

enum DType : int { F32 = 0, BF16 = 1 };

// ---------------------------------------------------------------- GEMM ----
// C[m, n] = sum_k A(m, k) B(k, n) over one or two K segments, followed by an
// epilogue.  Operand orientation:
//   a_kmaj = 1: A(m, k) = A[m * lda + k]   (k contiguous)
//   a_kmaj = 0: A(m, k) = A[k * lda + m]   (m contiguous)
//   b_kmaj = 1: B(k, n) = B[n * ldb + k]   (k contiguous)
//   b_kmaj = 0: B(k, n) = B[k * ldb + n]   (n contiguous)
// A and B hold the storage dtype of the launch; accumulation is fp32.
enum Epi : int {
  EPI_STORE = 0,     // out = acc + bias (+ bias2)          (out: f32 or dtype)
  EPI_GELU = 1,      // v = acc + bias: out = GELU(v), out2 = GELU'(v) if out2   (dtype)
  EPI_RESID = 2,     // out(f32) = resid(f32) + acc + bias   (resid may equal out)
  EPI_MUL_AUX = 3,   // out = acc * aux (aux = GELU' saved by EPI_GELU)  (aux, out: dtype)
};

struct GemmProblem {
  const void* A;
  const void* B;
  const void* A2;  // second K segment (K-concatenation); NULL if K2 == 0
  const void* B2;
  int64_t lda, ldb, lda2, ldb2;
  int M, N, K, K2;
  int epi;
  int out_f32;        // EPI_STORE: 1 -> out is fp32, 0 -> out is dtype
  const void* bias;   // dtype [N] or NULL
  const void* bias2;  // dtype [N] or NULL, added as well (K-concatenated layers)
  const float* resid; // EPI_RESID
  int64_t ldr;
  void* out;
  int64_t ldo;
  void* out2;         // EPI_GELU: GELU derivative at the pre-activation
  int64_t ldo2;
  const void* aux;    // EPI_MUL_AUX: elementwise factor
  int64_t ldaux;
  // 1: the k-contiguous operand's rows hold finite values in columns
  // K .. roundup(K, 8) - 1 (zero padding).  Lets a problem whose K is not a
  // multiple of 8 run on the pipelined kernel when the other operand is
  // MN-major (its rows past K read as zero).
  int kpad;
  // filled in by the launcher
  int tiles_m, tiles_n, tile_start;
  int splits;        // K split into this many slices (fp32 partials + reduce)
  int vec_out;       // rows of outputs / residual / aux (and the biases) allow 4-column vectors
  float* part;       // [splits][M][N] fp32 partials when splits > 1
};

constexpr int kMaxGroup = 4;
struct GemmGroup {
  GemmProblem p[kMaxGroup];
  int n;
  int total_tiles;
};

// Launches every problem of `g` (same dtype and operand orientation) as one
// grouped kernel.  Problems that would leave most compute units idle (few
// output tiles, long K, fp32 EPI_STORE output, single K segment) have their
// K range split across workgroups: each slice writes fp32 partials to
// `splitk_scratch` and a second kernel sums the slices in a fixed order, so
// results stay deterministic.  splitk_floats: capacity of the scratch (0
// disables splitting).  Returns hipSuccess or the launch error; `why`
// receives a static message for argument errors.
hipError_t gemm(DType dt, int a_kmaj, int b_kmaj, GemmGroup& g, int gelu_tanh, hipStream_t s,
                const char** why, float* splitk_scratch = nullptr, int64_t splitk_floats = 0);
// The share of the chip's workgroup slots the launch of `g` would occupy
// in its last round (1.0 when its tiles fill whole rounds; 1.0 as well for
// launches off the matrix-core path).  Lets a scheduler tell whether
// another launch can use compute units this one leaves idle.
double gemm_last_round_fill(DType dt, int a_kmaj, int b_kmaj, const GemmGroup& g, int64_t splitk_floats);

// ----------------------------------------------------------- LayerNorm ----
// Row LayerNorm over d of fp32 rows x.  Writes
//   y1 = LN(x; g1, b1)                               (dtype)  if y1
//   y2 = LN(x; g2, b2) + add2                        (dtype)  if y2 and add2
//   y2 = LN(x; g2, b2) + gF * xhatF + bF             (dtype)  if y2 and xhatF
//   y2 = LN(x; g2, b2)                               (dtype)  if y2 only
//   xhat_out = (x - mean) * rstd                     (dtype)  if xhat_out
// and saves mean, rstd (fp32 [M]) if non-NULL.  add2, xhatF, gF, bF: dtype.
struct LnFwdArgs {
  const float* x;
  int M, d;
  float eps;
  const void *g1, *b1;
  void* y1;
  const void *g2, *b2;
  void* y2;
  const void* add2;
  const void *xhatF, *gF, *bF;
  void* xhat_out;
  float* mean;
  float* rstd;
};
hipError_t ln_fwd(DType dt, const LnFwdArgs& a, hipStream_t s);

// LayerNorm backward over rows, with up to two LayerNorms of the same input
// x (fp32; shared mean/rstd):
//   dxhat = dy1 * g1 + dy2 * g2                                  (dy*: fp32)
//   dx = dres + rstd * (dxhat - mean(dxhat) - xhat * mean(dxhat * xhat))
// with xhat = (x - mean) * rstd recomputed.  Optionally
//   dacc (+)= dy2                       FAL: first-attention accumulator
//   dxhatF_acc (+)= gF * dy2            FAL+: accumulator of the shared
//                                       first-attention normalisation
// ("=" when the matching *_overwrite flag is set).  dx (fp32) may alias
// dres; dres may be NULL (treated as 0).  dx_lp (dtype copy of dx) is
// written if non-NULL.  Parameter gradients (fp32 [d], each optional):
//   dg1 = sum_rows dy1 * xhat, db1 = sum_rows dy1,
//   dg2 = sum_rows dy2 * xhat, db2 = sum_rows dy2,
//   dgF = sum_rows dy2 * xhatF, dbF = sum_rows dy2,
// reduced deterministically through `partials` (ln_bwd_scratch floats).
struct LnBwdArgs {
  const float* x;
  const float* mean;
  const float* rstd;
  int M, d;
  const float* dy1;
  const void* g1;
  const float* dy2;
  const void* g2;
  const float* dres;
  float* dx;
  void* dx_lp;
  float* dacc;
  int dacc_overwrite;
  const void* xhatF;
  const void* gF;
  float* dxhatF_acc;
  int dxhatF_overwrite;
  float *dg1, *db1, *dg2, *db2, *dgF, *dbF;
  float* partials;
};
hipError_t ln_bwd(DType dt, const LnBwdArgs& a, hipStream_t s);
int64_t ln_bwd_scratch(int M, int d);

// The FAL+ terms of the LN2 backward of up to kSideGroup consecutive
// blocks as one separate pass (so they can run beside the next blocks'
// backward, and the shared accumulator and xhatF are read once per group):
// dxhatF_acc (+)= gF[0] * dy2[0] + gF[1] * dy2[1] + ... added in that order
// ("=" when overwrite), and dgF[k] = sum_rows dy2[k] * xhatF (fixed order
// through falplus_side_scratch floats of scratch).  dy2[k], dxhatF_acc:
// fp32 [M, d]; xhatF, gF[k]: dtype.  falplus_side_ok tells whether one
// block's operands have the vector layout the pass needs (d % 4, aligned
// rows).
// (Groups of 8 measured no faster than 4 at GPT-2 small to ~1.3B shapes.)
constexpr int kSideGroup = 4;
struct FalPlusSide {
  int n;  // blocks in the group, 1 .. kSideGroup
  const float* dy2[kSideGroup];
  const void* gF[kSideGroup];
  float* dgF[kSideGroup];
};
bool falplus_side_ok(DType dt, int d, const float* dy2, const void* xhatF, const void* gF, const float* acc);
hipError_t falplus_side(DType dt, const FalPlusSide& g, const void* xhatF, float* dxhatF_acc, int overwrite, int M,
                        int d, float* scratch, hipStream_t s);
int64_t falplus_side_scratch(int M, int d);

// Backward of the affine-free normalisation xhat = (a - mean) * rstd given
// dxhat (fp32), added to a residual gradient in one pass:
//   da = dres + rstd * (dxhat - mean(dxhat) - xhat * mean(dxhat*xhat))
// with xhat recomputed from a (fp32); dres may be NULL (zero) or alias da;
// da_lp (dtype copy of da) is written if non-NULL.
hipError_t norm_bwd(DType dt, const float* a, const float* mean, const float* rstd, const float* dxhat,
                    int M, int d, const float* dres, float* da, void* da_lp, hipStream_t s);

// Sum `nblk` partial rows of width d: out[j] = sum_b part[b * stride + j].
hipError_t col_reduce(const float* part, int nblk, int64_t stride, int d, float* out, hipStream_t s);

// Several bias gradients at once: out_i[j] = sum_m x_i[m, j] for up to
// kColSumMax inputs of their own width N_i (multiple of 4) and storage
// (fp32 or dtype), two kernels in all.  out2_i, if set, receives the same
// sums (two biases with one gradient).  Fixed summation order.
constexpr int kColSumMax = 4;
struct ColSumInput {
  const void* x;
  int64_t ld;
  int N, f32;
  float* out;
  float* out2;
};
struct ColSumBatch {
  ColSumInput in[kColSumMax];
  int n, M;
};
hipError_t col_sum_batch(DType dt, const ColSumBatch& b, float* scratch, hipStream_t s);
// scratch floats for a batch whose widths add up to W
int64_t col_sum_batch_scratch(int M, int W);

// ------------------------------------------------------------ attention ----
// Multi-head attention on the packed QKV activations [M, dA + 2*dKV]
// (Q | K | V, dA = H*hd, dKV = Hkv*hd, head h at h*hd of its part; query
// head h reads key/value head h / (H / Hkv)), M = B*T; causal = 1: query t
// sees keys 0..t, 0: every key of its sequence.  O: dtype [M, ldo] (head h at column h*hd), LSE: fp32
// [B, H, T] (natural log of the softmax denominators including the
// 1/sqrt(hd) scale).
hipError_t attn_fwd(DType dt, const void* qkv, int B, int T, int H, int Hkv, int hd, int causal, void* O,
                    int64_t ldo, float* lse, hipStream_t s);
// Backward: from dO (dtype [M, ldo]) produce dQKV (dtype [M, dA + 2dKV]); a
// key/value head's gradient sums its group's query heads in head order.
// Dvec: fp32 [B, H, T] scratch (rowsum(dO * O)); dq_acc: fp32 [M, dA] scratch.
hipError_t attn_bwd(DType dt, const void* qkv, const void* O, int64_t ldo, const void* dO,
                    int64_t lddo, const float* lse, int B, int T, int H, int Hkv, int hd, int causal, void* dqkv,
                    float* Dvec, float* dq_acc, hipStream_t s);

// ------------------------------------------------ embedding / loss / misc ----
// X[m, :] = wte[tok[b, t]] + wpe[t]  (fp32 out), tokens [B, T+1].
hipError_t embed_fwd(DType dt, const int32_t* tokens, int B, int T, int V, int d, const void* wte,
                     const void* wpe, float* X, hipStream_t s);
// Sorts the (input id, position) pairs of the batch into sort_scratch
// (int32 of embed_bwd_scratch(M) elements).  Depends on the tokens only, so
// it can run ahead of (or beside) the rest of the step.  Requires
// B*T <= 16384.
hipError_t embed_sort(const int32_t* tokens, int B, int T, int V, int32_t* sort_scratch, hipStream_t s);
// dwte[v] += sum over positions with input id v of dX rows, in position
// order (deterministic; sort_scratch as written by embed_sort), dwpe[t] =
// sum_b dX[b, t].  partial: fp32 [M, d] scratch.
hipError_t embed_bwd(int B, int T, int d, const float* dX, float* dwte, float* dwpe,
                     const int32_t* sort_scratch, float* partial, hipStream_t s);
int64_t embed_bwd_scratch(int M);

// Cross-entropy over rows of logits [M, V] (dtype: fp32 or bf16, row
// stride ldl) with targets tokens[b, t + 1].  Writes dlogits =
// (softmax - onehot) / M as dtype [M, ldd] (columns V..ldd-1 zeroed;
// skipped when dlogits is NULL, ldd still a multiple of 4 >= V) and
// per-row loss (fp32 [M]); then loss = mean(row_loss) (fp32 scalar,
// fixed-order reduction).  Softmax, log-sum-exp and loss are fp32.
hipError_t cross_entropy(DType dt, const void* logits, int64_t ldl, const int32_t* tokens, int B,
                         int T, int V, void* dlogits, int64_t ldd, float* row_loss, float* loss,
                         hipStream_t s);
// dst[r, c] = src[r, c] widened to fp32, for r < rows and c < cols.
hipError_t rows_to_f32(DType dt, const void* src, int64_t lds, float* dst, int64_t ldd, int rows, int cols,
                       hipStream_t s);

// loss = sum(a * b) over n fp32 elements (fixed-order reduction); scratch of
// dot_scratch(n) floats.
hipError_t dot(const float* a, const float* b, int64_t n, float* loss, float* scratch,
               hipStream_t s);
int64_t dot_scratch(int64_t n);

// y = a + b (fp32, n elements); y may alias a.
hipError_t add_f32(const float* a, const float* b, float* y, int64_t n, hipStream_t s);
// Convert fp32 -> dtype.
hipError_t cast_from_f32(DType dt, const float* x, void* y, int64_t n, hipStream_t s);
// Read the whole 16-byte chunks of [p, p + bytes) and discard: warms the last-level
// cache with a read-only operand before the kernels that use it.
hipError_t cache_warm(const void* p, int64_t bytes, hipStream_t s);
// Fill fp32 with zero (a kernel, so it can live inside captured graphs).
hipError_t zero_f32(float* y, int64_t n, hipStream_t s);
// y = x over n fp32 elements (a kernel rather than a runtime copy, so every
// node of a captured step is a kernel).
hipError_t copy_f32(float* y, const float* x, int64_t n, hipStream_t s);

// ----------------------------------------------------------- optimizer ----
// AdamW over a flat fp32 buffer (Adam's bias-corrected moments, decoupled
// weight decay), after scaling the gradient by a global-norm clip factor.
constexpr int kNormBlocks = 2048;  // fp64 partial sums of the norm pass
struct AdamwConsts {
  float beta1, one_minus_beta1, beta2, one_minus_beta2;
  float eps;
  float rsqrt_bc2;  // 1 / sqrt(1 - beta2^step)
  float step_size;  // lr / (1 - beta1^step)
  float decay;      // 1 - lr * weight_decay
};
// part: kNormBlocks doubles of scratch; ctrl: 2 floats.
// ctrl[0] = ||g||_2 over n fp32 elements (fixed-order fp64 reduction),
// ctrl[1] = min(1, max_norm / (norm + 1e-6)) (1 when max_norm <= 0);
// norm_out (may be NULL) receives the norm.  g 16-byte aligned.
hipError_t grad_norm(const float* g, int64_t n, float max_norm, double* part, float* ctrl, float* norm_out,
                     hipStream_t s);
// One update of n elements with the gradient scaled by ctrl[1].  lp_mode 0:
// master is the parameter buffer; 1: fp32 copy written to lp; 2: bf16 copy
// (round to nearest even) written to lp.  fp32 arrays 16-byte aligned, lp
// 8-byte (bf16) or 16-byte (fp32) aligned.
hipError_t adamw_update(int lp_mode, float* master, void* lp, const float* g, float* m, float* v, int64_t n,
                        const AdamwConsts& k, const float* ctrl, hipStream_t s);
// The update kernel's grid covers 2048 elements per workgroup with at most
// 2^31 - 1 workgroups.
constexpr int64_t kAdamwMaxElems = (int64_t)0x7fffffff * 2048;
// grad_norm + adamw_update with their scratch (the norm partials and the
// control block) in a fixed device array of the library, one per GPU,
// instead of caller memory: no allocation anywhere.  The array's address on
// the current device is looked up once per device.  Calls that overlap on
// one GPU share the array.
hipError_t adamw_static_scratch(int lp_mode, float* master, void* lp, const float* g, float* m, float* v, int64_t n,
                                float max_norm, const AdamwConsts& k, float* norm_out, hipStream_t s);

}  // namespace fal
