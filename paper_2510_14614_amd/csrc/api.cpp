// C ABI of libfal.so (declared in include/fal.h): configuration checks,
// parameter layout, workspace carve-up and the host-side schedule of one
// training step of a GPT / FAL / FAL+ decoder stack.
//
// Block forward (Sec. 2 Eq. 1; Sec. 4.1 Eq. 2; Sec. 5 and Appendix D):
//   GPT   : H1 = LN1(X); A = MHA(H1); Xm = X + A; H2 = LN2(Xm);
//           Y = Xm + MLP(H2)
//   FAL   : block 0: H1 = LN1(X); A_1 = MHA(H1); F = LN_F(A_1);
//                    H2 = LN2(X) + F; Y = X + A_1 + MLP(H2)
//           block i>0: one LayerNorm pass gives H1 = LN1(X) and
//                    H2 = LN2(X) + F; then MHA(H1) and MLP(H2) are
//                    independent (Sec. 4.2) and are issued concurrently:
//                    SEQ     back to back on one stream,
//                    STREAMS MHA on the main stream, MLP on the aux stream,
//                    MERGED  QKV and FFN-up GEMMs as one grouped launch and
//                            the output and down projections as one GEMM
//                            over the concatenated inner dimension [O | G].
//   FAL+  : block 0 is the GPT block and also saves xhatF = norm(A_1);
//           block i>0: H2 = LN2(X + A) + gF_i * xhatF + bF_i.
// The backward mirrors this; FAL's MLP and MHA backward chains are again
// independent for i > 0 and meet in one LayerNorm backward that handles
// both LayerNorms of X at once and accumulates dF.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/fal.h"
#include "kernels.h"

using namespace fal;

namespace {

constexpr int64_t kAlignElems = 64;
constexpr size_t kAlignBytes = 256;

int64_t align_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

struct Dims {
  int L, d, H, hd, dA, f, V, Vp, T, B, M;
  int Hkv, dqkv;  // key/value heads; QKV width dA + 2 * Hkv * hd
  size_t es;  // bytes per stored element
};

Dims dims_of(const fal_config_t& c) {
  Dims D;
  D.L = c.n_layer; D.d = c.d_model; D.H = c.n_head; D.hd = c.head_dim;
  D.dA = c.n_head * c.head_dim; D.f = c.d_ff;
  D.Hkv = c.n_kv_head > 0 ? c.n_kv_head : c.n_head;
  D.dqkv = D.dA + 2 * D.Hkv * c.head_dim;
  D.V = c.has_embed_head ? c.vocab : 0;
  D.Vp = (int)align_up(D.V, 64);
  D.T = c.seq_len; D.B = c.batch; D.M = c.batch * c.seq_len;
  D.es = c.dtype == FAL_BF16 ? 2 : 4;
  return D;
}

const char* validate(const fal_config_t* c) {
  if (!c) return "config is NULL";
  if (c->n_layer < 1) return "n_layer must be >= 1";
  if (c->d_model < 8 || c->d_model % 8) return "d_model must be a positive multiple of 8";
  if (c->d_model > 4096) return "d_model above 4096 is not supported";
  if (c->n_head < 1) return "n_head must be >= 1";
  if (c->d_ff < 8 || c->d_ff % 8) return "d_ff must be a positive multiple of 8";
  if (c->seq_len < 1 || c->batch < 1) return "seq_len and batch must be >= 1";
  if (c->arch < FAL_ARCH_GPT || c->arch > FAL_ARCH_PARALLEL) return "unknown arch";
  if (c->dtype != FAL_F32 && c->dtype != FAL_BF16) return "unknown dtype";
  if (c->sched < FAL_SCHED_SEQ || c->sched > FAL_SCHED_STREAMS_MERGED) return "unknown sched";
  if (!(c->ln_eps > 0.f)) return "ln_eps must be > 0";
  if (c->gelu_tanh != 0 && c->gelu_tanh != 1) return "gelu_tanh must be 0 or 1";
  if (c->has_embed_head != 0 && c->has_embed_head != 1) return "has_embed_head must be 0 or 1";
  if (c->fal_block1_mode != 0 && c->fal_block1_mode != 1) return "fal_block1_mode must be 0 or 1";
  if (c->fal_block1_mode == 1 && c->arch != FAL_ARCH_FAL) return "fal_block1_mode 1 applies to FAL only";
  if (c->bidirectional != 0 && c->bidirectional != 1) return "bidirectional must be 0 or 1";
  if (c->n_kv_head < 0 || (c->n_kv_head > 0 && c->n_head % c->n_kv_head))
    return "n_kv_head must be 0 or divide n_head";
  if (c->bidirectional && c->has_embed_head)
    return "bidirectional attention is for the block stack (has_embed_head = 0): the next-token loss needs the causal mask";
  if (c->has_embed_head) {
    if (c->vocab < 1) return "vocab must be >= 1";
    if (c->vocab > 65535) return "vocab above 65535 is not supported";
    if ((int64_t)c->batch * c->seq_len > 16384) return "batch*seq_len above 16384 with an embedding is not supported";
  }
  if ((int64_t)c->batch * c->seq_len > (1 << 24)) return "batch*seq_len too large";
  return nullptr;
}

bool unsupported(const char* why) {
  return why && (strstr(why, "not supported") != nullptr);
}

const char* validate_hd(const fal_config_t* c) {
  const int hd = c->head_dim;
  if (hd != 16 && hd != 32 && hd != 64 && hd != 128) return "head_dim must be 16, 32, 64 or 128 (not supported otherwise)";
  if ((c->n_head * hd) % 8) return "n_head*head_dim must be a multiple of 8 (not supported otherwise)";
  return nullptr;
}

// The bf16 GEMM kernels address each operand through a buffer descriptor
// with 32-bit byte offsets, and a weight-gradient operand (contraction over
// the M token rows) is read up to 256 rows past its end inside that range.
// So every [M, width] operand of the step -- the saved activations [M, d],
// [M, dA + 2 dKV], [M, dA + f] and the logits [M, V] -- must span less than
// 2 GiB including those rows.  (The fp32 parity path indexes with 64 bits.)
const char* validate_extent(const fal_config_t* c) {
  if (c->dtype != FAL_BF16) return nullptr;
  const Dims D = dims_of(*c);
  const int64_t es = 2;
  int64_t width = std::max<int64_t>({(int64_t)D.d, (int64_t)D.dqkv, (int64_t)D.dA + D.f});
  if (c->has_embed_head) width = std::max<int64_t>(width, D.Vp);
  const int64_t limit = ((int64_t)1 << 31) - ((int64_t)1 << 20);
  if (((int64_t)D.M + 256) * width * es >= limit)
    return "batch*seq_len too large: a bf16 GEMM operand would span 2 GiB or more (not supported)";
  return nullptr;
}

struct Layout {
  int64_t goff[FAL_P_NGLOBAL];
  int64_t boff[FAL_B_NTENSOR];
  int64_t bsize[FAL_B_NTENSOR];
  int64_t gsize[FAL_P_NGLOBAL];
  int64_t block_base, block_stride, total;
};

Layout layout_of(const fal_config_t& c) {
  const Dims D = dims_of(c);
  Layout Lo;
  int64_t off = 0;
  const int64_t gs[FAL_P_NGLOBAL] = {(int64_t)D.V * D.d, (int64_t)D.T * D.d, D.d, D.d};
  for (int i = 0; i < FAL_P_NGLOBAL; ++i) {
    Lo.gsize[i] = c.has_embed_head ? gs[i] : 0;
    if (c.has_embed_head) {
      Lo.goff[i] = off;
      off += align_up(gs[i], kAlignElems);
    } else {
      Lo.goff[i] = -1;
    }
  }
  Lo.block_base = off;
  const int64_t d = D.d, dA = D.dA, f = D.f, q3 = D.dqkv;
  const int64_t bs[FAL_B_NTENSOR] = {d, d, d * q3, q3, dA * d, d, d, d, d * f, f, f * d, d, d, d};
  int64_t b = 0;
  for (int i = 0; i < FAL_B_NTENSOR; ++i) {
    Lo.boff[i] = b;
    Lo.bsize[i] = bs[i];
    b += align_up(bs[i], kAlignElems);
  }
  Lo.block_stride = b;
  Lo.total = off + b * D.L;
  return Lo;
}

// ------------------------------------------------------------ workspace --
struct Carve {
  char* base;
  size_t off = 0;
  template <typename T> T* take(int64_t n, size_t elem = sizeof(T)) {
    off = (off + kAlignBytes - 1) / kAlignBytes * kAlignBytes;
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += (size_t)n * elem;
    return p;
  }
};

struct LayerSlot {
  float *mean1, *rstd1, *mean2, *rstd2;
  void *h1, *h2, *qkv, *og, *dgelu;  // dgelu: GELU' at the FFN pre-activation
  float *lse, *xm;
};

struct Work {
  LayerSlot* slots = nullptr;  // host array [L]
  float *a1, *meanF, *rstdF;   // block 0 extras
  float* resid;                // [L+1][M, d]
  void* hf;
  float *meanf, *rstdf;
  void* logits;                // dtype [M, Vp]
  void* dlogits;               // [M, Vp]
  float* row_loss;
  void* first;                 // dtype [M, d]
  float* dfirst;               // [M, d]
  float *dxa, *dxb, *dxm, *da, *dh1, *dh2;
  void *lp_a, *lp_b, *dxm_lp, *da_lp, *dog, *dqkv;
  // FAL+: a ring of kSideGroup + 1 dH2 buffers indexed by layer, so a
  // group's deferred first-attention terms read its blocks' dH2 while the
  // next blocks write theirs
  float* dh2r[kSideGroup + 1];
  float* fp_part;  // FAL+: partial sums of those terms
  void *dog2[2], *dqkv2[2];  // per block parity: the pending bias sums of block i read block i's
  float* Dvec;
  float *part_main, *part_aux;
  float* bias_part;  // packed column-sum partials of one block's bias gradients
  float *splitk_main, *splitk_aux, *splitk_side;  // split-K partials, one region per stream
  int64_t splitk_floats;
  int32_t* keys;
  float* loss_tmp;
  double* opt_part;  // fp64 partial sums of the gradient-norm pass
  float* opt_ctrl;   // {norm, clip factor}
};

void carve(const fal_config_t& c, char* base, Work& W, size_t* total) {
  const Dims D = dims_of(c);
  Carve cv{base};
  const int64_t M = D.M, d = D.d, es = (int64_t)D.es;
  const bool need_xm = c.arch != FAL_ARCH_FAL && c.arch != FAL_ARCH_PARALLEL;
  for (int i = 0; i < D.L; ++i) {
    LayerSlot s{};
    s.mean1 = cv.take<float>(M);
    s.rstd1 = cv.take<float>(M);
    s.h1 = cv.take<char>(M * d * es);
    s.h2 = cv.take<char>(M * d * es);
    s.qkv = cv.take<char>(M * D.dqkv * es);
    s.og = cv.take<char>(M * (int64_t)(D.dA + D.f) * es);
    s.dgelu = cv.take<char>(M * D.f * es);
    s.lse = cv.take<float>((int64_t)D.B * D.H * D.T);
    if (need_xm || i == 0) {
      s.xm = cv.take<float>(M * d);
      s.mean2 = cv.take<float>(M);
      s.rstd2 = cv.take<float>(M);
    }
    if (W.slots) W.slots[i] = s;
  }
  W.a1 = cv.take<float>(M * d);
  W.meanF = cv.take<float>(M);
  W.rstdF = cv.take<float>(M);
  W.resid = cv.take<float>((int64_t)(D.L + 1) * M * d);
  if (c.has_embed_head) {
    W.hf = cv.take<char>(M * d * es);
    W.meanf = cv.take<float>(M);
    W.rstdf = cv.take<float>(M);
    W.logits = cv.take<char>(M * D.Vp * es);
    W.dlogits = cv.take<char>(M * D.Vp * es);
    W.row_loss = cv.take<float>(M);
    W.keys = cv.take<int32_t>(embed_bwd_scratch((int)M));
  } else {
    W.hf = nullptr; W.meanf = W.rstdf = nullptr; W.logits = nullptr; W.dlogits = nullptr;
    W.row_loss = nullptr; W.keys = nullptr;
  }
  W.first = cv.take<char>(M * d * es);
  W.dfirst = cv.take<float>(M * d);
  W.dxa = cv.take<float>(M * d);
  W.dxb = cv.take<float>(M * d);
  W.dxm = cv.take<float>(M * d);
  W.da = cv.take<float>(M * d);
  W.dh1 = cv.take<float>(M * d);
  W.dh2 = cv.take<float>(M * d);
  W.dh2r[0] = W.dh2;
  for (int k = 1; k <= kSideGroup; ++k) W.dh2r[k] = c.arch == FAL_ARCH_FALPLUS ? cv.take<float>(M * d) : W.dh2;
  W.fp_part = c.arch == FAL_ARCH_FALPLUS ? cv.take<float>(falplus_side_scratch((int)M, (int)d)) : nullptr;
  W.lp_a = cv.take<char>(M * d * es);
  W.lp_b = cv.take<char>(M * d * es);
  W.dxm_lp = cv.take<char>(M * d * es);
  W.da_lp = cv.take<char>(M * d * es);
  for (int k = 0; k < 2; ++k) {
    W.dog2[k] = cv.take<char>(M * (int64_t)(D.dA + D.f) * es);
    W.dqkv2[k] = cv.take<char>(M * D.dqkv * es);
  }
  W.dog = W.dog2[0];
  W.dqkv = W.dqkv2[0];
  W.Dvec = cv.take<float>((int64_t)D.B * D.H * D.T);
  const int64_t part = std::max<int64_t>({ln_bwd_scratch((int)M, (int)d), dot_scratch(M * d)});
  W.part_main = cv.take<float>(part);
  W.part_aux = cv.take<float>(part);
  W.bias_part = cv.take<float>(col_sum_batch_scratch((int)M, (int)(2 * d + D.f + D.dqkv)));
  // a split is only chosen while fewer than 512 output tiles of 128x128
  // exist, so (512 + 512) tiles of partials bound every split decision
  W.splitk_floats = (int64_t)1024 * 128 * 128;
  W.splitk_main = cv.take<float>(W.splitk_floats);
  W.splitk_aux = cv.take<float>(W.splitk_floats);
  W.splitk_side = cv.take<float>(W.splitk_floats);
  W.loss_tmp = cv.take<float>(64);
  W.opt_part = cv.take<double>(kNormBlocks);
  W.opt_ctrl = cv.take<float>(16);
  *total = cv.off + kAlignBytes;
}

}  // namespace

// ------------------------------------------------------------- context --
struct ProfSpan {
  int cls;
  hipEvent_t a, b;
  double flops, bytes;
};

struct fal_ctx {
  fal_config_t cfg;
  Dims D;
  Layout Lo;
  Work W;
  char* ws;
  size_t ws_bytes;
  hipStream_t sm, sa;
  hipEvent_t ev_fork, ev_join, ev_keys;
  // library stream for a block's bias-gradient sums, which run beside the
  // next block's backward; forked from and joined back to the main stream
  hipStream_t sb = nullptr;
  hipEvent_t ev_bfork = nullptr, ev_bdone = nullptr, ev_hdone = nullptr;
  int device;
  std::string err;
  // kernel timing (fal_profile_enable)
  bool prof_on = false;
  std::vector<hipEvent_t> prof_pool;
  size_t prof_used = 0;
  std::vector<ProfSpan> prof_spans;
  int64_t prof_n[FAL_PROF_NCLASS] = {};
  double prof_ms[FAL_PROF_NCLASS] = {}, prof_flops[FAL_PROF_NCLASS] = {}, prof_bytes[FAL_PROF_NCLASS] = {};
};

namespace {

struct Fail {};

#define FAL_TRY(expr)                                                              \
  do {                                                                             \
    hipError_t _e = (expr);                                                        \
    if (_e != hipSuccess) {                                                        \
      ctx->err = std::string(#expr) + ": " + hipGetErrorString(_e);                \
      throw Fail{};                                                                \
    }                                                                              \
  } while (0)

// Brackets one launch with HIP events on the stream it runs on when kernel
// timing is enabled; a no-op otherwise.
struct Span {
  fal_ctx* c;
  hipStream_t s;
  int idx = -1;
  Span(fal_ctx* ctx, int cls, hipStream_t st, double flops, double bytes) : c(ctx), s(st) {
    if (!c->prof_on) return;
    if (c->prof_used + 2 > c->prof_pool.size()) {
      for (int i = 0; i < 256; ++i) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return;
        c->prof_pool.push_back(e);
      }
    }
    ProfSpan sp{cls, c->prof_pool[c->prof_used], c->prof_pool[c->prof_used + 1], flops, bytes};
    c->prof_used += 2;
    if (hipEventRecord(sp.a, s) != hipSuccess) return;
    idx = (int)c->prof_spans.size();
    c->prof_spans.push_back(sp);
  }
  ~Span() {
    if (idx >= 0) (void)hipEventRecord(c->prof_spans[idx].b, s);
  }
};

struct Run {
  fal_ctx* ctx;
  DType dt;
  int tanh;
  bool fwd_only = false;  // forward without a backward: GELU' is not kept
  explicit Run(fal_ctx* c) : ctx(c), dt(c->cfg.dtype == FAL_BF16 ? BF16 : F32), tanh(c->cfg.gelu_tanh) {}

  const char* P(const void* base, int k) const {
    return static_cast<const char*>(base) + ctx->Lo.boff[k] * (int64_t)ctx->D.es;
  }
  float* G(float* base, int k) const { return base + ctx->Lo.boff[k]; }
  char* off(void* p, int64_t elems) const { return static_cast<char*>(p) + elems * (int64_t)ctx->D.es; }

  void gemm_run(int ak, int bk, GemmGroup& g, hipStream_t s) {
    const char* why = nullptr;
    double flops = 0.0, bytes = 0.0;
    for (int i = 0; i < g.n; ++i) {
      const GemmProblem& q = g.p[i];
      flops += 2.0 * q.M * (double)q.N * (q.K + q.K2);
      bytes += (double)ctx->D.es * ((double)q.M * (q.K + q.K2) + (double)q.N * (q.K + q.K2)) +
               (double)q.M * q.N * ((q.out_f32 || q.epi == EPI_RESID) ? 4.0 : (double)ctx->D.es);
    }
    Span span(ctx, FAL_PROF_GEMM, s, flops, bytes);
    // split-K scratch: one region per stream, so that a launch makes the
    // same choice (and sums in the same order) on any of them
    const bool aux = s == ctx->sa && ctx->sa != ctx->sm;
    float* sk = s == ctx->sb ? ctx->W.splitk_side : aux ? ctx->W.splitk_aux : ctx->W.splitk_main;
    hipError_t e = fal::gemm(dt, ak, bk, g, tanh, s, &why, sk, ctx->W.splitk_floats);
    if (e != hipSuccess) {
      ctx->err = std::string("gemm: ") + (why ? why : hipGetErrorString(e));
      throw Fail{};
    }
  }

  static GemmProblem prob(const void* A, int64_t lda, const void* B, int64_t ldb, int M, int N, int K) {
    GemmProblem p;
    memset(&p, 0, sizeof(p));
    p.A = A; p.lda = lda; p.B = B; p.ldb = ldb; p.M = M; p.N = N; p.K = K;
    return p;
  }

  void gemm1(int ak, int bk, const GemmProblem& p, hipStream_t s) {
    GemmGroup g;
    memset(&g, 0, sizeof(g));
    g.p[0] = p;
    g.n = 1;
    gemm_run(ak, bk, g, s);
  }
  void gemm2(int ak, int bk, const GemmProblem& p, const GemmProblem& q, hipStream_t s) {
    GemmGroup g;
    memset(&g, 0, sizeof(g));
    g.p[0] = p;
    g.p[1] = q;
    g.n = 2;
    gemm_run(ak, bk, g, s);
  }

  // ----- forward pieces ----------------------------------------------------
  GemmProblem qkv_prob(const LayerSlot& S, const void* bp) {
    const Dims& D = ctx->D;
    GemmProblem p = prob(S.h1, D.d, P(bp, FAL_B_W_QKV), D.dqkv, D.M, D.dqkv, D.d);
    p.epi = EPI_STORE; p.bias = P(bp, FAL_B_B_QKV); p.out = S.qkv; p.ldo = D.dqkv;
    return p;
  }
  GemmProblem fc_prob(const LayerSlot& S, const void* bp) {
    const Dims& D = ctx->D;
    GemmProblem p = prob(S.h2, D.d, P(bp, FAL_B_W_FC), D.f, D.M, D.f, D.d);
    p.epi = EPI_GELU; p.bias = P(bp, FAL_B_B_FC);
    p.out = off(S.og, D.dA); p.ldo = D.dA + D.f;
    p.out2 = fwd_only ? nullptr : S.dgelu; p.ldo2 = D.f;
    return p;
  }
  // out-projection: A = O (first dA columns of og)
  GemmProblem oproj_prob(const LayerSlot& S, const void* bp) {
    const Dims& D = ctx->D;
    GemmProblem p = prob(S.og, D.dA + D.f, P(bp, FAL_B_W_O), D.d, D.M, D.d, D.dA);
    p.bias = P(bp, FAL_B_B_O);
    return p;
  }
  GemmProblem down_prob(const LayerSlot& S, const void* bp) {
    const Dims& D = ctx->D;
    GemmProblem p = prob(off(S.og, D.dA), D.dA + D.f, P(bp, FAL_B_W_2), D.d, D.M, D.d, D.f);
    p.bias = P(bp, FAL_B_B_2);
    return p;
  }
  int causal() const { return ctx->cfg.bidirectional ? 0 : 1; }
  // twice the keys each query sees on average: T + 1 causal, 2T unmasked
  double attn_keys2() const { return ctx->cfg.bidirectional ? 2.0 * ctx->D.T : ctx->D.T + 1.0; }
  void attention_fwd(const LayerSlot& S, hipStream_t s) {
    const Dims& D = ctx->D;
    const double fl = 2.0 * D.B * D.H * (double)D.hd * D.T * attn_keys2();
    Span span(ctx, FAL_PROF_ATTN_FWD, s, fl, (double)D.es * D.M * ((double)D.dqkv + D.dA));
    FAL_TRY(attn_fwd(dt, S.qkv, D.B, D.T, D.H, D.Hkv, D.hd, causal(), S.og, D.dA + D.f, S.lse, s));
  }
  void ln(const LnFwdArgs& a, hipStream_t s) {
    const double row = 4.0 + (double)ctx->D.es * (!!a.y1 + !!a.y2 + !!a.add2 + !!a.xhatF + !!a.xhat_out);
    Span span(ctx, FAL_PROF_NORM, s, 0.0, row * a.M * a.d);
    FAL_TRY(ln_fwd(dt, a, s));
  }
  void lnbwd(const LnBwdArgs& a, hipStream_t s) {
    // every buffer the previous block's pending bias sums read that is not
    // double-buffered (its output gradient, dXm / dA) is first written by a
    // LayerNorm backward of this block
    bias_join();
    const double row = 8.0 + 4.0 * (!!a.dy1 + !!a.dy2 + !!a.dres) + 8.0 * (!!a.dacc + !!a.dxhatF_acc) +
                       (double)ctx->D.es * (!!a.dx_lp + !!a.xhatF);
    Span span(ctx, FAL_PROF_NORM, s, 0.0, row * a.M * a.d);
    FAL_TRY(ln_bwd(dt, a, s));
  }
  LnFwdArgs lnargs(const float* x, float* mean, float* rstd) {
    LnFwdArgs a;
    memset(&a, 0, sizeof(a));
    a.x = x; a.M = ctx->D.M; a.d = ctx->D.d; a.eps = ctx->cfg.ln_eps; a.mean = mean; a.rstd = rstd;
    return a;
  }

  void fork() {
    FAL_TRY(hipEventRecord(ctx->ev_fork, ctx->sm));
    FAL_TRY(hipStreamWaitEvent(ctx->sa, ctx->ev_fork, 0));
  }
  void join() {
    FAL_TRY(hipEventRecord(ctx->ev_join, ctx->sa));
    FAL_TRY(hipStreamWaitEvent(ctx->sm, ctx->ev_join, 0));
  }
  bool streams() const {
    return (ctx->cfg.sched == FAL_SCHED_STREAMS || ctx->cfg.sched == FAL_SCHED_STREAMS_MERGED) &&
           ctx->sa != ctx->sm;
  }
  bool merged() const { return ctx->cfg.sched == FAL_SCHED_MERGED; }
  bool block1_standard() const { return ctx->cfg.fal_block1_mode == 1; }
  bool merged_out() const {
    return ctx->cfg.sched == FAL_SCHED_MERGED || ctx->cfg.sched == FAL_SCHED_STREAMS_MERGED;
  }

  // The block's weights were last read a whole step (or half of one) ago
  // and have left the caches; streaming them in first lets the block's
  // GEMMs find them in the last-level cache.  That pays where the GEMMs are
  // short against their weights' first-touch latency: measured gains with
  // 14 MiB of bf16 weights per block at 8192 tokens and with 75 MiB at
  // 4096; a wash at 24 MiB / 8192; losses of 0.5-0.8 ms per step at
  // 24 MiB / 16384 and 96 MiB / 8192, where the serial read costs more
  // than it saves.
  void warm_params(const void* bp, hipStream_t s) {
    const int64_t bytes = ctx->Lo.block_stride * (int64_t)ctx->D.es;
    if (bytes > (16ll << 20) && ctx->D.M > 4096) return;
    FAL_TRY(cache_warm(bp, bytes, s));
  }

  void block_fwd(int layer, const void* bp, const float* x, float* y, void* first) {
    const Dims& D = ctx->D;
    const LayerSlot& S = ctx->W.slots[layer];
    const int arch = ctx->cfg.arch;
    hipStream_t sm = ctx->sm;
    warm_params(bp, sm);
    // FAL blocks after the first and every parallel block: two independent
    // branches off the block input (the parallel block has no F term)
    if ((arch == FAL_ARCH_FAL && layer > 0) || arch == FAL_ARCH_PARALLEL) {
      LnFwdArgs a = lnargs(x, S.mean1, S.rstd1);
      a.g1 = P(bp, FAL_B_LN1_G); a.b1 = P(bp, FAL_B_LN1_B); a.y1 = S.h1;
      a.g2 = P(bp, FAL_B_LN2_G); a.b2 = P(bp, FAL_B_LN2_B); a.y2 = S.h2;
      a.add2 = arch == FAL_ARCH_FAL ? first : nullptr;
      ln(a, sm);
      if (merged()) {
        gemm2(1, 0, qkv_prob(S, bp), fc_prob(S, bp), sm);
        attention_fwd(S, sm);
        GemmProblem p = oproj_prob(S, bp);
        const GemmProblem q = down_prob(S, bp);
        p.A2 = q.A; p.lda2 = q.lda; p.B2 = q.B; p.ldb2 = q.ldb; p.K2 = q.K; p.bias2 = q.bias;
        p.epi = EPI_RESID; p.resid = x; p.ldr = D.d; p.out = y; p.ldo = D.d;
        gemm1(1, 0, p, sm);
        return;
      }
      // Two streams: when the QKV GEMM leaves compute units idle in its
      // last round, the MLP branch forks off before it and the FFN-up GEMM
      // fills them; when the QKV GEMM fills whole rounds, the FFN-up GEMM
      // goes after it and overlaps the attention kernel (whose causal tail
      // leaves compute units idle) instead of splitting the CUs with it.
      hipStream_t s2 = sm;
      const GemmProblem pq = qkv_prob(S, bp);
      bool fc_first = true;
      if (streams()) {
        GemmGroup gq;
        memset(&gq, 0, sizeof(gq));
        gq.p[0] = pq;
        gq.n = 1;
        fc_first = gemm_last_round_fill(dt, 1, 0, gq, 0) < 0.9;
      }
      if (!fc_first) gemm1(1, 0, pq, sm);
      if (streams()) { fork(); s2 = ctx->sa; }
      gemm1(1, 0, fc_prob(S, bp), s2);
      if (fc_first) gemm1(1, 0, pq, sm);
      attention_fwd(S, sm);
      if (merged_out()) {
        if (streams()) join();
        GemmProblem p = oproj_prob(S, bp);
        const GemmProblem q = down_prob(S, bp);
        p.A2 = q.A; p.lda2 = q.lda; p.B2 = q.B; p.ldb2 = q.ldb; p.K2 = q.K; p.bias2 = q.bias;
        p.epi = EPI_RESID; p.resid = x; p.ldr = D.d; p.out = y; p.ldo = D.d;
        gemm1(1, 0, p, sm);
        return;
      }
      GemmProblem po = oproj_prob(S, bp);
      po.epi = EPI_RESID; po.resid = x; po.ldr = D.d; po.out = y; po.ldo = D.d;
      gemm1(1, 0, po, sm);
      if (streams()) join();
      GemmProblem pd = down_prob(S, bp);
      pd.epi = EPI_RESID; pd.resid = y; pd.ldr = D.d; pd.out = y; pd.ldo = D.d;
      gemm1(1, 0, pd, sm);
      return;
    }
    // Sequential blocks: GPT, FAL+, and FAL block 0 (which, with
    // fal_block1_mode 1, is the standard block that only emits F).
    {
      LnFwdArgs a = lnargs(x, S.mean1, S.rstd1);
      a.g1 = P(bp, FAL_B_LN1_G); a.b1 = P(bp, FAL_B_LN1_B); a.y1 = S.h1;
      ln(a, sm);
    }
    gemm1(1, 0, qkv_prob(S, bp), sm);
    attention_fwd(S, sm);
    const bool block0_first = layer == 0 && arch != FAL_ARCH_GPT;
    GemmProblem po = oproj_prob(S, bp);
    if (block0_first) {
      po.epi = EPI_STORE; po.out_f32 = 1; po.out = ctx->W.a1; po.ldo = D.d;
      gemm1(1, 0, po, sm);
      FAL_TRY(add_f32(x, ctx->W.a1, S.xm, (int64_t)D.M * D.d, sm));
      LnFwdArgs a = lnargs(ctx->W.a1, ctx->W.meanF, ctx->W.rstdF);
      if (arch == FAL_ARCH_FAL) {
        a.g1 = P(bp, FAL_B_LNF1_G); a.b1 = P(bp, FAL_B_LNF1_B); a.y1 = first;
      } else {
        a.xhat_out = first;
      }
      ln(a, sm);
    } else {
      po.epi = EPI_RESID; po.resid = x; po.ldr = D.d; po.out = S.xm; po.ldo = D.d;
      gemm1(1, 0, po, sm);
    }
    if (arch == FAL_ARCH_FAL && !block1_standard()) {
      // block 0 of FAL (Eq. 2 at i = 1): H2 = LN2(X_1) + F
      LnFwdArgs a = lnargs(x, S.mean2, S.rstd2);
      a.g2 = P(bp, FAL_B_LN2_G); a.b2 = P(bp, FAL_B_LN2_B); a.y2 = S.h2; a.add2 = first;
      ln(a, sm);
    } else {
      LnFwdArgs a = lnargs(S.xm, S.mean2, S.rstd2);
      a.g2 = P(bp, FAL_B_LN2_G); a.b2 = P(bp, FAL_B_LN2_B); a.y2 = S.h2;
      if (arch == FAL_ARCH_FALPLUS && layer > 0) {
        a.xhatF = first; a.gF = P(bp, FAL_B_LNF1_G); a.bF = P(bp, FAL_B_LNF1_B);
      }
      ln(a, sm);
    }
    gemm1(1, 0, fc_prob(S, bp), sm);
    GemmProblem pd = down_prob(S, bp);
    pd.epi = EPI_RESID; pd.resid = S.xm; pd.ldr = D.d; pd.out = y; pd.ldo = D.d;
    gemm1(1, 0, pd, sm);
  }

  // ----- backward pieces ---------------------------------------------------
  // dgrad of a linear layer y = x W: dx = dy W^T with W stored [in, out]
  GemmProblem dgrad(const void* dy, int64_t lddy, const void* W, int in, int out, int M) {
    return prob(dy, lddy, W, out, M, in, out);
  }
  // wgrad: dW[in, out] = x^T dy
  GemmProblem wgrad(const void* x, int64_t ldx, const void* dy, int64_t lddy, int in, int out, int M,
                    float* dW) {
    GemmProblem p = prob(x, ldx, dy, lddy, in, out, M);
    p.epi = EPI_STORE; p.out_f32 = 1; p.out = dW; p.ldo = out;
    return p;
  }
  // Bias gradients are column sums of the layer's output gradient.  They are
  // queued while a block's backward runs and computed together at its end
  // (two launches per block); a second bias with the same gradient (b_o and
  // b_2 of a FAL block) shares the sum.
  ColSumBatch bias{};
  void colsum(const void* x, int in_f32, int64_t ld, int N, float* out, float*, hipStream_t) {
    for (int k = 0; k < bias.n; ++k) {
      ColSumInput& in = bias.in[k];
      if (in.x == x && in.ld == ld && in.N == N && !in.out2) { in.out2 = out; return; }
    }
    if (bias.n == kColSumMax) {
      bias_join();  // the partial-sum scratch is shared with the library stream
      flush_bias(ctx->sm);
    }
    bias.in[bias.n++] = ColSumInput{x, ld, N, in_f32 || dt == F32 ? 1 : 0, out, nullptr};
  }
  // The block's queued bias sums on the library stream (contexts given two
  // streams), after everything the main stream has issued so far (the
  // block is joined by then); they run beside the next block's backward.
  // Only sums over at least 128 MiB of gradients go there: same-box A/B,
  // per step, of 108-110 MiB per block (GPT-2 small, 7B shard) 0.16-0.3 ms
  // slower, of 144-287 MiB (GPT-2 medium, MLM-48, 1.3B) 0.1-2.0 ms faster.
  bool bias_pending = false;
  double bias_bytes() const {
    double bytes = 0.0;
    for (int k = 0; k < bias.n; ++k) bytes += (double)ctx->D.M * bias.in[k].N * (bias.in[k].f32 ? 4.0 : (double)ctx->D.es);
    return bytes;
  }
  // FAL+ blocks' first-attention terms of their LN2 backward, gathered over
  // up to kSideGroup consecutive blocks and queued like the bias sums: they
  // feed only the accumulator block 1 consumes and each block's own LN_F
  // gain gradient, so in a context given two streams a full group runs
  // beside the next block's backward (whatever the bias sums do).  A block
  // keeps its dH2 in ring slot layer % (kSideGroup + 1), which the next
  // kSideGroup blocks do not write.
  struct FpJob {
    FalPlusSide g;
    const void* xF;
    float* acc;
    int ow;
  } fp{};
  bool fp_ready = false;  // the group is complete (full, or block 1's)
  void run_fp(hipStream_t s) {
    const double es = ctx->D.es;
    const double bytes = (double)ctx->D.M * ctx->D.d * (4.0 * fp.g.n + es * (1 + fp.g.n) + (fp.ow ? 4.0 : 8.0));
    Span span(ctx, FAL_PROF_NORM, s, 0.0, bytes);
    FAL_TRY(falplus_side(dt, fp.g, fp.xF, fp.acc, fp.ow, ctx->D.M, ctx->D.d, ctx->W.fp_part, s));
    fp = FpJob{};
    fp_ready = false;
  }
  void queue_fp(const float* dy2, const void* xF, const void* gF, float* acc, int ow, float* dgF, bool close) {
    if (fp.g.n == kSideGroup || (fp.g.n > 0 && (xF != fp.xF || acc != fp.acc || ow))) {
      // a full group not yet flushed, or not one group
      bias_join();  // an earlier group may still be adding to an accumulator
      run_fp(ctx->sm);
    }
    if (fp.g.n == 0) { fp.xF = xF; fp.acc = acc; fp.ow = ow; }
    fp.g.dy2[fp.g.n] = dy2; fp.g.gF[fp.g.n] = gF; fp.g.dgF[fp.g.n] = dgF;
    ++fp.g.n;
    fp_ready = close || fp.g.n == kSideGroup;
  }
  // the end of an entry point: a group still open runs on the main stream
  void finish() {
    bias_join();
    if (fp.g.n > 0) run_fp(ctx->sm);
  }
  void flush_bias_async() {
    const bool two = ctx->sa != ctx->sm;  // one-stream contexts stay on one stream
    const bool bias_side = bias.n > 0 && two && bias_bytes() >= 128.0 * (1 << 20);
    const bool fp_side = fp_ready && two;
    if (bias.n > 0 && !bias_side) flush_bias(ctx->sm);
    if (fp_ready && !fp_side) run_fp(ctx->sm);
    if (!bias_side && !fp_side) return;
    FAL_TRY(hipEventRecord(ctx->ev_bfork, ctx->sm));
    FAL_TRY(hipStreamWaitEvent(ctx->sb, ctx->ev_bfork, 0));
    if (bias_side) flush_bias(ctx->sb);
    if (fp_side) run_fp(ctx->sb);
    FAL_TRY(hipEventRecord(ctx->ev_bdone, ctx->sb));
    bias_pending = true;
  }
  void bias_join() {
    if (!bias_pending) return;
    FAL_TRY(hipStreamWaitEvent(ctx->sm, ctx->ev_bdone, 0));
    bias_pending = false;
  }
  void flush_bias(hipStream_t s) {
    if (bias.n == 0) return;
    bias.M = ctx->D.M;
    Span span(ctx, FAL_PROF_BIAS, s, 0.0, bias_bytes());
    FAL_TRY(col_sum_batch(dt, bias, ctx->W.bias_part, s));
    bias = ColSumBatch{};
  }

  // MLP branch backward: from dM (lp copy, and fp32 for the bias) to dH2
  // (fp32, in W.dh2).  Writes W_2, B_2, W_FC, B_FC gradients.
  void mlp_bwd(const LayerSlot& S, const void* bp, const void* dy_lp, const float* dy, float* gb,
               hipStream_t s, float* part) {
    const Dims& D = ctx->D;
    Work& W = ctx->W;
    void* dP = off(W.dog, D.dA);
    GemmProblem pg = dgrad(dy_lp, D.d, P(bp, FAL_B_W_2), D.f, D.d, D.M);
    pg.epi = EPI_MUL_AUX; pg.aux = S.dgelu; pg.ldaux = D.f; pg.out = dP; pg.ldo = D.dA + D.f;
    gemm1(1, 1, pg, s);
    gemm1(0, 0, wgrad(off(S.og, D.dA), D.dA + D.f, dy_lp, D.d, D.f, D.d, D.M, G(gb, FAL_B_W_2)), s);
    colsum(dy, 1, D.d, D.d, G(gb, FAL_B_B_2), part, s);
    GemmProblem ph = dgrad(dP, D.dA + D.f, P(bp, FAL_B_W_FC), D.d, D.f, D.M);
    ph.epi = EPI_STORE; ph.out_f32 = 1; ph.out = W.dh2; ph.ldo = D.d;
    gemm1(1, 1, ph, s);
    gemm1(0, 0, wgrad(S.h2, D.d, dP, D.dA + D.f, D.d, D.f, D.M, G(gb, FAL_B_W_FC)), s);
    colsum(dP, 0, D.dA + D.f, D.f, G(gb, FAL_B_B_FC), part, s);
  }

  // MHA branch backward: from dA (lp + fp32) to dH1 (fp32, in W.dh1).
  void mha_bwd(const LayerSlot& S, const void* bp, const void* da_lp, const float* da, float* gb,
               hipStream_t s, float* part) {
    const Dims& D = ctx->D;
    Work& W = ctx->W;
    GemmProblem po = dgrad(da_lp, D.d, P(bp, FAL_B_W_O), D.dA, D.d, D.M);
    po.epi = EPI_STORE; po.out = W.dog; po.ldo = D.dA + D.f;
    gemm1(1, 1, po, s);
    gemm1(0, 0, wgrad(S.og, D.dA + D.f, da_lp, D.d, D.dA, D.d, D.M, G(gb, FAL_B_W_O)), s);
    colsum(da, 1, D.d, D.d, G(gb, FAL_B_B_O), part, s);
    {
      const double fl = 4.0 * D.B * D.H * (double)D.hd * D.T * attn_keys2();
      Span span(ctx, FAL_PROF_ATTN_BWD, s, fl, (double)D.es * D.M * (2.0 * D.dqkv + 2.0 * D.dA));
      FAL_TRY(attn_bwd(dt, S.qkv, S.og, D.dA + D.f, W.dog, D.dA + D.f, S.lse, D.B, D.T, D.H, D.Hkv, D.hd,
                       causal(), W.dqkv, W.Dvec, nullptr, s));
    }
    GemmProblem ph = dgrad(W.dqkv, D.dqkv, P(bp, FAL_B_W_QKV), D.d, D.dqkv, D.M);
    ph.epi = EPI_STORE; ph.out_f32 = 1; ph.out = W.dh1; ph.ldo = D.d;
    gemm1(1, 1, ph, s);
    gemm1(0, 0, wgrad(S.h1, D.d, W.dqkv, D.dqkv, D.d, D.dqkv, D.M, G(gb, FAL_B_W_QKV)), s);
    colsum(W.dqkv, 0, D.dqkv, D.dqkv, G(gb, FAL_B_B_QKV), part, s);
  }

  LnBwdArgs lnb(const float* x, const float* mean, const float* rstd) {
    LnBwdArgs a;
    memset(&a, 0, sizeof(a));
    a.x = x; a.mean = mean; a.rstd = rstd; a.M = ctx->D.M; a.d = ctx->D.d;
    a.partials = ctx->W.part_main;
    return a;
  }

  // dy: fp32 gradient of the block output; dy_lp: its dtype copy.  first:
  // the first-attention tensor the forward read (FAL+: the normalisation of
  // A_1, whose product with dH2 gives the block's LN_{F,i} gain gradient).
  void block_bwd(int layer, const void* bp, const float* x, const void* first, const float* dy,
                 const void* dy_lp, float* dx, void* dx_lp, float* dfirst, float* gb) {
    ctx->W.dog = ctx->W.dog2[layer & 1];
    ctx->W.dh2 = ctx->W.dh2r[layer % (kSideGroup + 1)];
    ctx->W.dqkv = ctx->W.dqkv2[layer & 1];
    block_bwd_parts(layer, bp, x, first, dy, dy_lp, dx, dx_lp, dfirst, gb);
    // after the join: the aux stream's gradients are complete
    flush_bias_async();
  }
  void block_bwd_parts(int layer, const void* bp, const float* x, const void* first, const float* dy,
                       const void* dy_lp, float* dx, void* dx_lp, float* dfirst, float* gb) {
    const Dims& D = ctx->D;
    Work& W = ctx->W;
    const LayerSlot& S = W.slots[layer];
    const int arch = ctx->cfg.arch;
    hipStream_t sm = ctx->sm;
    const int64_t Md = (int64_t)D.M * D.d;
    const bool last = layer == D.L - 1;
    warm_params(bp, sm);
    // first-attention LayerNorm slot: zero unless used by this block
    const bool uses_lnF = (arch == FAL_ARCH_FAL && layer == 0 && (!block1_standard() || D.L > 1)) ||
                          (arch == FAL_ARCH_FALPLUS && layer > 0);
    if (!uses_lnF) {
      // both slots in one launch (the alignment padding between them is zero too)
      const int64_t n = ctx->Lo.boff[FAL_B_LNF1_B] + D.d - ctx->Lo.boff[FAL_B_LNF1_G];
      FAL_TRY(zero_f32(G(gb, FAL_B_LNF1_G), n, sm));
    }
    if ((arch == FAL_ARCH_FAL && layer > 0) || arch == FAL_ARCH_PARALLEL) {
      hipStream_t s2 = sm;
      float* part2 = W.part_main;
      if (streams()) { fork(); s2 = ctx->sa; part2 = W.part_aux; }
      mlp_bwd(S, bp, dy_lp, dy, gb, s2, part2);
      mha_bwd(S, bp, dy_lp, dy, gb, sm, W.part_main);
      if (streams()) join();
      LnBwdArgs a = lnb(x, S.mean1, S.rstd1);
      a.dy1 = W.dh1; a.g1 = P(bp, FAL_B_LN1_G); a.dy2 = W.dh2; a.g2 = P(bp, FAL_B_LN2_G);
      a.dres = dy; a.dx = dx; a.dx_lp = dx_lp;
      if (arch == FAL_ARCH_FAL) { a.dacc = dfirst; a.dacc_overwrite = last; }
      a.dg1 = G(gb, FAL_B_LN1_G); a.db1 = G(gb, FAL_B_LN1_B);
      a.dg2 = G(gb, FAL_B_LN2_G); a.db2 = G(gb, FAL_B_LN2_B);
      lnbwd(a, sm);
      return;
    }
    if (arch == FAL_ARCH_FAL && !block1_standard()) {  // block 0, Eq. 2
      mlp_bwd(S, bp, dy_lp, dy, gb, sm, W.part_main);
      if (last) FAL_TRY(copy_f32(dfirst, W.dh2, Md, sm));
      else FAL_TRY(add_f32(dfirst, W.dh2, dfirst, Md, sm));
      // dA_1 = dY + LN_F backward of the accumulated dF
      LnBwdArgs f = lnb(W.a1, W.meanF, W.rstdF);
      f.dy1 = dfirst; f.g1 = P(bp, FAL_B_LNF1_G); f.dres = dy; f.dx = W.da; f.dx_lp = W.da_lp;
      f.dg1 = G(gb, FAL_B_LNF1_G); f.db1 = G(gb, FAL_B_LNF1_B);
      lnbwd(f, sm);
      mha_bwd(S, bp, W.da_lp, W.da, gb, sm, W.part_main);
      // LN2 was applied to X_1 with its own statistics (mean2/rstd2 equal
      // mean1/rstd1 up to rounding; use each LayerNorm's own).
      LnBwdArgs a2 = lnb(x, S.mean2, S.rstd2);
      a2.dy2 = W.dh2; a2.g2 = P(bp, FAL_B_LN2_G); a2.dres = dy; a2.dx = dx;
      a2.dg2 = G(gb, FAL_B_LN2_G); a2.db2 = G(gb, FAL_B_LN2_B);
      lnbwd(a2, sm);
      LnBwdArgs a1 = lnb(x, S.mean1, S.rstd1);
      a1.dy1 = W.dh1; a1.g1 = P(bp, FAL_B_LN1_G); a1.dres = dx; a1.dx = dx; a1.dx_lp = dx_lp;
      a1.dg1 = G(gb, FAL_B_LN1_G); a1.db1 = G(gb, FAL_B_LN1_B);
      lnbwd(a1, sm);
      return;
    }
    // GPT and FAL+: MLP backward, LN2 backward (with the FAL+ first-attention
    // term), MHA backward, LN1 backward.
    mlp_bwd(S, bp, dy_lp, dy, gb, sm, W.part_main);
    LnBwdArgs a2 = lnb(S.xm, S.mean2, S.rstd2);
    a2.dy2 = W.dh2; a2.g2 = P(bp, FAL_B_LN2_G); a2.dres = dy; a2.dx = W.dxm; a2.dx_lp = W.dxm_lp;
    a2.dg2 = G(gb, FAL_B_LN2_G); a2.db2 = G(gb, FAL_B_LN2_B);
    if (arch == FAL_ARCH_FALPLUS && layer > 0) {
      a2.dbF = G(gb, FAL_B_LNF1_B);  // = db2, from the same partial sums
      if (W.fp_part && falplus_side_ok(dt, D.d, W.dh2, first, P(bp, FAL_B_LNF1_G), dfirst)) {
        queue_fp(W.dh2, first, P(bp, FAL_B_LNF1_G), dfirst, last ? 1 : 0, G(gb, FAL_B_LNF1_G), layer == 1);
      } else {
        if (fp.g.n > 0) {  // keep the accumulator's order of terms
          bias_join();
          run_fp(sm);
        }
        a2.xhatF = first; a2.gF = P(bp, FAL_B_LNF1_G);
        a2.dxhatF_acc = dfirst; a2.dxhatF_overwrite = last;
        a2.dgF = G(gb, FAL_B_LNF1_G);
      }
    }
    lnbwd(a2, sm);
    const void* da_lp = W.dxm_lp;
    const float* da = W.dxm;
    if (arch == FAL_ARCH_FALPLUS && layer == 0 && D.L > 1) {
      // dA_1 = dXm + backward of norm(A_1) applied to the accumulated
      // dxhatF, with its dtype copy, in one pass
      {
        Span span(ctx, FAL_PROF_NORM, sm, 0.0, (16.0 + (double)ctx->D.es) * Md);
        FAL_TRY(norm_bwd(dt, W.a1, W.meanF, W.rstdF, dfirst, D.M, D.d, W.dxm, W.da, W.da_lp, sm));
      }
      da_lp = W.da_lp;
      da = W.da;
    }
    if (arch == FAL_ARCH_FAL && layer == 0 && D.L > 1) {
      // standard block 1 of FAL: dA_1 = dXm + LN_F backward of the dF the
      // later blocks accumulated (which also gives the LN_F gradients)
      LnBwdArgs f = lnb(W.a1, W.meanF, W.rstdF);
      f.dy1 = dfirst; f.g1 = P(bp, FAL_B_LNF1_G); f.dres = W.dxm; f.dx = W.da; f.dx_lp = W.da_lp;
      f.dg1 = G(gb, FAL_B_LNF1_G); f.db1 = G(gb, FAL_B_LNF1_B);
      lnbwd(f, sm);
      da_lp = W.da_lp;
      da = W.da;
    }
    mha_bwd(S, bp, da_lp, da, gb, sm, W.part_main);
    LnBwdArgs a1 = lnb(x, S.mean1, S.rstd1);
    a1.dy1 = W.dh1; a1.g1 = P(bp, FAL_B_LN1_G); a1.dres = W.dxm; a1.dx = dx; a1.dx_lp = dx_lp;
    a1.dg1 = G(gb, FAL_B_LN1_G); a1.db1 = G(gb, FAL_B_LN1_B);
    lnbwd(a1, sm);
  }
};

}  // namespace

// ================================================================ ABI ====
extern "C" {

const char* fal_status_string(fal_status_t s) {
  switch (s) {
    case FAL_OK: return "ok";
    case FAL_ERR_INVALID_ARG: return "invalid argument";
    case FAL_ERR_UNSUPPORTED: return "unsupported";
    case FAL_ERR_WORKSPACE: return "workspace too small";
    case FAL_ERR_HIP: return "HIP error";
    case FAL_ERR_STATE: return "bad call order";
  }
  return "unknown status";
}

// Message of the last failed call made without a context on this thread.
static thread_local std::string g_noctx_err;

const char* fal_last_error(const fal_ctx_t* ctx) { return ctx ? ctx->err.c_str() : g_noctx_err.c_str(); }

fal_status_t fal_validate_config(const fal_config_t* cfg) {
  const char* why = validate(cfg);
  if (!why) why = validate_hd(cfg);
  if (!why) why = validate_extent(cfg);
  if (!why) return FAL_OK;
  return unsupported(why) ? FAL_ERR_UNSUPPORTED : FAL_ERR_INVALID_ARG;
}

fal_status_t fal_param_layout(const fal_config_t* cfg, int64_t* global_off, int64_t* block_off,
                              int64_t* block_base, int64_t* block_stride, int64_t* total) {
  fal_status_t st = fal_validate_config(cfg);
  if (st != FAL_OK) return st;
  const Layout Lo = layout_of(*cfg);
  if (global_off) memcpy(global_off, Lo.goff, sizeof(Lo.goff));
  if (block_off) memcpy(block_off, Lo.boff, sizeof(Lo.boff));
  if (block_base) *block_base = Lo.block_base;
  if (block_stride) *block_stride = Lo.block_stride;
  if (total) *total = Lo.total;
  return FAL_OK;
}

fal_status_t fal_workspace_bytes(const fal_config_t* cfg, size_t* bytes) {
  fal_status_t st = fal_validate_config(cfg);
  if (st != FAL_OK) return st;
  if (!bytes) return FAL_ERR_INVALID_ARG;
  Work W;
  carve(*cfg, nullptr, W, bytes);
  return FAL_OK;
}

fal_status_t fal_init(const fal_config_t* cfg, void* workspace, size_t ws_bytes, void* stream_main,
                      void* stream_aux, fal_ctx_t** out) {
  if (!out) return FAL_ERR_INVALID_ARG;
  *out = nullptr;
  fal_status_t st = fal_validate_config(cfg);
  if (st != FAL_OK) return st;
  size_t need = 0;
  {
    Work W;
    carve(*cfg, nullptr, W, &need);
  }
  if (!workspace || ws_bytes < need) return FAL_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlignBytes) return FAL_ERR_WORKSPACE;
  fal_ctx* ctx = new (std::nothrow) fal_ctx();
  if (!ctx) return FAL_ERR_INVALID_ARG;
  ctx->cfg = *cfg;
  ctx->D = dims_of(*cfg);
  ctx->Lo = layout_of(*cfg);
  ctx->ws = static_cast<char*>(workspace);
  ctx->ws_bytes = ws_bytes;
  ctx->sm = static_cast<hipStream_t>(stream_main);
  ctx->sa = stream_aux ? static_cast<hipStream_t>(stream_aux) : ctx->sm;
  ctx->W.slots = new (std::nothrow) LayerSlot[cfg->n_layer];
  if (!ctx->W.slots) { delete ctx; return FAL_ERR_INVALID_ARG; }
  size_t total = 0;
  carve(*cfg, ctx->ws, ctx->W, &total);
  if (hipGetDevice(&ctx->device) != hipSuccess ||
      hipEventCreateWithFlags(&ctx->ev_fork, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&ctx->ev_join, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&ctx->ev_keys, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&ctx->ev_bfork, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&ctx->ev_bdone, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&ctx->ev_hdone, hipEventDisableTiming) != hipSuccess ||
      hipStreamCreateWithFlags(&ctx->sb, hipStreamNonBlocking) != hipSuccess) {
    delete[] ctx->W.slots;
    delete ctx;
    return FAL_ERR_HIP;
  }
  *out = ctx;
  return FAL_OK;
}

fal_status_t fal_destroy(fal_ctx_t* ctx) {
  if (!ctx) return FAL_ERR_INVALID_ARG;
  for (hipEvent_t e : ctx->prof_pool) (void)hipEventDestroy(e);
  (void)hipEventDestroy(ctx->ev_fork);
  (void)hipEventDestroy(ctx->ev_join);
  (void)hipEventDestroy(ctx->ev_keys);
  if (ctx->ev_bfork) (void)hipEventDestroy(ctx->ev_bfork);
  if (ctx->ev_bdone) (void)hipEventDestroy(ctx->ev_bdone);
  if (ctx->ev_hdone) (void)hipEventDestroy(ctx->ev_hdone);
  if (ctx->sb) (void)hipStreamDestroy(ctx->sb);
  delete[] ctx->W.slots;
  delete ctx;
  return FAL_OK;
}

static fal_status_t check_ctx(fal_ctx_t* ctx) {
  if (!ctx) return FAL_ERR_INVALID_ARG;
  ctx->err.clear();
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != ctx->device) {
    ctx->err = "context used on a different HIP device than the one it was created on";
    return FAL_ERR_STATE;
  }
  return FAL_OK;
}

static fal_status_t bad(fal_ctx_t* ctx, const char* why) {
  ctx->err = why;
  return FAL_ERR_INVALID_ARG;
}

fal_status_t fal_block_fwd(fal_ctx_t* ctx, int32_t layer, const void* block_params, const float* x_in,
                           float* x_out, void* first_attn) {
  fal_status_t st = check_ctx(ctx);
  if (st != FAL_OK) return st;
  if (layer < 0 || layer >= ctx->D.L) return bad(ctx, "layer out of range");
  if (!block_params || !x_in || !x_out) return bad(ctx, "NULL block_params, x_in or x_out");
  if (x_in == x_out) return bad(ctx, "x_out may not alias x_in");
  const bool uses_first = ctx->cfg.arch == FAL_ARCH_FAL || ctx->cfg.arch == FAL_ARCH_FALPLUS;
  if (uses_first && !first_attn) return bad(ctx, "first_attn is required for FAL and FAL+");
  try {
    Run r(ctx);
    r.block_fwd(layer, block_params, x_in, x_out, first_attn);
  } catch (Fail&) {
    return FAL_ERR_HIP;
  }
  return FAL_OK;
}

fal_status_t fal_block_bwd(fal_ctx_t* ctx, int32_t layer, const void* block_params, const float* x_in,
                           const void* first_attn, const float* dx_out, float* dx_in, float* d_first_attn,
                           float* block_grads) {
  fal_status_t st = check_ctx(ctx);
  if (st != FAL_OK) return st;
  if (layer < 0 || layer >= ctx->D.L) return bad(ctx, "layer out of range");
  if (!block_params || !x_in || !dx_out || !dx_in || !block_grads)
    return bad(ctx, "NULL block_params, x_in, dx_out, dx_in or block_grads");
  if (dx_in == dx_out) return bad(ctx, "dx_in may not alias dx_out");
  const bool uses_first = ctx->cfg.arch == FAL_ARCH_FAL || ctx->cfg.arch == FAL_ARCH_FALPLUS;
  if (uses_first && !d_first_attn) return bad(ctx, "d_first_attn is required for FAL and FAL+");
  if (ctx->cfg.arch == FAL_ARCH_FALPLUS && !first_attn)
    return bad(ctx, "first_attn (the normalised first attention output) is required for FAL+");
  try {
    Run r(ctx);
    const int64_t Md = (int64_t)ctx->D.M * ctx->D.d;
    FAL_TRY(cast_from_f32(r.dt, dx_out, ctx->W.lp_a, Md, ctx->sm));
    r.block_bwd(layer, block_params, x_in, first_attn, dx_out, ctx->W.lp_a, dx_in, ctx->W.lp_b, d_first_attn,
                block_grads);
    r.finish();
  } catch (Fail&) {
    return FAL_ERR_HIP;
  }
  return FAL_OK;
}

fal_status_t fal_model_step(fal_ctx_t* ctx, const void* params, const int32_t* tokens, float* loss,
                            float* logits, float* grads) {
  fal_status_t st = check_ctx(ctx);
  if (st != FAL_OK) return st;
  if (!ctx->cfg.has_embed_head) return bad(ctx, "fal_model_step needs has_embed_head = 1 (use fal_stack_step)");
  if (!params || !tokens || !loss || !grads) return bad(ctx, "NULL params, tokens, loss or grads");
  const Dims& D = ctx->D;
  const Layout& Lo = ctx->Lo;
  Work& W = ctx->W;
  hipStream_t sm = ctx->sm;
  const int64_t Md = (int64_t)D.M * D.d;
  const char* pb = static_cast<const char*>(params);
  auto gparam = [&](int k) { return pb + Lo.goff[k] * (int64_t)D.es; };
  auto bparam = [&](int i) { return pb + (Lo.block_base + (int64_t)i * Lo.block_stride) * (int64_t)D.es; };
  auto bgrad = [&](int i) { return grads + Lo.block_base + (int64_t)i * Lo.block_stride; };
  try {
    Run r(ctx);
    // The embedding backward's (id, position) sort depends on the tokens
    // only: it runs on the aux stream beside the forward pass, and the
    // scatter at the end of the step waits for it.
    {
      hipStream_t sk = ctx->sa;
      if (sk != sm) r.fork();
      Span span(ctx, FAL_PROF_EMBED, sk, 0.0, (double)D.M * 8.0);
      FAL_TRY(embed_sort(tokens, D.B, D.T, D.V, W.keys, sk));
    }
    FAL_TRY(hipEventRecord(ctx->ev_keys, ctx->sa));
    {
      Span span(ctx, FAL_PROF_EMBED, sm, 0.0, (double)D.M * D.d * (2.0 * D.es + 4.0));
      FAL_TRY(embed_fwd(r.dt, tokens, D.B, D.T, D.V, D.d, gparam(FAL_P_WTE), gparam(FAL_P_WPE), W.resid, sm));
    }
    for (int i = 0; i < D.L; ++i) r.block_fwd(i, bparam(i), W.resid + i * Md, W.resid + (i + 1) * Md, W.first);
    const float* xl = W.resid + (int64_t)D.L * Md;
    {
      LnFwdArgs a = r.lnargs(xl, W.meanf, W.rstdf);
      a.g1 = gparam(FAL_P_LNF_G); a.b1 = gparam(FAL_P_LNF_B); a.y1 = W.hf;
      r.ln(a, sm);
    }
    GemmProblem ph = Run::prob(W.hf, D.d, gparam(FAL_P_WTE), D.d, D.M, D.V, D.d);
    // logits in the step's dtype (the LM-head product's precision); the
    // cross-entropy works in fp32 from them
    ph.epi = EPI_STORE; ph.out_f32 = r.dt == F32; ph.out = W.logits; ph.ldo = D.Vp;
    r.gemm1(1, 1, ph, sm);
    {
      Span span(ctx, FAL_PROF_CE, sm, 0.0, (double)D.M * (double)D.es * (D.V + D.Vp));
      FAL_TRY(cross_entropy(r.dt, W.logits, D.Vp, tokens, D.B, D.T, D.V, W.dlogits, D.Vp, W.row_loss, loss, sm));
    }
    if (logits) FAL_TRY(rows_to_f32(r.dt, W.logits, D.Vp, logits, D.V, D.M, D.V, sm));
    // head backward: dHf = dlogits wte ; dwte = dlogits^T Hf
    GemmProblem pd = Run::prob(W.dlogits, D.Vp, gparam(FAL_P_WTE), D.d, D.M, D.d, D.V);
    pd.epi = EPI_STORE; pd.out_f32 = 1; pd.out = W.dh1; pd.ldo = D.d;
    pd.kpad = 1;  // dlogits columns V .. Vp-1 are written as zeros
    r.gemm1(1, 0, pd, sm);
    // dwte = dlogits^T Hf beside the final LayerNorm and the last blocks'
    // backward (two-stream contexts): nothing reads dwte before the
    // embedding backward adds to it, and dlogits and Hf stay untouched
    const GemmProblem pw = r.wgrad(W.dlogits, D.Vp, W.hf, D.d, D.V, D.d, D.M, grads + Lo.goff[FAL_P_WTE]);
    const bool side = ctx->sa != ctx->sm;
    if (side) {
      FAL_TRY(hipEventRecord(ctx->ev_bfork, sm));
      FAL_TRY(hipStreamWaitEvent(ctx->sb, ctx->ev_bfork, 0));
      r.gemm1(0, 0, pw, ctx->sb);
      FAL_TRY(hipEventRecord(ctx->ev_hdone, ctx->sb));
    } else {
      r.gemm1(0, 0, pw, sm);
    }
    {
      LnBwdArgs a = r.lnb(xl, W.meanf, W.rstdf);
      a.dy1 = W.dh1; a.g1 = gparam(FAL_P_LNF_G); a.dx = W.dxa; a.dx_lp = W.lp_a;
      a.dg1 = grads + Lo.goff[FAL_P_LNF_G]; a.db1 = grads + Lo.goff[FAL_P_LNF_B];
      r.lnbwd(a, sm);
    }
    float *cur = W.dxa, *nxt = W.dxb;
    void *cur_lp = W.lp_a, *nxt_lp = W.lp_b;
    for (int i = D.L - 1; i >= 0; --i) {
      r.block_bwd(i, bparam(i), W.resid + i * Md, W.first, cur, cur_lp, nxt, nxt_lp, W.dfirst, bgrad(i));
      std::swap(cur, nxt);
      std::swap(cur_lp, nxt_lp);
    }
    r.finish();
    if (side) FAL_TRY(hipStreamWaitEvent(sm, ctx->ev_hdone, 0));
    {
      // dX read twice (position sums, scatter), touched wte-gradient rows read and written
      Span span(ctx, FAL_PROF_EMBED, sm, 0.0, (double)D.M * D.d * 16.0);
      FAL_TRY(hipStreamWaitEvent(sm, ctx->ev_keys, 0));
      FAL_TRY(embed_bwd(D.B, D.T, D.d, cur, grads + Lo.goff[FAL_P_WTE], grads + Lo.goff[FAL_P_WPE], W.keys, W.dh1,
                        sm));
    }
  } catch (Fail&) {
    return FAL_ERR_HIP;
  }
  return FAL_OK;
}

fal_status_t fal_model_forward(fal_ctx_t* ctx, const void* params, const int32_t* tokens, float* loss,
                               float* logits) {
  fal_status_t st = check_ctx(ctx);
  if (st != FAL_OK) return st;
  if (!ctx->cfg.has_embed_head) return bad(ctx, "fal_model_forward needs has_embed_head = 1 (use fal_stack_forward)");
  if (!params || !tokens) return bad(ctx, "NULL params or tokens");
  const Dims& D = ctx->D;
  const Layout& Lo = ctx->Lo;
  Work& W = ctx->W;
  hipStream_t sm = ctx->sm;
  const int64_t Md = (int64_t)D.M * D.d;
  const char* pb = static_cast<const char*>(params);
  auto gparam = [&](int k) { return pb + Lo.goff[k] * (int64_t)D.es; };
  auto bparam = [&](int i) { return pb + (Lo.block_base + (int64_t)i * Lo.block_stride) * (int64_t)D.es; };
  try {
    Run r(ctx);
    r.fwd_only = true;
    {
      Span span(ctx, FAL_PROF_EMBED, sm, 0.0, (double)D.M * D.d * (2.0 * D.es + 4.0));
      FAL_TRY(embed_fwd(r.dt, tokens, D.B, D.T, D.V, D.d, gparam(FAL_P_WTE), gparam(FAL_P_WPE), W.resid, sm));
    }
    for (int i = 0; i < D.L; ++i) r.block_fwd(i, bparam(i), W.resid + i * Md, W.resid + (i + 1) * Md, W.first);
    const float* xl = W.resid + (int64_t)D.L * Md;
    {
      LnFwdArgs a = r.lnargs(xl, W.meanf, W.rstdf);
      a.g1 = gparam(FAL_P_LNF_G); a.b1 = gparam(FAL_P_LNF_B); a.y1 = W.hf;
      r.ln(a, sm);
    }
    GemmProblem ph = Run::prob(W.hf, D.d, gparam(FAL_P_WTE), D.d, D.M, D.V, D.d);
    ph.epi = EPI_STORE; ph.out_f32 = r.dt == F32; ph.out = W.logits; ph.ldo = D.Vp;
    r.gemm1(1, 1, ph, sm);
    if (loss) {
      Span span(ctx, FAL_PROF_CE, sm, 0.0, (double)D.M * (double)D.es * D.V);
      FAL_TRY(cross_entropy(r.dt, W.logits, D.Vp, tokens, D.B, D.T, D.V, nullptr, D.Vp, W.row_loss, loss, sm));
    }
    if (logits) FAL_TRY(rows_to_f32(r.dt, W.logits, D.Vp, logits, D.V, D.M, D.V, sm));
  } catch (Fail&) {
    return FAL_ERR_HIP;
  }
  return FAL_OK;
}

fal_status_t fal_stack_forward(fal_ctx_t* ctx, const void* params, const float* x_in, float* x_out) {
  fal_status_t st = check_ctx(ctx);
  if (st != FAL_OK) return st;
  if (ctx->cfg.has_embed_head) return bad(ctx, "fal_stack_forward needs has_embed_head = 0");
  if (!params || !x_in) return bad(ctx, "NULL params or x_in");
  const Dims& D = ctx->D;
  const Layout& Lo = ctx->Lo;
  Work& W = ctx->W;
  const int64_t Md = (int64_t)D.M * D.d;
  if (x_out && x_out == x_in) return bad(ctx, "x_out may not alias x_in");
  const char* pb = static_cast<const char*>(params);
  auto bparam = [&](int i) { return pb + (Lo.block_base + (int64_t)i * Lo.block_stride) * (int64_t)D.es; };
  auto xin = [&](int i) { return i == 0 ? x_in : W.resid + i * Md; };
  try {
    Run r(ctx);
    r.fwd_only = true;
    for (int i = 0; i < D.L; ++i) r.block_fwd(i, bparam(i), xin(i), W.resid + (i + 1) * Md, W.first);
    if (x_out)
      FAL_TRY(copy_f32(x_out, W.resid + (int64_t)D.L * Md, Md, ctx->sm));
  } catch (Fail&) {
    return FAL_ERR_HIP;
  }
  return FAL_OK;
}

fal_status_t fal_stack_step(fal_ctx_t* ctx, const void* params, const float* x_in, const float* dy,
                            float* loss, float* grads, float* dx_in) {
  fal_status_t st = check_ctx(ctx);
  if (st != FAL_OK) return st;
  if (ctx->cfg.has_embed_head) return bad(ctx, "fal_stack_step needs has_embed_head = 0");
  if (!params || !x_in || !dy || !grads) return bad(ctx, "NULL params, x_in, dy or grads");
  const Dims& D = ctx->D;
  const Layout& Lo = ctx->Lo;
  Work& W = ctx->W;
  hipStream_t sm = ctx->sm;
  const int64_t Md = (int64_t)D.M * D.d;
  const char* pb = static_cast<const char*>(params);
  auto bparam = [&](int i) { return pb + (Lo.block_base + (int64_t)i * Lo.block_stride) * (int64_t)D.es; };
  auto bgrad = [&](int i) { return grads + Lo.block_base + (int64_t)i * Lo.block_stride; };
  auto xin = [&](int i) { return i == 0 ? x_in : W.resid + i * Md; };
  try {
    Run r(ctx);
    for (int i = 0; i < D.L; ++i) r.block_fwd(i, bparam(i), xin(i), W.resid + (i + 1) * Md, W.first);
    const float* xl = W.resid + (int64_t)D.L * Md;
    if (loss) FAL_TRY(dot(dy, xl, Md, loss, W.part_main, sm));
    FAL_TRY(cast_from_f32(r.dt, dy, W.lp_a, Md, sm));
    const float* cur = dy;
    float* bufs[2] = {W.dxa, W.dxb};
    void* lps[2] = {W.lp_a, W.lp_b};
    int k = 0;
    for (int i = D.L - 1; i >= 0; --i) {
      float* out = (i == 0 && dx_in) ? dx_in : bufs[k];
      r.block_bwd(i, bparam(i), xin(i), W.first, cur, lps[k], out, lps[k ^ 1], W.dfirst, bgrad(i));
      cur = out;
      k ^= 1;
    }
    r.finish();
  } catch (Fail&) {
    return FAL_ERR_HIP;
  }
  return FAL_OK;
}

static bool overlaps(const void* a, int64_t abytes, const void* b, int64_t bbytes) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + (uintptr_t)bbytes && y < x + (uintptr_t)abytes;
}

// Host checks shared by both AdamW entry points; on success fills the
// kernel constants and the dtype-copy mode (0 none, 1 fp32, 2 bf16).
static const char* adamw_args(const fal_adamw_t* hp, int64_t step, int64_t n, bool bf, float* master,
                              void* params, const float* grads, float* m, float* v, float* norm_out,
                              AdamwConsts* k, int* lp_mode_out) {
  if (!hp) return "NULL hyper-parameters";
  if (step < 1) return "step is 1-based";
  if (n < 0) return "negative element count";
  auto finite = [](float x) { return std::isfinite(x); };
  if (!finite(hp->lr) || !finite(hp->beta1) || !finite(hp->beta2) || !finite(hp->eps) ||
      !finite(hp->weight_decay) || !finite(hp->max_grad_norm))
    return "non-finite hyper-parameter";
  if (hp->lr < 0.f || hp->eps < 0.f || hp->weight_decay < 0.f) return "lr, eps and weight_decay must be >= 0";
  if (!(hp->beta1 >= 0.f && hp->beta1 < 1.f && hp->beta2 >= 0.f && hp->beta2 < 1.f))
    return "beta1 and beta2 must lie in [0, 1)";
  if (n > kAdamwMaxElems) return "element count above the update kernel's grid limit";
  if (n > 0 && (!master || !grads || !m || !v)) return "NULL master, grads, m or v";
  if (bf && n > 0 && !params) return "params (bf16 copy) is required for a bf16 config";
  const int lp_mode = (!params || params == master) ? 0 : (bf ? 2 : 1);
  if (bf && lp_mode == 0 && n > 0) return "params may not alias master for a bf16 config";
  auto al = [](const void* p, uintptr_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; };
  if (!al(master, 16) || !al(grads, 16) || !al(m, 16) || !al(v, 16) ||
      (lp_mode != 0 && !al(params, lp_mode == 2 ? 8 : 16)))
    return "fp32 arrays must be 16-byte aligned, params 8-byte (bf16) or 16-byte (fp32)";
  if (norm_out && !al(norm_out, 4)) return "grad_norm must be 4-byte aligned";
  const int64_t b4 = n * 4;
  const void* arr[5] = {master, grads, m, v, params};
  const int64_t len[5] = {b4, b4, b4, b4, lp_mode == 0 ? 0 : n * (lp_mode == 2 ? 2 : 4)};
  for (int i = 0; i < 5; ++i)
    for (int j = i + 1; j < 5; ++j)
      if (len[i] > 0 && len[j] > 0 && overlaps(arr[i], len[i], arr[j], len[j]))
        return "master, grads, m, v and params may not overlap";
  if (norm_out && n > 0)
    for (int i = 0; i < 5; ++i)
      if (len[i] > 0 && overlaps(norm_out, 4, arr[i], len[i])) return "grad_norm overlaps an array";
  // bias corrections and step size in double on the host
  const double bc1 = 1.0 - std::pow((double)hp->beta1, (double)step);
  const double bc2 = 1.0 - std::pow((double)hp->beta2, (double)step);
  if (!(bc1 > 0.0) || !(bc2 > 0.0)) return "bias correction underflows (beta too close to 1 for step)";
  k->beta1 = hp->beta1;
  k->one_minus_beta1 = (float)(1.0 - (double)hp->beta1);
  k->beta2 = hp->beta2;
  k->one_minus_beta2 = (float)(1.0 - (double)hp->beta2);
  k->eps = hp->eps;
  k->rsqrt_bc2 = (float)(1.0 / std::sqrt(bc2));
  k->step_size = (float)((double)hp->lr / bc1);
  k->decay = (float)(1.0 - (double)hp->lr * hp->weight_decay);
  *lp_mode_out = lp_mode;
  return nullptr;
}

fal_status_t fal_adamw_step(fal_ctx_t* ctx, const fal_adamw_t* hp, int64_t step, int64_t n, float* master,
                            void* params, const float* grads, float* m, float* v, float* norm_out) {
  fal_status_t st = check_ctx(ctx);
  if (st != FAL_OK) return st;
  AdamwConsts k;
  int lp_mode = 0;
  const char* why = adamw_args(hp, step, n, ctx->cfg.dtype == FAL_BF16, master, params, grads, m, v, norm_out, &k,
                               &lp_mode);
  if (why) return bad(ctx, why);
  hipStream_t sm = ctx->sm;
  try {
    const double bytes = 4.0 * n + (double)n * (28.0 + (lp_mode == 2 ? 2.0 : lp_mode == 1 ? 4.0 : 0.0));
    Span span(ctx, FAL_PROF_OPTIM, sm, 0.0, bytes);
    FAL_TRY(grad_norm(grads, n, hp->max_grad_norm, ctx->W.opt_part, ctx->W.opt_ctrl, norm_out, sm));
    FAL_TRY(adamw_update(lp_mode, master, params, grads, m, v, n, k, ctx->W.opt_ctrl, sm));
  } catch (Fail&) {
    return FAL_ERR_HIP;
  }
  return FAL_OK;
}

fal_status_t fal_adamw_step_noalloc(const fal_adamw_t* hp, int64_t step, int64_t n, int32_t dtype, float* master,
                                    void* params, const float* grads, float* m, float* v, float* norm_out,
                                    void* stream) {
  g_noctx_err.clear();
  if (dtype != FAL_F32 && dtype != FAL_BF16) {
    g_noctx_err = "unknown dtype";
    return FAL_ERR_INVALID_ARG;
  }
  AdamwConsts k;
  int lp_mode = 0;
  const char* why = adamw_args(hp, step, n, dtype == FAL_BF16, master, params, grads, m, v, norm_out, &k, &lp_mode);
  if (why) {
    g_noctx_err = why;
    return FAL_ERR_INVALID_ARG;
  }
  const hipError_t e = adamw_static_scratch(lp_mode, master, params, grads, m, v, n, hp->max_grad_norm, k, norm_out,
                                            static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    g_noctx_err = std::string("fal_adamw_step_noalloc: ") + hipGetErrorString(e);
    return FAL_ERR_HIP;
  }
  return FAL_OK;
}

fal_status_t fal_profile_enable(fal_ctx_t* ctx, int32_t enable) {
  fal_status_t st = check_ctx(ctx);
  if (st != FAL_OK) return st;
  if (hipStreamSynchronize(ctx->sm) != hipSuccess || hipStreamSynchronize(ctx->sa) != hipSuccess) {
    ctx->err = "stream synchronisation failed";
    return FAL_ERR_HIP;
  }
  ctx->prof_on = enable != 0;
  ctx->prof_spans.clear();
  ctx->prof_used = 0;
  for (int k = 0; k < FAL_PROF_NCLASS; ++k) {
    ctx->prof_n[k] = 0; ctx->prof_ms[k] = ctx->prof_flops[k] = ctx->prof_bytes[k] = 0.0;
  }
  while (enable && ctx->prof_pool.size() < 4096) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) { ctx->err = "hipEventCreate failed"; return FAL_ERR_HIP; }
    ctx->prof_pool.push_back(e);
  }
  return FAL_OK;
}

fal_status_t fal_profile_read(fal_ctx_t* ctx, int32_t cls, int64_t* launches, double* total_ms,
                              double* flops, double* bytes) {
  fal_status_t st = check_ctx(ctx);
  if (st != FAL_OK) return st;
  if (cls < 0 || cls >= FAL_PROF_NCLASS) return bad(ctx, "unknown profile class");
  if (!ctx->prof_spans.empty()) {
    if (hipStreamSynchronize(ctx->sm) != hipSuccess || hipStreamSynchronize(ctx->sa) != hipSuccess) {
      ctx->err = "stream synchronisation failed";
      return FAL_ERR_HIP;
    }
    for (const ProfSpan& sp : ctx->prof_spans) {
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, sp.a, sp.b) != hipSuccess) { ctx->err = "hipEventElapsedTime failed"; return FAL_ERR_HIP; }
      ctx->prof_n[sp.cls] += 1;
      ctx->prof_ms[sp.cls] += ms;
      ctx->prof_flops[sp.cls] += sp.flops;
      ctx->prof_bytes[sp.cls] += sp.bytes;
    }
    ctx->prof_spans.clear();
    ctx->prof_used = 0;
  }
  if (launches) *launches = ctx->prof_n[cls];
  if (total_ms) *total_ms = ctx->prof_ms[cls];
  if (flops) *flops = ctx->prof_flops[cls];
  if (bytes) *bytes = ctx->prof_bytes[cls];
  return FAL_OK;
}

fal_status_t fal_residual_out(fal_ctx_t* ctx, const float** x_last) {
  if (!ctx || !x_last) return FAL_ERR_INVALID_ARG;
  *x_last = ctx->W.resid + (int64_t)ctx->D.L * ctx->D.M * ctx->D.d;
  return FAL_OK;
}

}  // extern "C"
