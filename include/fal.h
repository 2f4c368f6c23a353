/*
 * fal.h -- C ABI of libfal.so: one training step (forward + backward) of a
 * GPT-style Pre-LN decoder stack in four block architectures, the forward
 * pass alone, and the AdamW update that follows a step, on one MI355X
 * (gfx950):
 *
 *   GPT   (Sec. 2, Eq. 1)  X_{i+1} = X_i + MHA_i(LN(X_i))
 *                                   + MLP_i(LN(X_i + MHA_i(LN(X_i))))
 *   FAL   (Sec. 4.1, Eq. 2) X_{i+1} = X_i + MHA_i(LN(X_i))
 *                                   + MLP_i(LN(X_i) + LN(MHA_1(LN(X_1))))
 *         The first-attention LayerNorm F = LN_F(MHA_1(LN(X_1))) is evaluated
 *         once, in block 0, and read by every block (Sec. 4.1).
 *   FAL+  (Sec. 5; Appendix D) block 0 is the GPT block; every later block
 *         adds its own LayerNorm of the first attention output to the GPT
 *         MLP input: MLP_i(LN(X_i + A_i) + LN_{F,i}(MHA_1(LN(X_1)))).
 *   PARALLEL (the configuration Sec. 6.1 and 6.4 compare against, after
 *         GPT-J and PaLM) MHA and MLP read the same block input, each
 *         through its own LayerNorm:
 *         X_{i+1} = X_i + MHA_i(LN1(X_i)) + MLP_i(LN2(X_i)).
 *         Scheduled like the FAL blocks (two independent branches).
 *
 * MHA = QKV projection, scaled-dot-product attention per head (causal; no
 * mask for encoder stacks; optionally grouped-query with shared key/value
 * heads), concatenation, output projection; MLP = up-projection, GELU (tanh
 * form by default), down-projection (Sec. 2).  Biases on every linear layer, learned
 * position embedding, final LayerNorm and an LM head tied to the token
 * embedding (GPT-2 conventions).
 *
 * Conventions shared by every entry point
 *  - All pointers marked "device" are HIP device pointers allocated by the
 *    caller; the library never allocates device memory.  The caller owns
 *    every buffer (parameters, gradients, tokens, outputs, workspace).
 *  - Tensors are dense, row-major.  Activations are token-major [M, d] with
 *    M = batch * seq_len (row m = b * seq_len + t).  Linear weights are stored
 *    [in, out] so a layer computes y = x W + b.
 *  - Parameters are stored in the config's dtype (fp32, or bf16); the
 *    residual stream (x_in, x_out, dx_*) and every gradient are fp32.
 *  - Work is enqueued asynchronously on the main stream given to fal_init.
 *    With the STREAMS schedule the library forks work onto the aux stream
 *    and joins back onto the main stream before the call returns.
 *  - Errors: every call validates its arguments on the host before any
 *    launch and returns a status; no call aborts.  The message of the last
 *    failure is available from fal_last_error.  A context is used from one
 *    host thread at a time.
 *  - Results are deterministic: the same inputs give bitwise-identical
 *    outputs run to run, and the SEQ and STREAMS schedules agree bitwise.
 */
#ifndef FAL_H
#define FAL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FAL_OK = 0,
  FAL_ERR_INVALID_ARG = 1, /* NULL pointer, bad size, bad enum value      */
  FAL_ERR_UNSUPPORTED = 2, /* valid but not implemented (e.g. head_dim)   */
  FAL_ERR_WORKSPACE = 3,   /* workspace NULL or smaller than required     */
  FAL_ERR_HIP = 4,         /* a HIP runtime call or kernel launch failed  */
  FAL_ERR_STATE = 5        /* call out of order (e.g. bwd before fwd)     */
} fal_status_t;

typedef enum { FAL_ARCH_GPT = 0, FAL_ARCH_FAL = 1, FAL_ARCH_FALPLUS = 2, FAL_ARCH_PARALLEL = 3 } fal_arch_t;
typedef enum { FAL_F32 = 0, FAL_BF16 = 1 } fal_dtype_t;

/* How the two branches of a FAL block are issued (Sec. 4.2: in FAL a block's
 * MHA and MLP have no dependency and may run concurrently).  Parallel blocks
 * are issued the same way.
 *  SEQ     : one stream, branches back to back.
 *  STREAMS : MHA branch on the main stream, MLP branch on the aux stream,
 *            joined with HIP events (same kernels as SEQ).
 *  MERGED  : the independent GEMMs of the two branches are issued as one
 *            grouped launch, and FAL's output projection and down-projection
 *            as one GEMM over the concatenated inner dimension.
 *  STREAMS_MERGED : the branches on two streams as in STREAMS (forward:
 *            QKV and attention on main, FFN-up on aux; backward: the MHA and
 *            MLP chains), and after the join the output and down
 *            projections as one GEMM over the concatenated inner dimension.
 * GPT and FAL+ blocks have no independent branches; the schedule only
 * affects FAL and parallel blocks. */
typedef enum {
  FAL_SCHED_SEQ = 0, FAL_SCHED_STREAMS = 1, FAL_SCHED_MERGED = 2, FAL_SCHED_STREAMS_MERGED = 3
} fal_sched_t;

typedef struct {
  int32_t n_layer;        /* L >= 1                                           */
  int32_t d_model;        /* d, multiple of 8                                 */
  int32_t n_head;         /* heads held on this GPU                           */
  int32_t head_dim;       /* 16, 32, 64 or 128                                */
  int32_t d_ff;           /* FFN width f, multiple of 8                       */
  int32_t vocab;          /* V (ignored when has_embed_head == 0)             */
  int32_t seq_len;        /* T                                                */
  int32_t batch;          /* B                                                */
  int32_t arch;           /* fal_arch_t                                       */
  int32_t dtype;          /* fal_dtype_t of parameters and saved activations  */
  int32_t sched;          /* fal_sched_t                                      */
  float ln_eps;           /* LayerNorm epsilon (GPT-2: 1e-5)                  */
  int32_t gelu_tanh;      /* 1: tanh-approximate GELU, 0: erf GELU            */
  int32_t has_embed_head; /* 1: embedding + final LN + tied head + CE loss;
                             0: block stack only (fal_stack_step)             */
  int32_t fal_block1_mode; /* FAL only (0 for GPT and FAL+).  0: block 1 applies
                             Eq. 2 like every later block, MLP_1(LN2(X_1) + F);
                             1: block 1 is the standard Pre-LN block (Eq. 1) and
                             only produces F = LN_F(A_1) for blocks >= 2 (the
                             "preparation stage" reading of Sec. 4.1).  Any
                             other value, or 1 with another arch, is
                             FAL_ERR_INVALID_ARG.                             */
  int32_t bidirectional;  /* 0: causal attention (query t sees keys 0..t);
                             1: no mask, every query sees every key of its
                             sequence: the encoder blocks of the paper's
                             masked-language-model depth study (Sec. 6.4,
                             after Cramming).  1 requires has_embed_head = 0
                             (the MLM head and loss are not part of this
                             library).                                       */
  int32_t n_kv_head;      /* key/value heads: 0 (or n_head) is multi-head
                             attention; a divisor of n_head gives grouped-
                             query attention, query head h reading key/value
                             head h / (n_head / n_kv_head) (Appendix E.1
                             evaluates two groups).                          */
} fal_config_t;

/* Parameter tensors.  Global tensors (present only when has_embed_head):
 *   WTE [V, d], WPE [T, d], LNF_G [d], LNF_B [d].
 * Per-block tensors, identical layout in every block (dA = n_head*head_dim,
 * dKV = n_kv_head*head_dim, dKV = dA without grouped-query attention):
 *   LN1_G [d] LN1_B [d] W_QKV [d, dA+2dKV] B_QKV [dA+2dKV] W_O [dA, d] B_O [d]
 *   LN2_G [d] LN2_B [d] W_FC [d, f] B_FC [f] W_2 [f, d] B_2 [d]
 *   LNF1_G [d] LNF1_B [d]   first-attention LayerNorm: used by block 0 in FAL
 *                           (the single LN_F) and by blocks >= 1 in FAL+
 *                           (LN_{F,i}); unused slots (GPT, parallel) get
 *                           zero gradients.
 * W_QKV's columns are [Q | K | V], each head h at columns h*head_dim of its
 * part (Q: n_head heads, K and V: n_kv_head heads each). */
enum {
  FAL_P_WTE = 0, FAL_P_WPE, FAL_P_LNF_G, FAL_P_LNF_B, FAL_P_NGLOBAL
};
enum {
  FAL_B_LN1_G = 0, FAL_B_LN1_B, FAL_B_W_QKV, FAL_B_B_QKV, FAL_B_W_O, FAL_B_B_O,
  FAL_B_LN2_G, FAL_B_LN2_B, FAL_B_W_FC, FAL_B_B_FC, FAL_B_W_2, FAL_B_B_2,
  FAL_B_LNF1_G, FAL_B_LNF1_B, FAL_B_NTENSOR
};

typedef struct fal_ctx fal_ctx_t; /* opaque */

/* Host only; no GPU needed.  FAL_OK if the config is valid and supported. */
fal_status_t fal_validate_config(const fal_config_t* cfg);

/* Host only.  Element offsets of the parameter tensors inside one flat
 * parameter buffer (the gradient buffer has the same layout, in fp32).
 *   global_off[FAL_P_NGLOBAL]  offsets of the global tensors (-1 if absent)
 *   block_off[FAL_B_NTENSOR]   offsets inside one block, relative to the
 *                              block's start
 *   block_base, block_stride   block i starts at block_base + i*block_stride
 *   total                      number of elements of the whole buffer
 * Every tensor starts at a multiple of 64 elements.  Any output pointer may
 * be NULL. */
fal_status_t fal_param_layout(const fal_config_t* cfg, int64_t* global_off, int64_t* block_off,
                              int64_t* block_base, int64_t* block_stride, int64_t* total);

/* Host only.  Bytes of device workspace fal_init needs for this config:
 * saved activations of every block, the residual stream, the LM-head
 * logits and the backward scratch. */
fal_status_t fal_workspace_bytes(const fal_config_t* cfg, size_t* bytes);

/* Creates a context bound to the current HIP device.  workspace: device
 * buffer of at least fal_workspace_bytes bytes, 256-byte aligned, owned by
 * the caller and kept alive until fal_destroy.  stream_main / stream_aux:
 * hipStream_t handles (NULL means the default stream; aux may equal main).
 * The context also creates one stream of its own (default priority): when
 * aux differs from main, the LM-head weight gradient and large blocks'
 * bias-gradient sums run there beside the following backward work; every
 * call joins it back into the main stream before it returns.  *out
 * receives the context. */
fal_status_t fal_init(const fal_config_t* cfg, void* workspace, size_t ws_bytes,
                      void* stream_main, void* stream_aux, fal_ctx_t** out);

fal_status_t fal_destroy(fal_ctx_t* ctx);

/* Forward of block `layer` (0-based): X_{i+1} from X_i for i = layer + 1.
 * Defines: GPT, the Pre-LN block of Sec. 2 (Eq. 1); FAL, the block output of
 * Sec. 4.1 (Eq. 2) with the first-attention LayerNorm applied once, in the
 * first block (Sec. 4.1 and its footnote); FAL+, the block equation of
 * Appendix D (Ablation study, "FAL+"): the first block is the GPT block,
 * every later block adds its own LayerNorm of the first attention output to
 * the MLP input; PARALLEL, the shared-input block Sec. 6.1 compares against.
 *   block_params  device, dtype, one block in the FAL_B_* layout
 *   x_in, x_out   device fp32 [M, d]; x_out = block output (may not alias x_in)
 *   first_attn    device dtype [M, d], caller-owned for the whole step.
 *                 FAL: block 0 writes F = LN_F(A_1) (A_1 = MHA_1(LN(X_1))),
 *                 later blocks read it.  FAL+: block 0 writes the shared
 *                 normalisation (A_1 - mean) * rstd of A_1, later blocks read
 *                 it and apply their own gain and shift.  GPT and parallel:
 *                 ignored (may be NULL).  Required (non-NULL) for FAL, FAL+.
 * Saves the activations block `layer`'s backward needs in the workspace
 * (block 0 of FAL / FAL+ also keeps A_1 and its LayerNorm statistics there).
 * Blocks must run in order 0 .. L-1 within a step.  Errors:
 * FAL_ERR_INVALID_ARG for a layer out of range, a NULL or aliased pointer. */
fal_status_t fal_block_fwd(fal_ctx_t* ctx, int32_t layer, const void* block_params,
                           const float* x_in, float* x_out, void* first_attn);

/* Backward of block `layer`; requires fal_block_fwd(layer) of the same step
 * (and, for block 0 of FAL / FAL+, the A_1 it saved).  The gradient of the
 * block equation named at fal_block_fwd; for FAL the first-attention term
 * receives dF = sum over blocks of dH2_i, and block 0 turns it into the
 * gradient of A_1 through LN_F's backward.  For FAL+ the per-block terms
 * gamma_{F,i} * xhat + beta_{F,i} share one normalisation xhat of A_1, and the
 * normalisation's backward is linear in its input gradient, so blocks >= 1
 * accumulate d(xhat) = sum gamma_{F,i} * dH2_i and block 0 applies one
 * normalisation backward to the sum.
 *   x_in          device fp32 [M, d], the same input given to the forward
 *   first_attn    device dtype [M, d], the tensor block 0's forward wrote
 *                 (FAL+: read for the gradient of gamma_{F,i}; FAL: unused,
 *                 may be NULL; GPT and parallel: ignored)
 *   dx_out        device fp32 [M, d], gradient w.r.t. the block output
 *   dx_in         device fp32 [M, d], receives the gradient w.r.t. x_in
 *                 (may not alias dx_out)
 *   d_first_attn  device fp32 [M, d] accumulator of the gradient w.r.t. the
 *                 first-attention tensor (FAL: F; FAL+: the normalisation).
 *                 Blocks run in order L-1 .. 0: block L-1 overwrites it,
 *                 blocks below accumulate into it, block 0 consumes it.
 *                 GPT and parallel: ignored (may be NULL).
 *   block_grads   device fp32, one block in the FAL_B_* layout, overwritten
 *                 (unused LN_F slots are written as zeros) */
fal_status_t fal_block_bwd(fal_ctx_t* ctx, int32_t layer, const void* block_params,
                           const float* x_in, const void* first_attn, const float* dx_out,
                           float* dx_in, float* d_first_attn, float* block_grads);

/* One whole training step of the language model (has_embed_head == 1):
 * embedding, the block stack of the config's architecture (the equations
 * named at fal_block_fwd), final LayerNorm, LM head tied to the token
 * embedding, mean next-token cross-entropy (the GPT-2 language-modelling
 * setup of Sec. 6.1), then the backward of all of it.
 *   params  device, dtype, full layout of fal_param_layout
 *   tokens  device int32 [B, T+1]; the model reads [:, :T] and predicts
 *           [:, 1:]; ids must lie in [0, V) (out-of-range ids are clamped)
 *   loss    device fp32 scalar: mean next-token cross-entropy over B*T
 *   logits  device fp32 [B*T, V] or NULL to skip writing them; the step
 *           keeps the logits in the config's dtype (bf16 in bf16 mode, the
 *           precision of the LM-head product) and widens them here
 *   grads   device fp32, full layout, overwritten
 * Errors: FAL_ERR_INVALID_ARG for NULL pointers or has_embed_head == 0. */
fal_status_t fal_model_step(fal_ctx_t* ctx, const void* params, const int32_t* tokens,
                            float* loss, float* logits, float* grads);

/* One training step of a block stack without embedding or head
 * (has_embed_head == 0; one GPU's share of a tensor-parallel model, Sec. 4.2
 * and Appendix B): forward of every block from x_in (the equations named at
 * fal_block_fwd), surrogate loss sum(dy * X_L) so the gradient entering the
 * last block is dy, backward.
 *   x_in   device fp32 [M, d]      dy   device fp32 [M, d]
 *   loss   device fp32 scalar or NULL
 *   grads  device fp32, full layout, overwritten
 *   dx_in  device fp32 [M, d] or NULL: gradient w.r.t. x_in
 * Errors: FAL_ERR_INVALID_ARG for NULL pointers or has_embed_head == 1. */
fal_status_t fal_stack_step(fal_ctx_t* ctx, const void* params, const float* x_in,
                            const float* dy, float* loss, float* grads, float* dx_in);

/* Optimizer hyper-parameters.  The paper's training setups (appendix) use
 * learning rate 1e-4, weight decay 0.001 and gradient clipping to global
 * norm 1 with an Adam-type optimizer; beta1 0.9, beta2 0.999, eps 1e-8 are
 * the usual AdamW defaults. */
typedef struct {
  float lr;            /* learning rate, >= 0                                 */
  float beta1, beta2;  /* moment decay rates, in [0, 1)                       */
  float eps;           /* added to sqrt of the second moment, >= 0            */
  float weight_decay;  /* decoupled: p <- p (1 - lr weight_decay), >= 0       */
  float max_grad_norm; /* clip threshold on the global L2 norm; <= 0: no clip */
} fal_adamw_t;

/* One AdamW update of a flat parameter buffer (the optimizer of the paper's
 * training setups, appendix), after clipping the gradient to a global norm:
 *   c = min(1, max_grad_norm / (||grads||_2 + 1e-6))   (1 without clipping)
 *   g = c grads;  m = beta1 m + (1 - beta1) g;  v = beta2 v + (1 - beta2) g^2
 *   master = master (1 - lr weight_decay)
 *            - lr / (1 - beta1^step) * m / (sqrt(v / (1 - beta2^step)) + eps)
 * applied to every element (alignment padding included: its gradient is
 * zero when the caller zero-filled the gradient buffer once, so it only
 * decays).  The norm is the square root of a fixed-order fp64 sum, so the
 * update is deterministic.
 *   step     1-based index of this update (bias corrections use beta^step)
 *   n        number of elements (normally `total` of fal_param_layout), >= 0
 *   master   device fp32 [n], the fp32 weights, updated in place
 *   params   device, config dtype [n]: receives master rounded to the dtype
 *            (bf16: round to nearest even) for the next step.  fp32 configs:
 *            NULL or equal to master when master is the parameter buffer.
 *   grads    device fp32 [n], read only (e.g. from fal_model_step)
 *   m, v     device fp32 [n] first and second moments, zero before step 1,
 *            updated in place
 *   grad_norm device fp32 scalar or NULL: the norm before clipping
 * fp32 arrays must be 16-byte aligned and params 8-byte (bf16) or 16-byte
 * (fp32) aligned; the arrays may not overlap (except params == master).
 * Non-finite gradients are not skipped: they reach the weights.  Enqueued
 * on the main stream; uses a few KB of the context's workspace. */
fal_status_t fal_adamw_step(fal_ctx_t* ctx, const fal_adamw_t* hp, int64_t step, int64_t n,
                            float* master, void* params, const float* grads, float* m, float* v,
                            float* grad_norm);

/* The AdamW update of fal_adamw_step without a context and without any
 * device allocation, for callers that cannot allocate device memory or
 * create a context: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same kernels in the same order as
 * fal_adamw_step, so the results are bitwise identical.  Its scratch (the
 * 2048 fp64 partial sums of the norm pass and the {norm, clip factor}
 * control block: 16 KiB + 256 B) is a fixed array in the library's device
 * memory, one per GPU, held until the process ends; its size does not
 * depend on n.  Every call rewrites that scratch before reading it, so
 * nothing needs clearing, but calls that overlap on one GPU (two streams or
 * two host threads) share it and race: the caller must serialise them.
 *   dtype   fal_dtype_t of params (FAL_BF16: bf16 copy of master; FAL_F32:
 *           fp32 copy, or NULL / master for an in-place update)
 *   stream  hipStream_t the work is enqueued on (NULL: the default stream)
 *   other arguments as for fal_adamw_step.
 * Errors: FAL_ERR_INVALID_ARG for the argument errors of fal_adamw_step, an
 * unknown dtype, or n above the update's limit of (2^31 - 1) * 2048
 * elements; FAL_ERR_HIP when a HIP call fails.  fal_last_error(NULL) returns
 * the message of the last failed call of this kind on the calling thread. */
fal_status_t fal_adamw_step_noalloc(const fal_adamw_t* hp, int64_t step, int64_t n, int32_t dtype,
                                    float* master, void* params, const float* grads, float* m, float* v,
                                    float* grad_norm, void* stream);

/* Forward pass only, without gradients (the paper's inference measurement,
 * Appendix D.3, times this forward step as the time to first token).
 * Same kernels and schedule as the forward half of fal_model_step; the GELU
 * derivative the backward would need is not written.
 *   params  device, dtype, full layout      tokens  device int32 [B, T+1]
 *   loss    device fp32 scalar or NULL: mean next-token cross-entropy
 *           (targets tokens[:, 1:]), bitwise equal to fal_model_step's
 *   logits  device fp32 [B*T, V] or NULL (widened from the dtype logits)
 * has_embed_head must be 1. */
fal_status_t fal_model_forward(fal_ctx_t* ctx, const void* params, const int32_t* tokens,
                               float* loss, float* logits);

/* Forward of the block stack only (has_embed_head == 0).
 *   x_in   device fp32 [M, d]
 *   x_out  device fp32 [M, d] or NULL; receives X_L (also readable through
 *          fal_residual_out); may not alias x_in */
fal_status_t fal_stack_forward(fal_ctx_t* ctx, const void* params, const float* x_in, float* x_out);

/* Device pointer to the final block output X_L (fp32 [M, d]) held in the
 * workspace after a step; valid until the next step. */
fal_status_t fal_residual_out(fal_ctx_t* ctx, const float** x_last);

/* Kernel timing, for measurement.  While enabled, each launch of the
 * classes below is bracketed by HIP events recorded on the stream the
 * kernel runs on; fal_profile_read synchronises the context's streams and
 * returns, per class since the last enable: the number of launches, the
 * summed event time in ms, and the summed algorithmic FLOPs and bytes of
 * those launches (GEMM: 2*M*N*K; attention forward: 2*B*H*hd*T*(T+1), the
 * causal half of QK^T and PV; attention backward: twice that; norm: bytes
 * of the rows read and written; cross-entropy: logits read and dlogits
 * written; embedding: rows gathered and written forward, the position-
 * gradient and scatter traffic backward; bias gradients: the column sums'
 * input; optimizer: the gradient read by the norm pass plus every array
 * the update reads and writes).  fal_profile_enable(ctx, 0) turns timing off; either call clears
 * the counters.  Host memory only; no device allocation. */
typedef enum {
  FAL_PROF_GEMM = 0, FAL_PROF_ATTN_FWD = 1, FAL_PROF_ATTN_BWD = 2, FAL_PROF_NORM = 3,
  FAL_PROF_CE = 4, FAL_PROF_EMBED = 5, FAL_PROF_BIAS = 6, FAL_PROF_OPTIM = 7,
  FAL_PROF_NCLASS = 8
} fal_prof_class_t;
fal_status_t fal_profile_enable(fal_ctx_t* ctx, int32_t enable);
fal_status_t fal_profile_read(fal_ctx_t* ctx, int32_t cls, int64_t* launches, double* total_ms,
                              double* flops, double* bytes);

const char* fal_status_string(fal_status_t status);
/* "" if none.  ctx NULL: the message of the last failed context-free call
 * (fal_adamw_step_noalloc) on the calling thread. */
const char* fal_last_error(const fal_ctx_t* ctx);

#ifdef __cplusplus
}
#endif
#endif /* FAL_H */
