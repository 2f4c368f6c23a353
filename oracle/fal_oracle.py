"""CPU fp64 oracle of one training step of a GPT / FAL / FAL+ decoder stack.

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow, obviously correct
definition that the GPU library is checked against.  Only the tests, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
product path never does.  It shares no code with the HIP library: every
function below is written from the paper's equations with numpy in float64.

What is computed (paper notation; X_i is the input of block i, 1-based in
the paper and 0-based here):

* Pre-LN GPT block (Sec. 2, Eq. 1):
      X_{i+1} = X_i + MHA_i(LN(X_i)) + MLP_i(LN(X_i + MHA_i(LN(X_i))))
* FAL block (Sec. 4.1, Eq. 2), applied to every block including the first:
      X_{i+1} = X_i + MHA_i(LN(X_i)) + MLP_i(LN(X_i) + LN(MHA_1(LN(X_1))))
  The LayerNorm of the first attention output is evaluated once, in the
  first block, and its result F is reused by every block (Sec. 4.1 and its
  footnote on repositioning the first layer's LN).
* FAL+ block (Sec. 5; Appendix D, FAL+ equation): block 1 is the standard
  block; every later block adds a per-block LayerNorm of the first attention
  output to its usual MLP input:
      X_{i+1} = X_i + MHA_i(LN(X_i))
                + MLP_i(LN(X_i + MHA_i(LN(X_i))) + LN(MHA_1(LN(X_1))))
* Parallel block (the configuration Sec. 6.1 and Sec. 6.4 compare against,
  after GPT-J and PaLM): MHA and MLP read the same block input, each through its own
  LayerNorm:
      X_{i+1} = X_i + MHA_i(LN1(X_i)) + MLP_i(LN2(X_i))

Readings taken where the paper is silent (each listed in the design notes):
  - the "LN(X_i)" at the MLP input is the block's own second LayerNorm
    (LN2_i), applied to X_i instead of X_i + A_i;
  - FAL uses one first-attention LayerNorm (its parameters live in block 0's
    lnF slot); FAL+ uses one per later block (block i's lnF slot) over one
    shared normalisation of A_1;
  - FAL block 1 applies Eq. 2 like every other block (fal_block1_mode 0);
    fal_block1_mode 1 keeps block 1 the standard block, which then only
    produces F = LN_F(A_1) for the later blocks (the "preparation stage"
    reading of Sec. 4.1);
  - FAL+ block 1 is the standard GPT block (the printed first case has a
    misplaced parenthesis);
  - the parallel block keeps GPT-2's two LayerNorms (LN1 before MHA, LN2
    before the MLP), both applied to X_i;
  - grouped-query attention (config n_kv_head, Appendix E.1 uses two
    groups): W_QKV's columns are [Q (n_head heads) | K (n_kv_head heads) |
    V (n_kv_head heads)], query head h reads key/value head
    h // (n_head / n_kv_head);
  - the bidirectional mask (config bidirectional = 1) is only the attention
    mask of the masked-language-model study's encoder blocks (Sec. 6.4,
    after Cramming); it applies to the block stack, whose MLM head and
    loss are outside this path;
  - GPT-2 conventions: tanh GELU, eps 1e-5, biases on every linear layer,
    learned position embedding, final LayerNorm, LM head tied to wte,
    no dropout; next-token cross-entropy averaged over B*T positions;
  - the optimizer of the training setups (appendix: lr 1e-4, weight decay
    0.001, gradient clipping to norm 1; the optimizer is not named) is
    AdamW with beta1 0.9, beta2 0.999, eps 1e-8, decay on every tensor and
    PyTorch's clipping rule (adamw_step, train).

Weights are stored [in, out] so that a linear layer is y = x @ W + b.
Parameters are dicts of arrays (see ``paper_2510_14614_amd.synth`` for the
names); gradients come back in dicts with the same keys.
"""
from __future__ import annotations

import math

import numpy as np

ARCH_GPT, ARCH_FAL, ARCH_FALPLUS, ARCH_PARALLEL = 0, 1, 2, 3

f64 = np.float64


# ---------------------------------------------------------------------------
# Primitives
# ---------------------------------------------------------------------------

def normalize(x, eps):
    """Row normalisation used inside LayerNorm: (x - mean) / sqrt(var + eps),
    with the biased variance over the last axis."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    return (x - mu) * rstd, rstd


def normalize_backward(dxhat, xhat, rstd):
    """Gradient of normalize() given the gradient of its output."""
    n = xhat.shape[-1]
    s1 = dxhat.sum(axis=-1, keepdims=True)
    s2 = (dxhat * xhat).sum(axis=-1, keepdims=True)
    return rstd * (dxhat - s1 / n - xhat * s2 / n)


def layer_norm(x, g, b, eps):
    """LayerNorm (Ba et al.), the LN of Eq. 1 and Eq. 2."""
    xhat, rstd = normalize(x, eps)
    return xhat * g + b, (xhat, rstd)


def layer_norm_backward(dy, cache, g):
    xhat, rstd = cache
    dg = (dy * xhat).sum(axis=0)
    db = dy.sum(axis=0)
    dx = normalize_backward(dy * g, xhat, rstd)
    return dx, dg, db


_SQRT_2_OVER_PI = math.sqrt(2.0 / math.pi)


def gelu(x, tanh_form=True):
    """GELU non-linearity of the MLP (Sec. 2): tanh approximation by default,
    exact erf form otherwise."""
    if tanh_form:
        return 0.5 * x * (1.0 + np.tanh(_SQRT_2_OVER_PI * (x + 0.044715 * x ** 3)))
    erf = np.vectorize(math.erf, otypes=[f64])
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def gelu_grad(x, tanh_form=True):
    if tanh_form:
        u = _SQRT_2_OVER_PI * (x + 0.044715 * x ** 3)
        t = np.tanh(u)
        du = _SQRT_2_OVER_PI * (1.0 + 3.0 * 0.044715 * x ** 2)
        return 0.5 * (1.0 + t) + 0.5 * x * (1.0 - t * t) * du
    erf = np.vectorize(math.erf, otypes=[f64])
    cdf = 0.5 * (1.0 + erf(x / math.sqrt(2.0)))
    pdf = np.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)
    return cdf + x * pdf


def attention(q, k, v, causal=True):
    """Scaled dot-product attention of each head; with the causal mask
    query t sees keys 0..t, without it (the bidirectional encoder of the
    masked-language-model study) every key of its sequence.
    q, k, v: [B, H, T, hd]."""
    hd = q.shape[-1]
    T = q.shape[-2]
    s = q @ np.swapaxes(k, -1, -2) / math.sqrt(hd)
    if causal:
        future = np.triu(np.ones((T, T), dtype=bool), k=1)
        s = np.where(future, -np.inf, s)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    return p @ v, p


def causal_attention(q, k, v):
    return attention(q, k, v, causal=True)


def causal_attention_backward(do, q, k, v, p):
    """Backward of attention given its probabilities p (any mask: masked
    entries of p are zero)."""
    hd = q.shape[-1]
    scale = 1.0 / math.sqrt(hd)
    dv = np.swapaxes(p, -1, -2) @ do
    dp = do @ np.swapaxes(v, -1, -2)
    ds = p * (dp - (dp * p).sum(axis=-1, keepdims=True))
    dq = ds @ k * scale
    dk = np.swapaxes(ds, -1, -2) @ q * scale
    return dq, dk, dv


def cross_entropy(logits, targets):
    """Mean next-token cross-entropy and its gradient w.r.t. the logits."""
    n = logits.shape[0]
    m = logits.max(axis=1, keepdims=True)
    lse = m + np.log(np.exp(logits - m).sum(axis=1, keepdims=True))
    rows = np.arange(n)
    loss = float((lse[:, 0] - logits[rows, targets]).mean())
    dlogits = np.exp(logits - lse)
    dlogits[rows, targets] -= 1.0
    return loss, dlogits / n


# ---------------------------------------------------------------------------
# Sub-layers (Sec. 2): MHA (QKV projection, per-head attention, concatenation,
# output projection) and MLP (up-projection, GELU, down-projection)
# ---------------------------------------------------------------------------

def _split_heads(x, B, T, H):
    return x.reshape(B, T, H, -1).transpose(0, 2, 1, 3)


def _merge_heads(x):
    B, H, T, hd = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B * T, H * hd)


def kv_heads(cfg):
    """Number of key/value heads: n_head for MHA, fewer for grouped-query
    attention (Appendix E.1 uses two groups)."""
    return getattr(cfg, "n_kv_head", 0) or cfg.n_head


def mha_forward(h, p, cfg):
    """MHA; with grouped-query attention the Hkv key/value heads are each
    shared by n_head / Hkv consecutive query heads (Ainslie et al.)."""
    B, T, H = cfg.batch, cfg.seq_len, cfg.n_head
    Hkv = kv_heads(cfg)
    dA, dKV = H * cfg.head_dim, Hkv * cfg.head_dim
    qkv = h @ p["w_qkv"] + p["b_qkv"]
    q = _split_heads(qkv[:, :dA], B, T, H)
    k = np.repeat(_split_heads(qkv[:, dA:dA + dKV], B, T, Hkv), H // Hkv, axis=1)
    v = np.repeat(_split_heads(qkv[:, dA + dKV:], B, T, Hkv), H // Hkv, axis=1)
    o4, prob = attention(q, k, v, causal=not getattr(cfg, "bidirectional", 0))
    o = _merge_heads(o4)
    a = o @ p["w_o"] + p["b_o"]
    return a, (h, q, k, v, prob, o)


def mha_backward(da, p, cache, cfg):
    h, q, k, v, prob, o = cache
    B, T, H = cfg.batch, cfg.seq_len, cfg.n_head
    grads = {"w_o": o.T @ da, "b_o": da.sum(axis=0)}
    do = _split_heads(da @ p["w_o"].T, B, T, H)
    dq, dk, dv = causal_attention_backward(do, q, k, v, prob)
    # a shared key/value head collects the gradients of every query head of its group
    Hkv = kv_heads(cfg)
    grp = H // Hkv
    dk = dk.reshape(B, Hkv, grp, T, -1).sum(axis=2)
    dv = dv.reshape(B, Hkv, grp, T, -1).sum(axis=2)
    dqkv = np.concatenate([_merge_heads(dq), _merge_heads(dk), _merge_heads(dv)], axis=1)
    grads["w_qkv"] = h.T @ dqkv
    grads["b_qkv"] = dqkv.sum(axis=0)
    dh = dqkv @ p["w_qkv"].T
    return dh, grads


def mlp_forward(u, p, cfg):
    pre = u @ p["w_fc"] + p["b_fc"]
    g = gelu(pre, cfg.gelu_tanh)
    return g @ p["w_2"] + p["b_2"], (u, pre, g)


def mlp_backward(dm, p, cache, cfg):
    u, pre, g = cache
    grads = {"w_2": g.T @ dm, "b_2": dm.sum(axis=0)}
    dpre = (dm @ p["w_2"].T) * gelu_grad(pre, cfg.gelu_tanh)
    grads["w_fc"] = u.T @ dpre
    grads["b_fc"] = dpre.sum(axis=0)
    return dpre @ p["w_fc"].T, grads


# ---------------------------------------------------------------------------
# Blocks
# ---------------------------------------------------------------------------

def _block1_standard(cfg):
    return getattr(cfg, "fal_block1_mode", 0) == 1


def block_forward(cfg, i, x, p, first):
    """One decoder block.  ``first`` is the state carried from block 0 to the
    later blocks: FAL stores F = LN_F(A_1) under "F"; FAL+ stores the shared
    normalisation of A_1 under "xhatF" (its LayerNorms differ per block)."""
    eps = cfg.ln_eps
    h1, ln1 = layer_norm(x, p["ln1_g"], p["ln1_b"], eps)
    a, mha = mha_forward(h1, p, cfg)
    c = {"ln1": ln1, "mha": mha}
    if cfg.arch == ARCH_FAL and i == 0 and _block1_standard(cfg):
        # FAL with a standard first block: Eq. 1 in block 1, which also
        # produces F = LN_F(A_1) for every later block.
        first["F"], first["lnF"] = layer_norm(a, p["lnF_g"], p["lnF_b"], eps)
        xm = x + a
        u, c["ln2"] = layer_norm(xm, p["ln2_g"], p["ln2_b"], eps)
    elif cfg.arch == ARCH_GPT or (cfg.arch == ARCH_FALPLUS and i == 0):
        # Eq. 1: the MLP reads LN(X_i + A_i).
        xm = x + a
        u, c["ln2"] = layer_norm(xm, p["ln2_g"], p["ln2_b"], eps)
        if cfg.arch == ARCH_FALPLUS:
            # FAL+ block 1 is standard; it also records norm(A_1), which every
            # later block scales with its own first-attention LayerNorm.
            first["xhatF"], first["rstdF"] = normalize(a, eps)
    elif cfg.arch == ARCH_FAL:
        # Eq. 2: the MLP reads LN(X_i) + LN(MHA_1(LN(X_1))).
        if i == 0:
            first["F"], first["lnF"] = layer_norm(a, p["lnF_g"], p["lnF_b"], eps)
        h2, c["ln2"] = layer_norm(x, p["ln2_g"], p["ln2_b"], eps)
        u = h2 + first["F"]
        xm = x + a
    elif cfg.arch == ARCH_PARALLEL:
        # MHA and MLP both read X_i
        h2, c["ln2"] = layer_norm(x, p["ln2_g"], p["ln2_b"], eps)
        u = h2
        xm = x + a
    elif cfg.arch == ARCH_FALPLUS:
        # FAL+ (Appendix D), i >= 2 in the paper's numbering.
        xm = x + a
        h2, c["ln2"] = layer_norm(xm, p["ln2_g"], p["ln2_b"], eps)
        u = h2 + (first["xhatF"] * p["lnF_g"] + p["lnF_b"])
    else:
        raise ValueError(f"unknown arch {cfg.arch}")
    m, c["mlp"] = mlp_forward(u, p, cfg)
    return xm + m, c


def block_backward(cfg, i, dy, p, c, first, dfirst):
    """Backward of block_forward.  ``dfirst`` accumulates the gradient that
    flows into the shared first-attention state ("F" for FAL, "xhatF" for
    FAL+) from every block; block 0 consumes it.  Returns (dx, grads)."""
    grads = {k: np.zeros_like(v) for k, v in p.items()}
    du, g_mlp = mlp_backward(dy, p, c["mlp"], cfg)
    grads.update(g_mlp)
    if cfg.arch == ARCH_FAL and i == 0 and _block1_standard(cfg):
        dxm_ln, grads["ln2_g"], grads["ln2_b"] = layer_norm_backward(du, c["ln2"], p["ln2_g"])
        dxm = dy + dxm_ln
        da = dxm
        if "F" in dfirst:  # the later blocks' use of F
            dA1, grads["lnF_g"], grads["lnF_b"] = layer_norm_backward(dfirst["F"], first["lnF"], p["lnF_g"])
            da = da + dA1
        dx = dxm
    elif cfg.arch == ARCH_GPT or (cfg.arch == ARCH_FALPLUS and i == 0):
        dxm_ln, grads["ln2_g"], grads["ln2_b"] = layer_norm_backward(du, c["ln2"], p["ln2_g"])
        dxm = dy + dxm_ln
        da = dxm
        if cfg.arch == ARCH_FALPLUS and "xhatF" in dfirst:
            da = da + normalize_backward(dfirst["xhatF"], first["xhatF"], first["rstdF"])
        dx = dxm
    elif cfg.arch == ARCH_FAL:
        dfirst["F"] = dfirst.get("F", 0.0) + du
        dx_ln2, grads["ln2_g"], grads["ln2_b"] = layer_norm_backward(du, c["ln2"], p["ln2_g"])
        dx = dy + dx_ln2
        da = dy
        if i == 0:
            dA1, grads["lnF_g"], grads["lnF_b"] = layer_norm_backward(
                dfirst["F"], first["lnF"], p["lnF_g"])
            da = da + dA1
    elif cfg.arch == ARCH_PARALLEL:
        dx_ln2, grads["ln2_g"], grads["ln2_b"] = layer_norm_backward(du, c["ln2"], p["ln2_g"])
        dx = dy + dx_ln2
        da = dy
    else:  # FAL+, i >= 1
        dxm_ln, grads["ln2_g"], grads["ln2_b"] = layer_norm_backward(du, c["ln2"], p["ln2_g"])
        grads["lnF_g"] = (du * first["xhatF"]).sum(axis=0)
        grads["lnF_b"] = du.sum(axis=0)
        dfirst["xhatF"] = dfirst.get("xhatF", 0.0) + du * p["lnF_g"]
        dxm = dy + dxm_ln
        da = dxm
        dx = dxm
    dh1, g_mha = mha_backward(da, p, c["mha"], cfg)
    grads.update(g_mha)
    dx_ln1, grads["ln1_g"], grads["ln1_b"] = layer_norm_backward(dh1, c["ln1"], p["ln1_g"])
    return dx + dx_ln1, grads


# ---------------------------------------------------------------------------
# Whole step
# ---------------------------------------------------------------------------

def _as64(d):
    return {k: np.asarray(v, dtype=f64) for k, v in d.items()}


def stack_forward(cfg, blocks, x1):
    first = {}
    xs, caches = [x1], []
    for i, p in enumerate(blocks):
        y, c = block_forward(cfg, i, xs[-1], p, first)
        xs.append(y)
        caches.append(c)
    return xs, caches, first


def stack_backward(cfg, blocks, caches, first, dy):
    dfirst = {}
    dblocks = [None] * len(blocks)
    for i in range(len(blocks) - 1, -1, -1):
        dy, dblocks[i] = block_backward(cfg, i, dy, blocks[i], caches[i], first, dfirst)
    return dy, dblocks


def train_step(cfg, gparams, blocks, tokens):
    """Forward + backward of the language model on tokens [B, T+1].

    Returns dict(loss, logits [B*T, V], grads_global, grads_blocks)."""
    g = _as64(gparams)
    blocks = [_as64(b) for b in blocks]
    B, T = cfg.batch, cfg.seq_len
    tokens = np.asarray(tokens)
    ids = tokens[:, :T].reshape(-1)
    targets = tokens[:, 1:].reshape(-1)
    x1 = g["wte"][ids] + np.tile(g["wpe"][:T], (B, 1))
    xs, caches, first = stack_forward(cfg, blocks, x1)
    hf, lnf = layer_norm(xs[-1], g["lnf_g"], g["lnf_b"], cfg.ln_eps)
    logits = hf @ g["wte"].T
    loss, dlogits = cross_entropy(logits, targets)
    dg = {"wte": dlogits.T @ hf}
    dhf = dlogits @ g["wte"]
    dxl, dg["lnf_g"], dg["lnf_b"] = layer_norm_backward(dhf, lnf, g["lnf_g"])
    dx1, dblocks = stack_backward(cfg, blocks, caches, first, dxl)
    np.add.at(dg["wte"], ids, dx1)
    dg["wpe"] = np.zeros_like(g["wpe"])
    dg["wpe"][:T] = dx1.reshape(B, T, -1).sum(axis=0)
    return {"loss": loss, "logits": logits, "grads_global": dg, "grads_blocks": dblocks}


def stack_step(cfg, blocks, x1, gout):
    """Block stack without embedding or head: surrogate loss sum(G * X_{L+1}),
    so the gradient entering the last block is exactly G."""
    blocks = [_as64(b) for b in blocks]
    x1 = np.asarray(x1, dtype=f64)
    gout = np.asarray(gout, dtype=f64)
    xs, caches, first = stack_forward(cfg, blocks, x1)
    loss = float((gout * xs[-1]).sum())
    dx1, dblocks = stack_backward(cfg, blocks, caches, first, gout)
    return {"loss": loss, "y": xs[-1], "dx1": dx1, "grads_blocks": dblocks}


def forward_logits(cfg, gparams, blocks, tokens):
    """Logits only (used by invariance checks)."""
    g = _as64(gparams)
    blocks = [_as64(b) for b in blocks]
    B, T = cfg.batch, cfg.seq_len
    ids = np.asarray(tokens)[:, :T].reshape(-1)
    x1 = g["wte"][ids] + np.tile(g["wpe"][:T], (B, 1))
    xs, _, _ = stack_forward(cfg, blocks, x1)
    hf, _ = layer_norm(xs[-1], g["lnf_g"], g["lnf_b"], cfg.ln_eps)
    return hf @ g["wte"].T


# ---------------------------------------------------------------------------
# Optimizer and training loop
#
# The appendix's training setups give learning rate 1e-4, weight decay 0.001
# and gradient clipping to global norm 1; the optimizer itself is not named.
# Reading taken: AdamW, i.e. Adam's bias-corrected first and second moment
# estimates (Kingma & Ba) with weight decay applied to the parameters
# directly rather than through the gradient (Loshchilov & Hutter), with the
# usual defaults beta1 0.9, beta2 0.999, eps 1e-8, decay on every tensor.
# Clipping scales all gradients by min(1, clip / (norm + 1e-6)), the norm
# being the L2 norm of every gradient entry taken together.
# ---------------------------------------------------------------------------

ADAMW_PAPER = {"lr": 1e-4, "beta1": 0.9, "beta2": 0.999, "eps": 1e-8, "weight_decay": 1e-3,
               "max_grad_norm": 1.0}


def global_grad_norm(grads):
    """sqrt of the sum of squares of every entry of every gradient tensor."""
    return math.sqrt(sum(float(np.sum(np.square(np.asarray(g, dtype=f64)))) for g in grads))


def clip_coefficient(norm, max_grad_norm):
    """Factor the gradients are scaled by; 1 when clipping is off (<= 0)."""
    if max_grad_norm <= 0:
        return 1.0
    return min(1.0, max_grad_norm / (norm + 1e-6))


def adamw_step(params, grads, m, v, step, lr, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0,
               max_grad_norm=0.0):
    """One AdamW update of a list of tensors.

    step is the 1-based index of this update (the bias corrections use
    beta^step).  m and v are the moment estimates after step-1 updates
    (zeros before the first).  Returns (params, m, v, grad_norm) as new
    float64 arrays; grad_norm is the norm before clipping."""
    if step < 1:
        raise ValueError("step is 1-based")
    norm = global_grad_norm(grads)
    c = clip_coefficient(norm, max_grad_norm)
    bc1 = 1.0 - beta1 ** step
    bc2 = 1.0 - beta2 ** step
    out_p, out_m, out_v = [], [], []
    for p, g, m0, v0 in zip(params, grads, m, v):
        g = c * np.asarray(g, dtype=f64)
        m1 = beta1 * np.asarray(m0, dtype=f64) + (1.0 - beta1) * g
        v1 = beta2 * np.asarray(v0, dtype=f64) + (1.0 - beta2) * g * g
        p1 = np.asarray(p, dtype=f64) * (1.0 - lr * weight_decay)
        p1 = p1 - lr * (m1 / bc1) / (np.sqrt(v1 / bc2) + eps)
        out_p.append(p1)
        out_m.append(m1)
        out_v.append(v1)
    return out_p, out_m, out_v, norm


def _param_list(gparams, blocks):
    names = [("g", k) for k in gparams] + [(i, k) for i, b in enumerate(blocks) for k in b]
    vals = [gparams[k] for k in gparams] + [b[k] for b in blocks for k in b]
    return names, vals


def _unpack(names, vals, n_blocks):
    g, blocks = {}, [dict() for _ in range(n_blocks)]
    for (owner, k), x in zip(names, vals):
        if owner == "g":
            g[k] = x
        else:
            blocks[owner][k] = x
    return g, blocks


def train(cfg, gparams, blocks, token_batches, hp, first_step=1):
    """Training loop: for each batch one forward + backward (train_step)
    followed by one AdamW update of every parameter tensor.

    Returns dict(losses, grad_norms, gparams, blocks, m, v) with the
    parameters after the last update."""
    names, p = _param_list(_as64(gparams), [_as64(b) for b in blocks])
    m = [np.zeros_like(x) for x in p]
    v = [np.zeros_like(x) for x in p]
    losses, norms = [], []
    for j, tok in enumerate(token_batches):
        g, bl = _unpack(names, p, len(blocks))
        r = train_step(cfg, g, bl, tok)
        grads = [r["grads_global"][k] if owner == "g" else r["grads_blocks"][owner][k] for owner, k in names]
        p, m, v, norm = adamw_step(p, grads, m, v, first_step + j, **hp)
        losses.append(r["loss"])
        norms.append(norm)
    g, bl = _unpack(names, p, len(blocks))
    return {"losses": losses, "grad_norms": norms, "gparams": g, "blocks": bl, "m": m, "v": v}
