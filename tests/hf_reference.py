"""Independent reference for the oracle: HuggingFace ``transformers`` GPT-2
(the textbook Pre-LN GPT-2 implementation) in float64 on the CPU, with torch
autograd for the gradients.

GPT baseline (Eq. 1) is the unmodified library model.  FAL (Eq. 2), FAL+
(Appendix D) and the parallel block (MHA and MLP on the same input) are
expressed by swapping each block's second LayerNorm module for one that
reroutes its input, everything else (attention, MLP, residual
adds, embedding, head, loss, backward) stays the library's own code.
"""
import numpy as np
import torch
from transformers import GPT2Config, GPT2LMHeadModel

from paper_2510_14614_amd.config import ARCH_FAL, ARCH_FALPLUS, ARCH_PARALLEL


class _RoutedLN2(torch.nn.Module):
    """Replacement for block i's ln_2.  HF calls it with X_i + A_i."""

    def __init__(self, ln2, lnF, i, arch, state):
        super().__init__()
        self.ln2, self.lnF, self.i, self.arch, self.state = ln2, lnF, i, arch, state

    def forward(self, h):
        st = self.state
        if self.arch == ARCH_FAL:
            if self.i == 0:
                st["F"] = self.lnF(st["A1"])              # LN of the first attention, once
                if st["block1_standard"]:
                    return self.ln2(h)                    # standard block 1 (only emits F)
            return self.ln2(st["x_in"][self.i]) + st["F"]  # LN(X_i) + LN(MHA_1(LN(X_1)))
        if self.arch == ARCH_PARALLEL:
            return self.ln2(st["x_in"][self.i])           # LN2(X_i): the block's own input
        if self.arch == ARCH_FALPLUS and self.i > 0:
            return self.ln2(h) + self.lnF(st["A1"])       # LN(X_i + A_i) + LN_i(MHA_1(...))
        return self.ln2(h)


def build(cfg, gparams, blocks):
    assert cfg.d_attn == cfg.d_model
    conf = GPT2Config(vocab_size=cfg.vocab, n_positions=cfg.seq_len, n_embd=cfg.d_model,
                      n_layer=cfg.n_layer, n_head=cfg.n_head, n_inner=cfg.d_ff,
                      activation_function="gelu_new" if cfg.gelu_tanh else "gelu",
                      resid_pdrop=0.0, embd_pdrop=0.0, attn_pdrop=0.0,
                      layer_norm_epsilon=cfg.ln_eps, bos_token_id=0, eos_token_id=0)
    conf._attn_implementation = "eager"
    model = GPT2LMHeadModel(conf).double().eval()
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    tr = model.transformer
    with torch.no_grad():
        tr.wte.weight.copy_(t(gparams["wte"]))
        tr.wpe.weight.copy_(t(gparams["wpe"]))
        tr.ln_f.weight.copy_(t(gparams["lnf_g"]))
        tr.ln_f.bias.copy_(t(gparams["lnf_b"]))
    state = {"x_in": {}, "block1_standard": getattr(cfg, "fal_block1_mode", 0) == 1}
    lnFs = []
    for i, (blk, p) in enumerate(zip(tr.h, blocks)):
        with torch.no_grad():
            blk.ln_1.weight.copy_(t(p["ln1_g"])); blk.ln_1.bias.copy_(t(p["ln1_b"]))
            blk.attn.c_attn.weight.copy_(t(p["w_qkv"])); blk.attn.c_attn.bias.copy_(t(p["b_qkv"]))
            blk.attn.c_proj.weight.copy_(t(p["w_o"])); blk.attn.c_proj.bias.copy_(t(p["b_o"]))
            blk.ln_2.weight.copy_(t(p["ln2_g"])); blk.ln_2.bias.copy_(t(p["ln2_b"]))
            blk.mlp.c_fc.weight.copy_(t(p["w_fc"])); blk.mlp.c_fc.bias.copy_(t(p["b_fc"]))
            blk.mlp.c_proj.weight.copy_(t(p["w_2"])); blk.mlp.c_proj.bias.copy_(t(p["b_2"]))
        lnF = torch.nn.LayerNorm(cfg.d_model, eps=cfg.ln_eps).double()
        with torch.no_grad():
            lnF.weight.copy_(t(p["lnF_g"])); lnF.bias.copy_(t(p["lnF_b"]))
        lnFs.append(lnF)

        def pre_hook(mod, args, kwargs, i=i):
            hs = args[0] if args else kwargs["hidden_states"]
            state["x_in"][i] = hs
        blk.register_forward_pre_hook(pre_hook, with_kwargs=True)
        if i == 0:
            def attn_hook(mod, args, out):
                state["A1"] = out[0]
            blk.attn.register_forward_hook(attn_hook)
        blk.ln_2 = _RoutedLN2(blk.ln_2, lnF, i, cfg.arch, state)
    model.fal_lnF = torch.nn.ModuleList(lnFs)
    return model


def run(cfg, gparams, blocks, tokens):
    """Returns loss, logits [B*T, V], global grads, block grads (numpy)."""
    model = build(cfg, gparams, blocks)
    T = cfg.seq_len
    tok = torch.tensor(np.asarray(tokens, dtype=np.int64))
    out = model(input_ids=tok[:, :T])
    logits = out.logits.reshape(-1, cfg.vocab)
    loss = torch.nn.functional.cross_entropy(logits, tok[:, 1:].reshape(-1))
    loss.backward()
    tr = model.transformer
    gg = {"wte": tr.wte.weight.grad, "wpe": tr.wpe.weight.grad,
          "lnf_g": tr.ln_f.weight.grad, "lnf_b": tr.ln_f.bias.grad}
    gb = []
    for blk, lnF in zip(tr.h, model.fal_lnF):
        z = lambda p: p.grad if p.grad is not None else torch.zeros_like(p)
        gb.append({
            "ln1_g": z(blk.ln_1.weight), "ln1_b": z(blk.ln_1.bias),
            "w_qkv": z(blk.attn.c_attn.weight), "b_qkv": z(blk.attn.c_attn.bias),
            "w_o": z(blk.attn.c_proj.weight), "b_o": z(blk.attn.c_proj.bias),
            "ln2_g": z(blk.ln_2.ln2.weight), "ln2_b": z(blk.ln_2.ln2.bias),
            "w_fc": z(blk.mlp.c_fc.weight), "b_fc": z(blk.mlp.c_fc.bias),
            "w_2": z(blk.mlp.c_proj.weight), "b_2": z(blk.mlp.c_proj.bias),
            "lnF_g": z(lnF.weight), "lnF_b": z(lnF.bias),
        })
    np_ = lambda d: {k: v.detach().numpy() for k, v in d.items()}
    return loss.item(), logits.detach().numpy(), np_(gg), [np_(b) for b in gb]
