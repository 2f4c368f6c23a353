"""Helpers for the GPU parity tests: run the library through the C ABI on
seeded synthetic inputs and compare against the CPU oracle."""
import sys

import numpy as np

from paper_2510_14614_amd import fal, synth
from paper_2510_14614_amd.config import Config

TOL = {0: 1e-4, 1: 2e-2}  # max relative error (inf-norm), fp32 / bf16


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.abs(ref).max()
    if den == 0.0:
        return 0.0 if np.abs(got).max() == 0.0 else np.inf
    return float(np.abs(got - ref).max() / den)


def gpu_model_step(cfg: Config, g, blocks, tokens, want_logits=True, ctx=None):
    import torch
    F = ctx or fal.Fal(cfg)
    F.load_params(g, blocks)
    tok = torch.from_numpy(np.ascontiguousarray(tokens, dtype=np.int32)).cuda()
    logits = torch.zeros(cfg.tokens, cfg.vocab, dtype=torch.float32, device="cuda") if want_logits else None
    loss = F.model_step(tok, logits)
    torch.cuda.synchronize()
    gg, gb = F.grads_numpy()
    out = {"loss": float(loss.item()), "grads_global": gg, "grads_blocks": gb,
           "logits": logits.cpu().numpy() if want_logits else None}
    if ctx is None:
        F.close()
    return out


def gpu_stack_step(cfg: Config, blocks, x1, gout, ctx=None):
    import torch
    F = ctx or fal.Fal(cfg)
    F.load_params({}, blocks)
    x = torch.from_numpy(np.ascontiguousarray(x1, dtype=np.float32)).cuda()
    dy = torch.from_numpy(np.ascontiguousarray(gout, dtype=np.float32)).cuda()
    dx = torch.zeros_like(x)
    loss = F.stack_step(x, dy, dx)
    torch.cuda.synchronize()
    _, gb = F.grads_numpy()
    out = {"loss": float(loss.item()), "grads_blocks": gb, "dx1": dx.cpu().numpy()}
    if ctx is None:
        F.close()
    return out


def compare_step(cfg, gpu, ref, tol=None, label=""):
    """Assert every compared tensor is within tol; returns the error table."""
    tol = TOL[cfg.dtype] if tol is None else tol
    errs = {}
    # a surrogate loss sum(G * X) can cancel; scale by sum |G * X| there
    errs["loss"] = abs(gpu["loss"] - ref["loss"]) / max(abs(ref["loss"]), ref.get("loss_scale", 0.0))
    if gpu.get("logits") is not None and "logits" in ref:
        errs["logits"] = rel_err(gpu["logits"], ref["logits"])
    if "dx1" in gpu:
        errs["dx1"] = rel_err(gpu["dx1"], ref["dx1"])
    for k, v in gpu.get("grads_global", {}).items():
        errs[f"d{k}"] = rel_err(v, ref["grads_global"][k])
    for i, blk in enumerate(gpu["grads_blocks"]):
        for k, v in blk.items():
            errs[f"b{i}.d{k}"] = rel_err(v, ref["grads_blocks"][i][k])
    worst = max(errs.items(), key=lambda kv: kv[1])
    log(f"[{label}] worst {worst[0]} = {worst[1]:.3e} (tol {tol:g}); loss gpu {gpu['loss']:.6f} ref {ref['loss']:.6f}")
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"{label}: over tolerance {tol}: {bad}"
    return errs
