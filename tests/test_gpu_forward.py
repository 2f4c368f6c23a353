"""GPU parity of the forward-only entry points (fal_model_forward,
fal_stack_forward) against the CPU fp64 oracle, and their agreement with
the forward half of the training step (same kernels: bitwise)."""
import numpy as np
import pytest

import oracle
from paper_2510_14614_amd import fal, synth
from paper_2510_14614_amd.config import ARCH_FAL, ARCH_FALPLUS, ARCH_GPT, ARCH_PARALLEL, SCHED_STREAMS_MERGED, Config

from gpu_helpers import TOL, log, rel_err

pytestmark = pytest.mark.gpu

ARCHS = [ARCH_GPT, ARCH_FAL, ARCH_FALPLUS, ARCH_PARALLEL]


def _ragged(arch, dtype, **kw):
    base = dict(n_layer=2, d_model=192, n_head=3, head_dim=64, d_ff=328, vocab=1003, seq_len=100,
                batch=3, arch=arch, dtype=dtype, sched=SCHED_STREAMS_MERGED)
    base.update(kw)
    return Config(**base)


@pytest.mark.parametrize("dtype", [0, 1])
@pytest.mark.parametrize("arch", ARCHS)
def test_model_forward_matches_oracle_and_step(arch, dtype):
    import torch
    cfg = _ragged(arch, dtype)
    log(f"model forward arch={arch} dtype={dtype}")
    g, blocks = synth.make_params(cfg, seed=40)
    tok = synth.make_tokens(cfg, seed=41, dist="zipf")
    F = fal.Fal(cfg)
    F.load_params(g, blocks)
    t = torch.from_numpy(tok).cuda()
    lf = torch.zeros(cfg.tokens, cfg.vocab, device="cuda")
    loss_f = float(F.model_forward(t, lf).item())
    logits_f = lf.cpu().numpy()
    # the training step's forward half: identical loss and logits
    ls = torch.zeros_like(lf)
    loss_s = float(F.model_step(t, ls).item())
    torch.cuda.synchronize()
    assert loss_f == loss_s
    np.testing.assert_array_equal(logits_f, ls.cpu().numpy())
    # the oracle
    ref_logits = oracle.forward_logits(cfg, g, blocks, tok)
    ref_loss, _ = oracle.cross_entropy(ref_logits, tok[:, 1:].reshape(-1))
    e_loss = abs(loss_f - ref_loss) / abs(ref_loss)
    e_logits = rel_err(logits_f, ref_logits)
    log(f"  loss {loss_f:.6f} ref {ref_loss:.6f} err {e_loss:.2e}; logits err {e_logits:.2e}")
    assert e_loss <= TOL[dtype] and e_logits <= TOL[dtype]
    # optional outputs: logits only, then nothing at all
    lf2 = torch.zeros_like(lf)
    assert F.model_forward(t, lf2, loss=False) is None
    F.model_forward(t, None, loss=False)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(lf2.cpu().numpy(), logits_f)
    F.close()


@pytest.mark.parametrize("dtype", [0, 1])
@pytest.mark.parametrize("arch", ARCHS)
def test_stack_forward_matches_oracle_and_step(arch, dtype):
    import torch
    # the tensor-parallel shard layout: d_model (384) != n_head * head_dim (256)
    cfg = Config(n_layer=2, d_model=384, n_head=2, head_dim=128, d_ff=344, vocab=0, seq_len=136,
                 batch=2, arch=arch, dtype=dtype, has_embed_head=0)
    log(f"stack forward arch={arch} dtype={dtype}")
    _, blocks = synth.make_params(cfg, seed=42)
    x1, gout = synth.make_stack_inputs(cfg, seed=43)
    F = fal.Fal(cfg)
    F.load_params({}, blocks)
    x = torch.from_numpy(x1).cuda()
    y = torch.zeros_like(x)
    F.stack_forward(x, y)
    yf = y.cpu().numpy()
    dy = torch.from_numpy(gout).cuda()
    F.stack_step(x, dy)
    torch.cuda.synchronize()
    # X_L of the step, read from the workspace the context carves
    off = F.residual_out() - F._ws.data_ptr()
    ys = F._ws[off:off + 4 * y.numel()].view(torch.float32).reshape(y.shape)
    np.testing.assert_array_equal(yf, ys.cpu().numpy())
    xs, _, _ = oracle.stack_forward(cfg, [{k: v.astype(np.float64) for k, v in b.items()} for b in blocks],
                                    x1.astype(np.float64))
    e = rel_err(yf, xs[-1])
    log(f"  X_L err {e:.2e}")
    assert e <= TOL[dtype]
    F.close()


def test_forward_rejects_wrong_workload():
    import torch
    cfg = _ragged(ARCH_FAL, 1)
    F = fal.Fal(cfg)
    x = torch.zeros(cfg.tokens, cfg.d_model, device="cuda")
    st = fal.lib().fal_stack_forward(F.ctx, fal.c_void_p(F.params.data_ptr()), fal.c_void_p(x.data_ptr()), None)
    assert st == fal.FAL_ERR_INVALID_ARG
    st = fal.lib().fal_model_forward(F.ctx, None, None, None, None)
    assert st == fal.FAL_ERR_INVALID_ARG
    F.close()
