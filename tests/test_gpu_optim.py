"""GPU parity of the optimizer (fal_adamw_step through the C ABI) and of the
training loop (fal_model_step + fal_adamw_step) against the CPU fp64
oracle.

Tolerances come from the fp32 arithmetic of the update: every quantity is
a handful of fp32 operations away from its inputs, so weights agree to a
few fp32 ulps of the weight (relative 2e-6) plus relative 4e-6 of the
summed update scales so far.  The update scale of a step is the update the
terms of the first moment would give without cancelling,
lr/(1-beta1^t) (beta1 |m| + (1-beta1) |c g|) / (sqrt(v_hat) + eps): the
rounding error of the new first moment is relative to those terms, not to
their (possibly tiny) sum.  Moments agree to relative 2e-6 of the tensor's
largest entry, and the norm (an fp64 sum rounded once to fp32)
to relative 1e-6.  bf16 weights are the round-to-nearest-even image of the
fp32 master weights."""
from ctypes import byref, c_void_p

import numpy as np
import pytest

import oracle
from paper_2510_14614_amd import fal, get_config, synth
from paper_2510_14614_amd.config import ARCH_FAL, ARCH_FALPLUS, ARCH_GPT, SCHED_STREAMS_MERGED, Config

from gpu_helpers import TOL, log

pytestmark = pytest.mark.gpu

HP = dict(lr=1e-2, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1, max_grad_norm=1.0)


def _dev(x, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x))
    return (t.to(dtype) if dtype is not None else t).cuda()


def _ptr(t):
    return c_void_p(t.data_ptr()) if t is not None else None


def _adamw(F, step, n, master, params, grads, m, v, norm, **hp):
    p = fal.adamw_params(**dict(HP, **hp))
    return fal.lib().fal_adamw_step(F.ctx, byref(p), step, n, _ptr(master), _ptr(params), _ptr(grads),
                                    _ptr(m), _ptr(v), _ptr(norm))


def _update_scale(m_prev, g, v_new, step, c, hp):
    b1 = hp["beta1"]
    bc1, bc2 = 1 - b1 ** step, 1 - hp["beta2"] ** step
    return hp["lr"] / bc1 * (b1 * np.abs(m_prev) + (1 - b1) * np.abs(c * g)) / (np.sqrt(v_new / bc2) + hp["eps"])


def _check_state(tag, n, got, ref, upd):
    """upd: per element, the summed update scales of the oracle's steps."""
    import torch
    torch.cuda.synchronize()
    gm, gmm, gv = (t.cpu().numpy().astype(np.float64) for t in got)
    rp, rm, rv = ref
    if n == 0:
        return
    err = np.abs(gm - rp)
    bound = 2e-6 * np.abs(rp) + 4e-6 * upd + 1e-30
    worst = int(np.argmax(err / bound))
    assert np.all(err <= bound), (f"{tag} master: element {worst} got {gm[worst]!r} ref {rp[worst]!r} "
                                  f"update sum {upd[worst]!r}")
    np.testing.assert_allclose(gmm, rm, rtol=2e-6, atol=2e-6 * np.abs(rm).max(), err_msg=f"{tag} m")
    np.testing.assert_allclose(gv, rv, rtol=2e-6, atol=2e-6 * np.abs(rv).max(), err_msg=f"{tag} v")


# sizes: empty, below one vector, ragged tails, exact update chunks (2048
# elements), several chunks, more than one sweep of the norm grid (2^21
# float4 units per sweep is 2048 workgroups x 256 threads x 4 elements)
SIZES = [0, 1, 5, 4096, 3 * 2048 + 7, (1 << 20) + 3, 5_000_003]


@pytest.mark.parametrize("lp_mode", ["bf16", "f32_copy", "f32_inplace"])
@pytest.mark.parametrize("n", SIZES)
def test_adamw_matches_oracle(n, lp_mode):
    import torch
    dtype = 1 if lp_mode == "bf16" else 0
    cfg = get_config("tiny", dtype=dtype)
    log(f"adamw n={n} mode={lp_mode}")
    F = fal.Fal(cfg)
    p0 = synth.make_flat(n, seed=100)
    # moments as a run leaves them: v >= m^2, so |m| / sqrt(v) <= 1
    m0 = synth.make_flat(n, seed=101, scale=1e-3)
    v0 = m0 * m0 + synth.make_flat(n, seed=102, scale=1e-7, positive=True)
    master, m, v = _dev(p0), _dev(m0), _dev(v0)
    if lp_mode == "bf16":
        params = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    elif lp_mode == "f32_copy":
        params = torch.zeros(n, dtype=torch.float32, device="cuda")
    else:
        params = None
    norm = torch.full((1,), -1.0, dtype=torch.float32, device="cuda")
    rp, rm, rv = [p0.astype(np.float64)], [m0.astype(np.float64)], [v0.astype(np.float64)]
    upd = np.zeros(n)
    # gradient norms about 10, 0.1 and 3: clipping on, off, on
    for step, (seed, target) in enumerate([(103, 10.0), (104, 0.1), (105, 3.0)], start=4):
        g = synth.make_flat(n, seed=seed, scale=target / np.sqrt(max(n, 1)))
        st = _adamw(F, step, n, master, params, _dev(g), m, v, norm)
        assert st == fal.FAL_OK, fal.lib().fal_last_error(F.ctx)
        m_prev = rm[0]
        rp, rm, rv, rnorm = oracle.adamw_step(rp, [g], rm, rv, step, **HP)
        upd += _update_scale(m_prev, g.astype(np.float64), rv[0], step,
                             oracle.clip_coefficient(rnorm, HP["max_grad_norm"]), HP)
        torch.cuda.synchronize()
        assert abs(norm.item() - rnorm) <= 1e-6 * rnorm + 1e-30, (norm.item(), rnorm)
        _check_state(f"n={n} step={step}", n, (master, m, v), (rp[0], rm[0], rv[0]), upd)
        if lp_mode == "bf16":
            got = params.float().cpu().numpy()
            # the copy is exactly the rounding of the fp32 master ...
            np.testing.assert_array_equal(got, synth.round_to_bf16(master.cpu().numpy()))
            # ... and the rounded oracle weight is within the master bound
            # plus half a bf16 step on either side
            ref = synth.round_to_bf16(rp[0].astype(np.float32)).astype(np.float64)
            got = got.astype(np.float64)
            lim = 2e-6 * np.abs(rp[0]) + 4e-6 * upd + 2.0 ** -8 * (np.abs(got) + np.abs(ref)) + 1e-30
            assert np.all(np.abs(got - ref) <= lim)
        elif lp_mode == "f32_copy":
            np.testing.assert_array_equal(params.cpu().numpy(), master.cpu().numpy())
    F.close()


def test_adamw_deterministic_and_clip_off():
    import torch
    cfg = get_config("tiny", dtype=1)
    F = fal.Fal(cfg)
    n = 3_000_001
    g = _dev(synth.make_flat(n, seed=110, scale=0.01))
    outs = []
    for _ in range(2):
        master = _dev(synth.make_flat(n, seed=111))
        params = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
        m, v = torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
        norm = torch.zeros(1, device="cuda")
        assert _adamw(F, 1, n, master, params, g, m, v, norm, max_grad_norm=0.0) == fal.FAL_OK
        torch.cuda.synchronize()
        outs.append((master.cpu().numpy(), params.view(torch.int16).cpu().numpy(), norm.item()))
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])
    assert outs[0][2] == outs[1][2]
    # clipping off: first step from zero moments is the closed form
    # p (1 - lr wd) - lr g / (|g| + eps) (norm about 17, unclipped)
    p0 = synth.make_flat(n, seed=111).astype(np.float64)
    gg = synth.make_flat(n, seed=110, scale=0.01).astype(np.float64)
    ref = p0 * (1 - HP["lr"] * HP["weight_decay"]) - HP["lr"] * gg / (np.abs(gg) + HP["eps"])
    err = np.abs(outs[0][0] - ref)
    assert np.all(err <= 2e-6 * np.abs(ref) + 4e-6 * HP["lr"]), err.max()
    F.close()


def test_adamw_rejects_bad_arguments():
    import torch
    cfg = get_config("tiny", dtype=1)
    F = fal.Fal(cfg)
    n = 1024
    mk = lambda: torch.zeros(n + 8, dtype=torch.float32, device="cuda")
    master, g, m, v = mk(), mk(), mk(), mk()
    params = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    E = fal.FAL_ERR_INVALID_ARG
    assert _adamw(F, 0, n, master, params, g, m, v, None) == E            # step is 1-based
    assert _adamw(F, 1, -1, master, params, g, m, v, None) == E           # negative n
    assert _adamw(F, 1, n, master, None, g, m, v, None) == E              # bf16 copy missing
    assert _adamw(F, 1, n, master, params, g, g, v, None) == E            # grads aliases m
    assert _adamw(F, 1, n, master, params, g, m, v, None, beta1=1.0) == E
    assert _adamw(F, 1, n, master, params, g, m, v, None, lr=-1.0) == E
    assert _adamw(F, 1, n, master, params, g, m, v, None, eps=float("nan")) == E
    # 4-byte offset: not 16-byte aligned
    bad = c_void_p(master.data_ptr() + 4)
    p = fal.adamw_params(**HP)
    st = fal.lib().fal_adamw_step(F.ctx, byref(p), 1, n, bad, _ptr(params), _ptr(g), _ptr(m), _ptr(v), None)
    assert st == E
    # overlapping ranges: m starts inside master
    st = fal.lib().fal_adamw_step(F.ctx, byref(p), 1, n, _ptr(master), _ptr(params), _ptr(g),
                                  c_void_p(master.data_ptr() + 16 * 4), _ptr(v), None)
    assert st == E
    # the context still works after rejected calls
    assert _adamw(F, 1, n, master, params, g, m, v, None) == fal.FAL_OK
    torch.cuda.synchronize()
    F.close()


def _train_gpu(cfg, g, blocks, batches, hp):
    import torch
    F = fal.Fal(cfg)
    F.load_params(g, blocks)
    F.init_optimizer()
    losses, norms = [], []
    for tok in batches:
        t = torch.from_numpy(np.ascontiguousarray(tok, dtype=np.int32)).cuda()
        losses.append(float(F.train_step(t, **hp).item()))
        norms.append(float(F.grad_norm.item()))
    flat = F.master.detach().cpu().numpy().astype(np.float64)
    F.close()
    return losses, norms, flat


def _flat_ref(cfg, r):
    F_layout = fal.param_layout(cfg)
    return fal.flatten_params(cfg, r["gparams"], r["blocks"], F_layout).astype(np.float64)


@pytest.mark.parametrize("arch", [ARCH_GPT, ARCH_FAL, ARCH_FALPLUS])
def test_training_loop_fp32(arch):
    # four updates on four different batches; the loss of batch k is
    # computed with the weights after k-1 updates, so it checks the updates
    cfg = get_config("tiny", arch=arch, dtype=0)
    log(f"training loop fp32 arch={arch}")
    g, blocks = synth.make_params(cfg, seed=20)
    batches = [synth.make_tokens(cfg, seed=21 + k) for k in range(4)]
    hp = dict(oracle.ADAMW_PAPER, lr=1e-3)
    losses, norms, flat = _train_gpu(cfg, g, blocks, batches, hp)
    r = oracle.train(cfg, g, blocks, batches, hp)
    log(f"  losses gpu {losses} ref {r['losses']}")
    for a, b in zip(losses, r["losses"]):
        assert abs(a - b) <= TOL[0] * abs(b)
    for a, b in zip(norms, r["grad_norms"]):
        assert abs(a - b) <= TOL[0] * b
    # weights: Adam's step is about lr * sign(g) for small moments, so an
    # element whose gradient is tiny next to its tensor's largest can move
    # differently; nearly all elements must agree closely
    ref = _flat_ref(cfg, r)
    err = np.abs(flat - ref)
    assert err.max() <= 2 * len(batches) * hp["lr"], err.max()
    assert np.quantile(err, 0.99) <= 1e-2 * hp["lr"], np.quantile(err, 0.99)


@pytest.mark.parametrize("arch", [ARCH_GPT, ARCH_FAL])
def test_training_loop_bf16_ragged(arch):
    # ragged shapes in every GEMM dimension; one batch memorised over six
    # updates: the loss follows the oracle's trajectory and goes down
    cfg = Config(n_layer=2, d_model=192, n_head=3, head_dim=64, d_ff=328, vocab=1000, seq_len=100,
                 batch=3, arch=arch, dtype=1, sched=SCHED_STREAMS_MERGED)
    log(f"training loop bf16 ragged arch={arch}")
    g, blocks = synth.make_params(cfg, seed=30)
    tok = synth.make_tokens(cfg, seed=31, dist="zipf")
    hp = dict(oracle.ADAMW_PAPER, lr=1e-3)  # the oracle's losses fall at every step here
    losses, norms, _ = _train_gpu(cfg, g, blocks, [tok] * 6, hp)
    r = oracle.train(cfg, g, blocks, [tok] * 6, hp)
    log(f"  losses gpu {losses} ref {r['losses']}")
    for a, b in zip(losses, r["losses"]):
        assert abs(a - b) <= TOL[1] * abs(b)
    assert losses[-1] < losses[0] - 1.0
    assert all(b < a for a, b in zip(losses, losses[1:])), losses


def test_adamw_full_size_sampled():
    # the whole GPT-2-small parameter buffer (bf16 weights, fp32 master),
    # the size the training loop updates; the norm is checked in full and
    # the update on a sample of elements the oracle computes one by one
    import torch
    cfg = get_config("gpt2-small", dtype=1)
    n = fal.param_layout(cfg)["total"]
    log(f"adamw full size n={n}")
    F = fal.Fal(cfg.replace(batch=1))
    p0 = synth.make_flat(n, seed=120)
    g = synth.make_flat(n, seed=121, scale=5.0 / np.sqrt(n))
    master, gd = _dev(p0), _dev(g)
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    params = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    norm = torch.zeros(1, device="cuda")
    assert _adamw(F, 1, n, master, params, gd, m, v, norm) == fal.FAL_OK
    torch.cuda.synchronize()
    rnorm = oracle.global_grad_norm([g])
    assert abs(norm.item() - rnorm) <= 1e-6 * rnorm
    c = oracle.clip_coefficient(rnorm, HP["max_grad_norm"])
    rng = np.random.Generator(np.random.PCG64(122))
    idx = np.unique(np.concatenate([rng.integers(0, n, 200_000), np.arange(4096), np.arange(n - 4096, n)]))
    z = np.zeros(idx.size)
    rp, rm, rv, _ = oracle.adamw_step([p0[idx]], [c * g[idx].astype(np.float64)], [z], [z], 1,
                                      **dict(HP, max_grad_norm=0.0))
    it = torch.from_numpy(idx).cuda()
    got = [master[it], m[it], v[it]]
    upd = _update_scale(z, g[idx].astype(np.float64), rv[0], 1, c, HP)
    _check_state("full", idx.size, got, (rp[0], rm[0], rv[0]), upd)
    np.testing.assert_array_equal(params[it].float().cpu().numpy(), synth.round_to_bf16(got[0].cpu().numpy()))
    F.close()
