"""Pins of the oracle's optimizer and training loop against things other
than itself: PyTorch's AdamW and gradient clipping (float64, CPU), the
closed form of the first update, invariances of Adam's update, and the
loss of a memorised batch going down."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2510_14614_amd import get_config, synth


def _tensors(rng, shapes, scale=1.0):
    return [rng.standard_normal(s) * scale for s in shapes]


SHAPES = [(7, 5), (13,), (3, 4, 2)]


@pytest.mark.parametrize("clip", [0.0, 1.0, 50.0])
@pytest.mark.parametrize("wd", [0.0, 1e-3, 0.1])
def test_adamw_matches_torch(clip, wd):
    rng = np.random.default_rng(7)
    p0 = _tensors(rng, SHAPES)
    lr, b1, b2, eps = 3e-2, 0.9, 0.95, 1e-8
    tp = [torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in p0]
    opt = torch.optim.AdamW(tp, lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd)
    p, m, v = p0, [np.zeros_like(x) for x in p0], [np.zeros_like(x) for x in p0]
    for step in range(1, 7):
        # gradient scale varies so clipping is active on some steps only
        grads = _tensors(rng, SHAPES, scale=[0.05, 3.0, 0.3, 10.0, 0.01, 1.0][step - 1])
        for t, g in zip(tp, grads):
            t.grad = torch.tensor(g, dtype=torch.float64)
        ref_norm = math.sqrt(sum(float(np.sum(g * g)) for g in grads))
        if clip > 0:
            tn = torch.nn.utils.clip_grad_norm_(tp, clip)
            assert abs(float(tn) - ref_norm) <= 1e-12 * ref_norm
        opt.step()
        p, m, v, norm = oracle.adamw_step(p, grads, m, v, step, lr, b1, b2, eps, wd, clip)
        assert abs(norm - ref_norm) <= 1e-12 * ref_norm
        for t, x, mx, vx in zip(tp, p, m, v):
            st = opt.state[t]
            np.testing.assert_allclose(x, t.detach().numpy(), rtol=1e-12, atol=1e-14)
            np.testing.assert_allclose(mx, st["exp_avg"].numpy(), rtol=1e-12, atol=1e-15)
            np.testing.assert_allclose(vx, st["exp_avg_sq"].numpy(), rtol=1e-12, atol=1e-18)


def test_adamw_first_step_closed_form():
    # from zero moments the bias-corrected estimates are g and g^2 exactly,
    # so the first update is p (1 - lr wd) - lr g / (|g| + eps)
    rng = np.random.default_rng(3)
    p0 = _tensors(rng, SHAPES)
    g = _tensors(rng, SHAPES, scale=0.1)
    lr, wd, eps = 1e-2, 0.05, 1e-3
    z = [np.zeros_like(x) for x in p0]
    p1, m1, v1, _ = oracle.adamw_step(p0, g, z, z, 1, lr, 0.8, 0.99, eps, wd, 0.0)
    for a, b, gg, mm, vv in zip(p1, p0, g, m1, v1):
        np.testing.assert_allclose(a, b * (1 - lr * wd) - lr * gg / (np.abs(gg) + eps), rtol=1e-13, atol=1e-16)
        np.testing.assert_allclose(mm, 0.2 * gg, rtol=1e-14)
        np.testing.assert_allclose(vv, 0.01 * gg * gg, rtol=1e-14)


def test_adamw_second_step_closed_form():
    # constant gradient g on both steps: m_hat = g, v_hat = g^2 again, so the
    # step is the same sign step; with wd 0 the parameter moves by 2 lr
    # g/(|g| + eps) in total
    rng = np.random.default_rng(4)
    p0 = _tensors(rng, SHAPES)
    g = _tensors(rng, SHAPES, scale=0.5)
    z = [np.zeros_like(x) for x in p0]
    lr, eps = 1e-2, 1e-6
    p, m, v, _ = oracle.adamw_step(p0, g, z, z, 1, lr, 0.9, 0.999, eps, 0.0, 0.0)
    p, m, v, _ = oracle.adamw_step(p, g, m, v, 2, lr, 0.9, 0.999, eps, 0.0, 0.0)
    for a, b, gg in zip(p, p0, g):
        np.testing.assert_allclose(a, b - 2 * lr * gg / (np.abs(gg) + eps), rtol=1e-12, atol=1e-15)


def test_clipping_makes_update_scale_free():
    # with the clip active the clipped gradient has norm max_grad_norm / (1 +
    # 1e-6 / norm) whatever the raw scale; with eps 0 Adam's step is scale
    # free as well, so scaling every gradient leaves the update unchanged
    rng = np.random.default_rng(5)
    p0 = _tensors(rng, SHAPES)
    g = _tensors(rng, SHAPES)
    z = [np.zeros_like(x) for x in p0]
    a = oracle.adamw_step(p0, g, z, z, 1, 1e-2, 0.9, 0.999, 0.0, 0.0, 1.0)
    b = oracle.adamw_step(p0, [37.0 * x for x in g], z, z, 1, 1e-2, 0.9, 0.999, 0.0, 0.0, 1.0)
    for x, y in zip(a[0], b[0]):
        np.testing.assert_allclose(x, y, rtol=1e-12)
    # clipped moment: m = (1 - beta1) * g * clip / (norm + 1e-6)
    norm = a[3]
    for mm, gg in zip(a[1], g):
        np.testing.assert_allclose(mm, 0.1 * gg / (norm + 1e-6), rtol=1e-12)
    # below the threshold nothing is scaled
    small = [1e-3 * x for x in g]
    c = oracle.adamw_step(p0, small, z, z, 1, 1e-2, 0.9, 0.999, 1e-8, 0.0, 1.0)
    for mm, gg in zip(c[1], small):
        np.testing.assert_allclose(mm, 0.1 * gg, rtol=1e-14)


def test_zero_learning_rate_keeps_parameters():
    rng = np.random.default_rng(6)
    p0 = _tensors(rng, SHAPES)
    g = _tensors(rng, SHAPES)
    z = [np.zeros_like(x) for x in p0]
    p1, m1, _, _ = oracle.adamw_step(p0, g, z, z, 1, 0.0, 0.9, 0.999, 1e-8, 0.5, 0.0)
    for a, b in zip(p1, p0):
        np.testing.assert_array_equal(a, b)
    assert all(np.abs(mm).max() > 0 for mm in m1)
    # weight decay alone (zero gradient) shrinks by exactly 1 - lr wd
    p2, _, _, norm = oracle.adamw_step(p0, z, z, z, 1, 0.1, 0.9, 0.999, 1e-8, 0.5, 1.0)
    assert norm == 0.0
    for a, b in zip(p2, p0):
        np.testing.assert_allclose(a, b * 0.95, rtol=1e-15)


def test_step_must_be_one_based():
    with pytest.raises(ValueError):
        oracle.adamw_step([np.zeros(2)], [np.zeros(2)], [np.zeros(2)], [np.zeros(2)], 0, 1e-3)


def test_train_loop_memorises_a_batch():
    # repeated updates on one batch drive its loss down; the first loss is
    # the plain step's loss, and the loop's parameter bookkeeping is the
    # identity when the learning rate and decay are zero
    cfg = get_config("tiny", n_layer=2)
    g, blocks = synth.make_params(cfg, seed=0)
    tok = synth.make_tokens(cfg, seed=1)
    hp = dict(oracle.ADAMW_PAPER, lr=1e-3)
    r = oracle.train(cfg, g, blocks, [tok] * 6, hp)
    base = oracle.train_step(cfg, g, blocks, tok)["loss"]
    assert abs(r["losses"][0] - base) <= 1e-12 * base
    assert all(b < a for a, b in zip(r["losses"], r["losses"][1:])), r["losses"]
    assert r["losses"][-1] < r["losses"][0] - 0.5
    # clipping is active on this run (norms above 1)
    assert min(r["grad_norms"]) > 1.0
    z = oracle.train(cfg, g, blocks, [tok] * 2, dict(hp, lr=0.0))
    assert z["losses"][0] == z["losses"][1]
    for k in g:
        np.testing.assert_array_equal(z["gparams"][k], np.asarray(g[k], dtype=np.float64))
    for a, b in zip(z["blocks"], blocks):
        for k in b:
            np.testing.assert_array_equal(a[k], np.asarray(b[k], dtype=np.float64))
