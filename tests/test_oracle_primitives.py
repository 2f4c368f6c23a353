"""Pins for the oracle's primitives: closed forms, textbook values, brute
force on tiny inputs and independent library routines (torch, fp64, CPU)."""
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_layer_norm_hand_example():
    # x = [1, 2, 3, 4]: mean 2.5, biased variance 1.25.
    x = np.array([[1.0, 2.0, 3.0, 4.0]])
    y, _ = oracle.layer_norm(x, np.ones(4), np.zeros(4), 0.0)
    expect = np.array([-1.5, -0.5, 0.5, 1.5]) / math.sqrt(1.25)
    np.testing.assert_allclose(y[0], expect, rtol=0, atol=1e-15)


def test_layer_norm_moments_closed_form():
    rng = np.random.default_rng(0)
    x = rng.normal(3.0, 2.0, size=(7, 64))
    eps = 1e-5
    y, _ = oracle.layer_norm(x, np.ones(64), np.zeros(64), eps)
    var = x.var(axis=1)
    np.testing.assert_allclose(y.mean(axis=1), 0.0, atol=1e-14)
    np.testing.assert_allclose(y.var(axis=1), var / (var + eps), rtol=1e-12)


def test_layer_norm_matches_torch():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(5, 32))
    g = 1 + 0.1 * rng.normal(size=32)
    b = 0.1 * rng.normal(size=32)
    dy = rng.normal(size=(5, 32))
    y, cache = oracle.layer_norm(x, g, b, 1e-5)
    dx, dg, db = oracle.layer_norm_backward(dy, cache, g)
    tx = torch.tensor(x, requires_grad=True)
    tg = torch.tensor(g, requires_grad=True)
    tb = torch.tensor(b, requires_grad=True)
    ty = torch.nn.functional.layer_norm(tx, (32,), tg, tb, 1e-5)
    ty.backward(torch.tensor(dy))
    np.testing.assert_allclose(y, ty.detach().numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dg, tg.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(db, tb.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_gelu_erf_against_normal_table():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "normal_cdf.txt")) if l.strip() and not l.startswith("#")]
    for xs, phis in rows:
        x, phi = float(xs), float(phis)
        got = oracle.gelu(np.array([x]), tanh_form=False)[0]
        assert abs(got - x * phi) < 1e-14


def test_gelu_special_values():
    for tf in (True, False):
        assert oracle.gelu(np.array([0.0]), tf)[0] == 0.0
        big = oracle.gelu(np.array([30.0, -30.0]), tf)
        assert big[0] == 30.0
        assert abs(big[1]) < 1e-100
        # derivative at 0 is 1/2 for both forms
        assert abs(oracle.gelu_grad(np.array([0.0]), tf)[0] - 0.5) < 1e-15


@pytest.mark.parametrize("tanh_form", [True, False])
def test_gelu_matches_torch_and_fd(tanh_form):
    x = np.linspace(-6, 6, 241)
    approx = "tanh" if tanh_form else "none"
    ref = torch.nn.functional.gelu(torch.tensor(x), approximate=approx).numpy()
    np.testing.assert_allclose(oracle.gelu(x, tanh_form), ref, rtol=1e-13, atol=1e-15)
    h = 1e-6
    fd = (oracle.gelu(x + h, tanh_form) - oracle.gelu(x - h, tanh_form)) / (2 * h)
    np.testing.assert_allclose(oracle.gelu_grad(x, tanh_form), fd, rtol=1e-7, atol=1e-9)


def _brute_force_attention(q, k, v, causal=True):
    """Explicit loops: o[t] = sum_s exp(q.k_s/sqrt(hd)) v_s / sum exp over
    s <= t (causal) or every s."""
    B, H, T, hd = q.shape
    o = np.zeros_like(q)
    for b in range(B):
        for h in range(H):
            for t in range(T):
                n = t + 1 if causal else T
                scores = [sum(q[b, h, t, c] * k[b, h, s, c] for c in range(hd)) / math.sqrt(hd)
                          for s in range(n)]
                mx = max(scores)
                w = [math.exp(sc - mx) for sc in scores]
                z = sum(w)
                for c in range(hd):
                    o[b, h, t, c] = sum(w[s] * v[b, h, s, c] for s in range(n)) / z
    return o


def test_attention_brute_force():
    rng = np.random.default_rng(2)
    q, k, v = (rng.normal(size=(2, 2, 6, 3)) for _ in range(3))
    o, _ = oracle.causal_attention(q, k, v)
    np.testing.assert_allclose(o, _brute_force_attention(q, k, v), rtol=1e-12, atol=1e-14)


def test_bidirectional_attention_brute_force():
    rng = np.random.default_rng(5)
    q, k, v = (rng.normal(size=(2, 2, 6, 3)) for _ in range(3))
    o, _ = oracle.attention(q, k, v, causal=False)
    np.testing.assert_allclose(o, _brute_force_attention(q, k, v, causal=False), rtol=1e-12, atol=1e-14)
    # the last query sees every key under either mask
    oc, _ = oracle.attention(q, k, v, causal=True)
    np.testing.assert_allclose(o[:, :, -1], oc[:, :, -1], rtol=1e-13, atol=1e-15)
    # identical keys: every query gets the mean of all values
    k = np.repeat(rng.normal(size=(1, 1, 1, 3)), 6, axis=2)
    o, _ = oracle.attention(q[:1, :1], k, v[:1, :1], causal=False)
    np.testing.assert_allclose(o, np.broadcast_to(v[:1, :1].mean(axis=2, keepdims=True), o.shape),
                               rtol=1e-13, atol=1e-15)


def test_bidirectional_attention_matches_torch_sdpa_and_grads():
    rng = np.random.default_rng(6)
    q, k, v, do = (rng.normal(size=(2, 3, 7, 4)) for _ in range(4))
    o, p = oracle.attention(q, k, v, causal=False)
    dq, dk, dv = oracle.causal_attention_backward(do, q, k, v, p)
    tq, tk, tv = (torch.tensor(a, requires_grad=True) for a in (q, k, v))
    to = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=False)
    to.backward(torch.tensor(do))
    np.testing.assert_allclose(o, to.detach().numpy(), rtol=1e-11, atol=1e-13)
    for mine, ref in ((dq, tq), (dk, tk), (dv, tv)):
        np.testing.assert_allclose(mine, ref.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    # T = 1: the only key is the query's own, so O = V.
    q, k, v = (rng.normal(size=(1, 2, 1, 4)) for _ in range(3))
    o, _ = oracle.causal_attention(q, k, v)
    np.testing.assert_array_equal(o, v)
    # identical keys: uniform weights over the visible prefix -> prefix mean of V.
    q = rng.normal(size=(1, 1, 5, 4))
    k = np.repeat(rng.normal(size=(1, 1, 1, 4)), 5, axis=2)
    v = rng.normal(size=(1, 1, 5, 4))
    o, _ = oracle.causal_attention(q, k, v)
    prefix_mean = np.cumsum(v, axis=2) / np.arange(1, 6)[None, None, :, None]
    np.testing.assert_allclose(o, prefix_mean, rtol=1e-13, atol=1e-15)


def test_attention_matches_torch_sdpa_and_grads():
    rng = np.random.default_rng(4)
    q, k, v, do = (rng.normal(size=(2, 3, 7, 4)) for _ in range(4))
    o, p = oracle.causal_attention(q, k, v)
    dq, dk, dv = oracle.causal_attention_backward(do, q, k, v, p)
    tq, tk, tv = (torch.tensor(a, requires_grad=True) for a in (q, k, v))
    to = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    to.backward(torch.tensor(do))
    np.testing.assert_allclose(o, to.detach().numpy(), rtol=1e-11, atol=1e-13)
    for mine, ref in ((dq, tq), (dk, tk), (dv, tv)):
        np.testing.assert_allclose(mine, ref.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_cross_entropy_closed_forms():
    V = 37
    logits = np.zeros((4, V))
    targets = np.array([0, 5, 36, 7])
    loss, dl = oracle.cross_entropy(logits, targets)
    assert abs(loss - math.log(V)) < 1e-14
    np.testing.assert_allclose(dl.sum(axis=1), 0.0, atol=1e-16)
    rng = np.random.default_rng(5)
    logits = rng.normal(size=(6, V)) * 3
    targets = rng.integers(0, V, size=6)
    loss, dl = oracle.cross_entropy(logits, targets)
    tl = torch.tensor(logits, requires_grad=True)
    tloss = torch.nn.functional.cross_entropy(tl, torch.tensor(targets))
    tloss.backward()
    assert abs(loss - tloss.item()) < 1e-13
    np.testing.assert_allclose(dl, tl.grad.numpy(), rtol=1e-11, atol=1e-15)
    np.testing.assert_allclose(dl.sum(axis=1), 0.0, atol=1e-15)
