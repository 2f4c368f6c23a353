"""fal_adamw_step_noalloc -- the AdamW update with no context and no device
allocation (its scratch is a fixed array in the library, one per GPU) --
against fal_adamw_step through the C ABI on the same inputs.

The two entry points run the same kernels in the same order, so weights,
weight copy, moments and norm must agree bitwise (stronger than the fp32
tolerances of the oracle comparison in the optimizer tests, which the
existing entry point meets).  Two calls in a row, the second with a smaller
buffer and clipping in the other state: the scratch keeps the first call's
contents, and nothing of it may leak into the second.
"""
from ctypes import byref, c_void_p

import numpy as np
import pytest

from paper_2510_14614_amd import fal, get_config, synth

from gpu_helpers import log

pytestmark = pytest.mark.gpu

HP = dict(lr=1e-2, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1, max_grad_norm=1.0)


def _ptr(t):
    return c_void_p(t.data_ptr()) if t is not None else None


def _state(n, seed, lp_mode):
    """Two identical device copies of (master, params, grads, m, v, norm)."""
    import torch
    p0 = synth.make_flat(n, seed=seed)
    m0 = synth.make_flat(n, seed=seed + 1, scale=1e-3)
    v0 = m0 * m0 + synth.make_flat(n, seed=seed + 2, scale=1e-7, positive=True)
    # gradient norm about 10 (clipping active) for even seeds, 0.1 (inactive) for odd
    g0 = synth.make_flat(n, seed=seed + 3, scale=(10.0 if seed % 2 == 0 else 0.1) / np.sqrt(max(n, 1)))
    out = []
    for _ in range(2):
        master = torch.from_numpy(p0.copy()).cuda()
        if lp_mode == "bf16":
            params = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
        elif lp_mode == "f32_copy":
            params = torch.zeros(n, dtype=torch.float32, device="cuda")
        else:
            params = None
        out.append({"master": master, "params": params, "grads": torch.from_numpy(g0.copy()).cuda(),
                    "m": torch.from_numpy(m0.copy()).cuda(), "v": torch.from_numpy(v0.copy()).cuda(),
                    "norm": torch.full((1,), -1.0, dtype=torch.float32, device="cuda")})
    return out


@pytest.mark.parametrize("lp_mode", ["bf16", "f32_copy", "f32_inplace"])
def test_noalloc_adamw_bitwise_equals_context_entry_point(lp_mode):
    import torch
    dtype = 1 if lp_mode == "bf16" else 0
    F = fal.Fal(get_config("tiny", dtype=dtype))
    stream = torch.cuda.current_stream()
    # two calls in a row: 5,000,003 elements (more than one sweep of the norm
    # grid, ragged tail), then 1,048,579 (fewer, clipping off)
    for call, (n, seed, step) in enumerate([(5_000_003, 200, 3), (1_048_579, 301, 4)]):
        log(f"no-alloc adamw call {call} n={n} mode={lp_mode}")
        ref, got = _state(n, seed, lp_mode)
        hp = fal.adamw_params(**HP)
        st = fal.lib().fal_adamw_step(F.ctx, byref(hp), step, n, _ptr(ref["master"]), _ptr(ref["params"]),
                                      _ptr(ref["grads"]), _ptr(ref["m"]), _ptr(ref["v"]), _ptr(ref["norm"]))
        assert st == fal.FAL_OK, fal.lib().fal_last_error(F.ctx)
        st = fal.lib().fal_adamw_step_noalloc(byref(hp), step, n, dtype, _ptr(got["master"]), _ptr(got["params"]),
                                              _ptr(got["grads"]), _ptr(got["m"]), _ptr(got["v"]), _ptr(got["norm"]),
                                              c_void_p(stream.cuda_stream))
        assert st == fal.FAL_OK, fal.lib().fal_last_error(None)
        torch.cuda.synchronize()
        for k in ("master", "params", "m", "v", "norm"):
            if ref[k] is None:
                continue
            assert torch.equal(ref[k], got[k]), (call, k)
        # the update did happen (the weights moved), and the norm is the one
        # of this call's gradient, not a leftover of the previous call
        assert not torch.equal(got["master"], torch.from_numpy(synth.make_flat(n, seed=seed)).cuda())
        gn = float(torch.linalg.vector_norm(got["grads"].double()).item())
        assert abs(got["norm"].item() - gn) <= 1e-6 * gn
    F.close()


def test_noalloc_adamw_binding_and_argument_errors():
    import torch
    n = 4099
    ref, got = _state(n, 400, "bf16")
    hp = fal.adamw_params(**HP)
    F = fal.Fal(get_config("tiny", dtype=1))
    assert fal.lib().fal_adamw_step(F.ctx, byref(hp), 1, n, _ptr(ref["master"]), _ptr(ref["params"]),
                                    _ptr(ref["grads"]), _ptr(ref["m"]), _ptr(ref["v"]),
                                    _ptr(ref["norm"])) == fal.FAL_OK
    # through the Python binding, on a stream of its own
    s = torch.cuda.Stream()
    fal.adamw_step_noalloc(hp, 1, n, 1, got["master"], got["params"], got["grads"], got["m"], got["v"],
                           got["norm"], stream=s)
    torch.cuda.synchronize()
    for k in ("master", "params", "m", "v", "norm"):
        assert torch.equal(ref[k], got[k]), k
    # errors come back before anything is launched, with a message
    with pytest.raises(fal.FalError) as e:
        fal.adamw_step_noalloc(hp, 0, n, 1, got["master"], got["params"], got["grads"], got["m"], got["v"])
    assert e.value.status == fal.FAL_ERR_INVALID_ARG and "1-based" in str(e.value)
    with pytest.raises(fal.FalError) as e:
        fal.adamw_step_noalloc(hp, 1, n, 1, got["master"], None, got["grads"], got["m"], got["v"])
    assert e.value.status == fal.FAL_ERR_INVALID_ARG
    F.close()
