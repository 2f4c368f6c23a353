"""Host-only checks of the C ABI (no GPU needed): the library loads, exports
every function include/fal.h declares, validates configs, and reports the
parameter layout and workspace size."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2510_14614_amd import fal, get_config, synth
from paper_2510_14614_amd.config import CONFIGS

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "fal.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(fal_[a-z_]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(fal.ABI_FUNCTIONS)


def test_library_exports_every_declared_symbol():
    lib = fal.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_named_configs_valid(name):
    assert fal.validate_config(get_config(name)) == fal.FAL_OK
    assert fal.workspace_bytes(get_config(name)) > 0


@pytest.mark.parametrize("bad,status", [
    (dict(n_layer=0), fal.FAL_ERR_INVALID_ARG),
    (dict(d_model=60), fal.FAL_ERR_INVALID_ARG),
    (dict(d_ff=0), fal.FAL_ERR_INVALID_ARG),
    (dict(arch=7), fal.FAL_ERR_INVALID_ARG),
    (dict(dtype=3), fal.FAL_ERR_INVALID_ARG),
    (dict(sched=-1), fal.FAL_ERR_INVALID_ARG),
    (dict(ln_eps=0.0), fal.FAL_ERR_INVALID_ARG),
    (dict(fal_block1_mode=2), fal.FAL_ERR_INVALID_ARG),
    (dict(arch=0, fal_block1_mode=1), fal.FAL_ERR_INVALID_ARG),
    (dict(arch=2, fal_block1_mode=1), fal.FAL_ERR_INVALID_ARG),
    (dict(arch=3, fal_block1_mode=1), fal.FAL_ERR_INVALID_ARG),
    (dict(arch=4), fal.FAL_ERR_INVALID_ARG),
    (dict(bidirectional=2, has_embed_head=0), fal.FAL_ERR_INVALID_ARG),
    (dict(bidirectional=1), fal.FAL_ERR_INVALID_ARG),  # needs the block stack
    (dict(n_kv_head=3), fal.FAL_ERR_INVALID_ARG),      # must divide n_head (4)
    (dict(n_kv_head=-1), fal.FAL_ERR_INVALID_ARG),
    (dict(head_dim=24), fal.FAL_ERR_UNSUPPORTED),
    (dict(vocab=70000), fal.FAL_ERR_UNSUPPORTED),
    (dict(d_model=8192), fal.FAL_ERR_UNSUPPORTED),
])
def test_invalid_configs_rejected(bad, status):
    assert fal.validate_config(get_config("tiny", **bad)) == status


def test_fal_block1_mode_accepted_for_fal():
    cfg = get_config("tiny", arch=1, fal_block1_mode=1)
    assert fal.validate_config(cfg) == fal.FAL_OK


def test_param_layout_offsets():
    for name in sorted(CONFIGS):
        cfg = get_config(name)
        lay = fal.param_layout(cfg)
        gs, bs = synth.global_shapes(cfg), synth.block_shapes(cfg)
        spans = []
        if cfg.has_embed_head:
            for k, n in enumerate(fal.GLOBAL_TENSORS):
                o = lay["global"][k]
                assert o % 64 == 0
                spans.append((o, o + int(np.prod(gs[n]))))
        else:
            assert all(o == -1 for o in lay["global"])
        for i in range(cfg.n_layer):
            base = lay["block_base"] + i * lay["block_stride"]
            for k, n in enumerate(fal.BLOCK_TENSORS):
                o = base + lay["block"][k]
                assert o % 64 == 0
                spans.append((o, o + int(np.prod(bs[n]))))
        spans.sort()
        for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
            assert a1 <= b0
        assert spans[-1][1] <= lay["total"]


def test_flatten_roundtrip():
    cfg = get_config("tiny")
    g, blocks = synth.make_params(cfg, seed=0)
    flat = fal.flatten_params(cfg, g, blocks)
    g2, b2 = fal.unflatten(cfg, flat, synth.global_shapes(cfg), synth.block_shapes(cfg))
    for k in g:
        np.testing.assert_array_equal(g[k], g2[k])
    for a, b in zip(blocks, b2):
        for k in a:
            np.testing.assert_array_equal(a[k], b[k])


def test_workspace_grows_with_layers():
    a = fal.workspace_bytes(get_config("tiny", n_layer=2))
    b = fal.workspace_bytes(get_config("tiny", n_layer=4))
    assert b > a


def test_init_rejects_bad_arguments_without_gpu():
    lib = fal.lib()
    c = fal.to_c(get_config("tiny"))
    ctx = ctypes.c_void_p()
    assert lib.fal_init(ctypes.byref(c), None, 0, None, None, ctypes.byref(ctx)) == fal.FAL_ERR_WORKSPACE
    assert lib.fal_init(ctypes.byref(c), None, 0, None, None, None) == fal.FAL_ERR_INVALID_ARG
    bad = fal.to_c(get_config("tiny", head_dim=24))
    assert lib.fal_init(ctypes.byref(bad), None, 0, None, None, ctypes.byref(ctx)) == fal.FAL_ERR_UNSUPPORTED
    assert lib.fal_destroy(None) == fal.FAL_ERR_INVALID_ARG
    assert lib.fal_model_step(None, None, None, None, None, None) == fal.FAL_ERR_INVALID_ARG
    assert lib.fal_block_fwd(None, 0, None, None, None, None) == fal.FAL_ERR_INVALID_ARG
    assert lib.fal_last_error(None) == b""
    assert lib.fal_status_string(fal.FAL_ERR_WORKSPACE) == b"workspace too small"
