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


@pytest.mark.parametrize("name", ["tiny", "gpt2-small", "gpt-1.3b"])
def test_falplus_workspace_holds_the_side_pass_ring(name):
    # FAL+ keeps the MLP-input gradient dH2 of up to four consecutive blocks
    # for the grouped first-attention pass (a ring of five fp32 [M, d]
    # buffers, four beyond the one every architecture has) plus that pass's
    # partial sums (four blocks x one row per 32 rows x d fp32); otherwise
    # its workspace is the GPT one
    from paper_2510_14614_amd.config import ARCH_FALPLUS, ARCH_GPT
    gpt = get_config(name, arch=ARCH_GPT)
    fp = get_config(name, arch=ARCH_FALPLUS)
    M, d = gpt.tokens, gpt.d_model
    extra = 4 * M * d * 4 + 4 * ((M + 31) // 32) * d * 4
    diff = fal.workspace_bytes(fp) - fal.workspace_bytes(gpt)
    assert extra <= diff <= extra + 5 * 256, (diff, extra)


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
    assert lib.fal_block_bwd(None, 0, None, None, None, None, None, None, None) == fal.FAL_ERR_INVALID_ARG
    assert lib.fal_last_error(None) == b""
    assert lib.fal_status_string(fal.FAL_ERR_WORKSPACE) == b"workspace too small"


def test_gemm_operand_extent_limit():
    # The bf16 GEMM kernels address operands with 32-bit offsets: a block
    # stack whose [M, dA + f] activations (with the 256-row read-ahead of a
    # weight-gradient operand) would reach 2 GiB is rejected as unsupported,
    # one just below the limit is accepted.  d 1024, dA 1024, f 4096: rows of
    # 10240 bytes in bf16, so the limit lies at M + 256 = 209612 rows.
    base = dict(n_layer=4, d_model=1024, n_head=16, head_dim=64, d_ff=4096, vocab=0, seq_len=2048,
                arch=1, dtype=1, has_embed_head=0)
    from paper_2510_14614_amd.config import Config
    assert fal.validate_config(Config(batch=102, **base)) == fal.FAL_OK          # M = 208896
    assert fal.validate_config(Config(batch=103, **base)) == fal.FAL_ERR_UNSUPPORTED  # M = 210944
    assert fal.validate_config(Config(batch=128, **base)) == fal.FAL_ERR_UNSUPPORTED  # M = 262144
    # with the LM head the logits [M, V] (V padded to 65536) are the widest
    # operand: 15616 x 65536 x 2 bytes fit, 16640 x 65536 x 2 do not
    lm = dict(n_layer=1, d_model=64, n_head=1, head_dim=64, d_ff=64, vocab=65535, seq_len=1024, arch=1, dtype=1)
    assert fal.validate_config(Config(batch=15, **lm)) == fal.FAL_OK
    assert fal.validate_config(Config(batch=16, **lm)) == fal.FAL_ERR_UNSUPPORTED
    # fp32 parity mode indexes with 64 bits and is not limited this way
    assert fal.validate_config(Config(batch=103, **{**base, "dtype": 0})) == fal.FAL_OK


def test_noalloc_adamw_rejects_bad_arguments_without_gpu():
    # argument errors return before any HIP call, with a message readable
    # through fal_last_error(NULL)
    from ctypes import byref
    lib = fal.lib()
    hp = fal.adamw_params()
    assert lib.fal_adamw_step_noalloc(None, 1, 0, 1, None, None, None, None, None, None, None) == \
        fal.FAL_ERR_INVALID_ARG
    assert b"hyper-parameters" in lib.fal_last_error(None)
    assert lib.fal_adamw_step_noalloc(byref(hp), 1, 0, 7, None, None, None, None, None, None, None) == \
        fal.FAL_ERR_INVALID_ARG
    assert lib.fal_last_error(None) == b"unknown dtype"
    assert lib.fal_adamw_step_noalloc(byref(hp), 0, 0, 1, None, None, None, None, None, None, None) == \
        fal.FAL_ERR_INVALID_ARG
    assert lib.fal_adamw_step_noalloc(byref(hp), 1, -1, 1, None, None, None, None, None, None, None) == \
        fal.FAL_ERR_INVALID_ARG
    assert lib.fal_adamw_step_noalloc(byref(hp), 1, 2048 * 0x7fffffff + 1, 0, None, None, None, None, None, None,
                                      None) == fal.FAL_ERR_INVALID_ARG
    assert b"grid limit" in lib.fal_last_error(None)
    bad = fal.adamw_params(beta1=1.0)
    assert lib.fal_adamw_step_noalloc(byref(bad), 1, 0, 1, None, None, None, None, None, None, None) == \
        fal.FAL_ERR_INVALID_ARG
