"""A whole training step captured as a HIP graph (both streams, and for large
blocks the context's own bias-sum stream; every launch a kernel) replays
bitwise-equal to the eager step, with eager steps and synchronisations
between the replays; and the two-stream step agrees bitwise with the same
step on one stream."""
import numpy as np
import pytest

from paper_2510_14614_amd import fal, synth
from paper_2510_14614_amd.config import ARCH_FAL, ARCH_FALPLUS, ARCH_GPT, SCHED_STREAMS_MERGED, Config

from gpu_helpers import log

pytestmark = pytest.mark.gpu


def _cfg(arch, n_layer, large):
    if large:
        # bias-gradient inputs of 144 MiB per block: their sums run on the
        # context's own stream beside the next block's backward
        return Config(n_layer=n_layer, d_model=1024, n_head=8, head_dim=128, d_ff=4096, vocab=1000, seq_len=1024,
                      batch=8, arch=arch, dtype=1, sched=SCHED_STREAMS_MERGED)
    return Config(n_layer=n_layer, d_model=192, n_head=3, head_dim=64, d_ff=328, vocab=1000, seq_len=100,
                  batch=3, arch=arch, dtype=1, sched=SCHED_STREAMS_MERGED)


@pytest.mark.parametrize("arch,n_layer,large", [(ARCH_FAL, 2, 0), (ARCH_FAL, 1, 0), (ARCH_FALPLUS, 2, 0),
                                                (ARCH_FALPLUS, 9, 0), (ARCH_FAL, 3, 1)])
def test_captured_step_replays_bitwise(arch, n_layer, large):
    import torch
    cfg = _cfg(arch, n_layer, large)
    log(f"graph capture arch={arch} L={n_layer} large={large}")
    g, blocks = synth.make_params(cfg, seed=70)
    tok = torch.from_numpy(synth.make_tokens(cfg, seed=71, dist="zipf")).cuda()
    stream = torch.cuda.Stream()
    F = fal.Fal(cfg, stream_main=stream)
    F.load_params(g, blocks)
    logits = torch.zeros(cfg.tokens, cfg.vocab, device="cuda")
    with torch.cuda.stream(stream):
        F.model_step(tok, logits)
    torch.cuda.synchronize()
    ref = (F.loss.clone(), F.grads.clone(), logits.clone())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        F.model_step(tok, logits)
    torch.cuda.synchronize()
    for k in range(3):
        F.grads.zero_()
        logits.zero_()
        graph.replay()
        torch.cuda.synchronize()
        got = (F.loss.clone(), F.grads.clone(), logits.clone())
        assert all(torch.equal(a, b) for a, b in zip(got, ref)), k
        with torch.cuda.stream(stream):  # eager work between the replays
            F.model_step(tok, logits)
        torch.cuda.synchronize()
        assert torch.equal(F.loss, ref[0])
    del graph
    F.close()


@pytest.mark.parametrize("arch,n_layer,large", [(ARCH_GPT, 3, 1), (ARCH_FAL, 3, 1), (ARCH_FALPLUS, 9, 0)])
def test_two_streams_bitwise_equal_one_stream(arch, n_layer, large):
    # blocks above the bias-sum threshold: with two streams the sums run on
    # the context's own stream beside the next block's backward (and FAL's
    # branches on the aux stream); FAL+'s first-attention terms of layers
    # 8..5 and 4..1 run there as two grouped passes, and layers 3..1 write
    # the dH2 ring slots of layers 8..6 after the first group was joined.
    # On one stream everything runs in order on the main stream.  Loss,
    # logits and every gradient agree bitwise.
    import torch
    cfg = _cfg(arch, n_layer, large)
    log(f"one vs two streams, arch={arch} L={n_layer} large={large}")
    g, blocks = synth.make_params(cfg, seed=72)
    tok = torch.from_numpy(synth.make_tokens(cfg, seed=73, dist="zipf")).cuda()
    outs = []
    for two in (False, True):
        stream = torch.cuda.Stream()
        F = fal.Fal(cfg, stream_main=stream, stream_aux=None if two else stream)
        F.load_params(g, blocks)
        logits = torch.zeros(cfg.tokens, cfg.vocab, device="cuda")
        with torch.cuda.stream(stream):
            F.model_step(tok, logits)
        torch.cuda.synchronize()
        outs.append((F.loss.clone(), F.grads.clone(), logits))
        F.close()
    for a, b in zip(*outs):
        assert torch.equal(a, b)
