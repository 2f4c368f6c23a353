"""A whole training step captured as a HIP graph (both streams, every launch
a kernel) replays bitwise-equal to the eager step, with eager steps and
synchronisations between the replays."""
import numpy as np
import pytest

from paper_2510_14614_amd import fal, synth
from paper_2510_14614_amd.config import ARCH_FAL, ARCH_FALPLUS, SCHED_STREAMS_MERGED, Config

from gpu_helpers import log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("arch,n_layer", [(ARCH_FAL, 2), (ARCH_FAL, 1), (ARCH_FALPLUS, 2)])
def test_captured_step_replays_bitwise(arch, n_layer):
    import torch
    cfg = Config(n_layer=n_layer, d_model=192, n_head=3, head_dim=64, d_ff=328, vocab=1000, seq_len=100,
                 batch=3, arch=arch, dtype=1, sched=SCHED_STREAMS_MERGED)
    log(f"graph capture arch={arch} L={n_layer}")
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
