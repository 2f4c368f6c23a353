"""Training-step throughput of the FAL hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config gpt2-small]
                    [--arch fal] [--sched streams_merged] [--no-compare] [--no-cpu-baseline]
                    [--single-stream]

One step = one full forward + backward of the language model (embedding,
every block, final LayerNorm, tied LM head, cross-entropy) through
libfal's fal_model_step (or fal_stack_step for the block-stack shard
workload) on a fixed batch of synthetic tokens already resident in HBM.
W untimed warm-up steps, then exactly K timed steps bracketed by
synchronisation.  Prints one JSON line.

Also reported, from the same process:
  * roofline of the dominant kernel class (the bf16 MFMA GEMMs): algorithmic
    FLOPs / summed launch time, both from HIP events the library records on
    the stream each GEMM runs on, during K more steps of the same schedule
    run with the aux stream equal to the main stream (identical launches,
    no overlap between kernels, so each span times one kernel);
  * the same-kernel sequential GPT baseline and FAL+ on the same config
    (tokens/s and the ratio to it);
  * cpu_baseline: the fp64 CPU oracle timed on this host on a bounded sample
    (batch 1 of the same config).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "training tokens/s on 1 MI355X (FAL vs GPT baseline); MFMA util % of bf16 peak"
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="gpt2-small")
    ap.add_argument("--arch", default="fal", choices=["gpt", "fal", "falplus", "fal+"])
    ap.add_argument("--sched", default="streams_merged", choices=["seq", "streams", "merged", "streams_merged"])
    ap.add_argument("--no-compare", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-batch", type=int, default=1)
    ap.add_argument("--single-stream", action="store_true",
                    help="run the timed steps with the aux stream equal to the main stream")
    return ap.parse_args()


def describe(cfg, arch_name, sched_name):
    return (f"{arch_name} training step, L{cfg.n_layer} d{cfg.d_model} H{cfg.n_head}x{cfg.head_dim} "
            f"f{cfg.d_ff} V{cfg.vocab} T{cfg.seq_len} B{cfg.batch}, bf16 storage / fp32 accumulate, "
            f"{sched_name} schedule")


class Runner:
    def __init__(self, cfg, single_stream=False):
        import torch

        from paper_2510_14614_amd import fal, synth
        self.torch = torch
        self.cfg = cfg
        main = torch.cuda.current_stream()
        self.F = fal.Fal(cfg, stream_main=main, stream_aux=main if single_stream else None)
        g, blocks = synth.make_params(cfg, seed=0, mode="throughput")
        self.F.load_params(g, blocks)
        if cfg.has_embed_head:
            tok = synth.make_tokens(cfg, seed=1)
            self.tok = torch.from_numpy(tok).cuda()
        else:
            x1, gout = synth.make_stack_inputs(cfg, seed=2)
            self.x1 = torch.from_numpy(x1).cuda()
            self.dy = torch.from_numpy(gout).cuda()
            self.dx = torch.empty_like(self.x1)

    def step(self):
        if self.cfg.has_embed_head:
            self.F.model_step(self.tok)
        else:
            self.F.stack_step(self.x1, self.dy, self.dx)

    def time(self, steps, warmup):
        torch = self.torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        s = self.F.stream_main
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(s)
        t0 = time.perf_counter()
        for _ in range(steps):
            self.step()
        e1.record(s)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = e0.elapsed_time(e1) / steps
        return ms, wall

    def profile(self, steps):
        self.F.profile_enable(True)
        for _ in range(steps):
            self.step()
        self.torch.cuda.synchronize()
        prof = self.F.profile_read()
        self.F.profile_enable(False)
        return prof

    def close(self):
        self.F.close()


def cpu_baseline(cfg, sample_batch):
    """Time the fp64 oracle on `sample_batch` sequences of the same config."""
    import numpy as np
    import threadpoolctl

    import oracle
    from paper_2510_14614_amd import synth
    sc = cfg.replace(batch=sample_batch, dtype=0)
    g, blocks = synth.make_params(cfg, seed=0, mode="throughput")
    threads = max((p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()), default=1)
    t0 = time.perf_counter()
    if sc.has_embed_head:
        tok = synth.make_tokens(sc, seed=1)
        oracle.train_step(sc, g, blocks, tok)
    else:
        x1, gout = synth.make_stack_inputs(sc, seed=2)
        oracle.stack_step(sc, blocks, x1, gout)
    sec = time.perf_counter() - t0
    return {"value": sc.tokens / sec, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"one fwd+bwd step of the same model at batch {sample_batch} "
                      f"({sc.tokens} tokens), numpy float64, {sec:.1f} s",
            "host_cpus": os.cpu_count()}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported by this build "
              f"(the hot path is single-GPU; see the sharding notes in DESIGN.md).", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2510_14614_amd import get_config
    from paper_2510_14614_amd.config import ARCH_NAMES, SCHED_NAMES, SCHED_SEQ

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    arch = ARCH_NAMES[args.arch]
    sched = SCHED_NAMES[args.sched]
    cfg = get_config(args.config, arch=arch, sched=sched, dtype=1)

    r = Runner(cfg, single_stream=args.single_stream)
    ms, wall = r.time(args.steps, args.warmup)
    r.close()
    # Kernel roofline from a serialized pass (aux stream = main stream: the
    # same launches without overlap, so each event span is one kernel alone).
    rp = Runner(cfg, single_stream=True)
    rp.time(1, 1)
    prof = rp.profile(args.steps)
    rp.close()
    tokens_per_s = cfg.tokens / (ms / 1000.0)
    flops_step = cfg.train_flops_per_token() * cfg.tokens

    g = prof["gemm"]
    gemm_avg_ms = g["ms"] / max(g["launches"], 1)
    gemm_tflops = g["flops"] / (g["ms"] / 1000.0) / 1e12 if g["ms"] > 0 else 0.0
    kernels = {}
    for name, p in prof.items():
        if p["launches"] == 0:
            continue
        ent = {"launches_per_step": p["launches"] / args.steps, "ms_per_step": p["ms"] / args.steps}
        if p["flops"] > 0:
            ent["TFLOP/s"] = p["flops"] / (p["ms"] / 1000.0) / 1e12
            ent["frac_bf16_peak"] = ent["TFLOP/s"] / PEAK_BF16_TFLOPS
        if p["bytes"] > 0 and p["flops"] == 0:
            ent["GB/s"] = p["bytes"] / (p["ms"] / 1000.0) / 1e9
            ent["frac_hbm_peak"] = ent["GB/s"] / PEAK_HBM_GBS
        kernels[name] = ent

    out = {
        "metric": METRIC,
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (Zipf(1.1) token ids, N(0,0.02) weights)",
        "config": {"workload": describe(cfg, args.arch.upper(), args.sched), "name": args.config,
                   "global_batch": cfg.batch, "seq_len": cfg.seq_len, "parallelism": "single GPU"},
        "mfu": flops_step / (ms / 1000.0) / 1e12 / PEAK_BF16_TFLOPS,
        "roofline": {
            "bound": "mfma",
            "kernel": "gemm_bf16_mfma (all bf16 GEMM launches of the step)",
            "achieved": gemm_tflops,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": gemm_tflops / PEAK_BF16_TFLOPS,
            "traffic": None,
            "avg_launch_ms": gemm_avg_ms,
            "avg_launch_gflop": g["flops"] / max(g["launches"], 1) / 1e9,
        },
        "kernels": kernels,
        "wall_s_timed": wall,
    }

    if not args.no_compare:
        comp = {}
        for name, a, s in (("gpt_seq", "gpt", SCHED_SEQ), ("falplus_seq", "falplus", SCHED_SEQ)):
            if ARCH_NAMES[a] == arch:
                continue
            c2 = cfg.replace(arch=ARCH_NAMES[a], sched=s)
            r2 = Runner(c2)
            ms2, _ = r2.time(args.steps, args.warmup)
            r2.close()
            comp[name] = {"tokens_per_s": c2.tokens / (ms2 / 1000.0), "ms_per_step": ms2}
        if "gpt_seq" in comp:
            comp["speedup_over_gpt_same_kernels"] = tokens_per_s / comp["gpt_seq"]["tokens_per_s"]
        comp["paper_context"] = ("paper: FAL single-GPU throughput up to 1.18x (1.08x average) over "
                                 "GPT-2 774M on RTX 3090/4090/A6000; context, not the target")
        out["comparison"] = comp

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_sample_batch)

    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
