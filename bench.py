"""Training-step throughput of the FAL hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config gpt-1.3b]
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
  * the same-kernel sequential GPT baseline, FAL+, and the parallel block
    (same schedule as the measured run) on the same config
    (tokens/s and the ratio to it);
  * training_with_optimizer: the same step followed by the AdamW update of
    every parameter (tokens/s and the update's own time and bandwidth);
  * forward_only: the forward step without gradients (fal_model_forward /
    fal_stack_forward), this architecture and the sequential GPT;
  * cpu_baseline: the fp64 CPU oracle timed on this host on a bounded sample:
    one training step of one sequence through the full-width model with one
    and with two blocks (full vocabulary), the full-depth step time
    extrapolated linearly in the block count.

The default workload is the ~1.3B GPT shape (24 blocks, d 2048, 16 heads of
128, FFN 8192, vocabulary 50257, T 2048, B 4) in the FAL architecture, the
configuration at which FAL is compared with the same-kernel GPT baseline.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "training tokens/s on 1 MI355X (FAL vs GPT baseline); MFMA util % of bf16 peak"
# Measured HBM traffic of the GEMM calls of a workload (rocprofv3
# FETCH_SIZE / WRITE_SIZE, calibrated on a plain copy), one file per config
# and architecture; valid only while the sources it was measured on are
# unchanged.
TRAFFIC_DIR = os.path.join(ROOT, "profiles")


def traffic_file(config, arch):
    return os.path.join(TRAFFIC_DIR, f"gemm_bf16_{config}_{arch}_traffic.md")


TRAFFIC_SOURCES = ("paper_2510_14614_amd/csrc/gemm.hip", "paper_2510_14614_amd/csrc/kernels.h",
                   "paper_2510_14614_amd/csrc/common.h")
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="gpt-1.3b")
    ap.add_argument("--arch", default="fal", choices=["gpt", "fal", "falplus", "fal+", "parallel"])
    ap.add_argument("--sched", default="streams_merged", choices=["seq", "streams", "merged", "streams_merged"])
    ap.add_argument("--no-compare", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-optimizer", action="store_true",
                    help="skip the extra measurement of step + AdamW update")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of the step captured as a HIP graph instead of eager launches")
    ap.add_argument("--no-forward", action="store_true",
                    help="skip the extra forward-only measurement (FAL and GPT)")
    ap.add_argument("--single-stream", action="store_true",
                    help="run the timed steps with the aux stream equal to the main stream")
    ap.add_argument("--summarize-stats", nargs=2, metavar=("STATS_CSV", "OUT_MD"),
                    help="offline: write a kernel summary from a rocprofv3 --stats kernel_stats.csv")
    ap.add_argument("--summarize-mfma", nargs=3, metavar=("PMC_CSV", "TRACE_CSV", "OUT_MD"),
                    help="offline: write the MFMA-utilisation summary from a rocprofv3 --pmc "
                         "SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_VALU_MFMA_BUSY_CYCLES "
                         "counter_collection.csv and the kernel_trace.csv of the same run")
    ap.add_argument("--summarize-hbm", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "PROBE_MIB", "OUT_MD"),
                    help="offline: write HBM bytes and GB/s per kernel class from two rocprofv3 "
                         "--kernel-trace --pmc runs (FETCH_SIZE, WRITE_SIZE) made with --copy-probe PROBE_MIB")
    ap.add_argument("--summarize-traffic", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "PROBE_MIB", "OUT_MD"),
                    help="offline: write the GEMM traffic summary from two rocprofv3 --pmc counter_collection.csv "
                         "of runs made with --copy-probe PROBE_MIB")
    ap.add_argument("--cmd", action="append", default=[], help="command line(s) recorded in a summary")
    ap.add_argument("--label", default="gpt-1.3b FAL", help="workload named in a summary's title")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="after the measurements, run one plain device copy of MIB MiB (fp32 x 2.0 into a second "
                         "buffer): the known-size reference for HBM traffic counters")
    return ap.parse_args()


def describe(cfg, arch_name, sched_name):
    mask = "bidirectional attention" if cfg.bidirectional else "causal attention"
    return (f"{arch_name} training step, L{cfg.n_layer} d{cfg.d_model} H{cfg.n_head}x{cfg.head_dim} "
            f"f{cfg.d_ff} V{cfg.vocab} T{cfg.seq_len} B{cfg.batch}, {mask}, bf16 storage / fp32 accumulate, "
            f"{sched_name} schedule")


_INPUTS = {}


def device_inputs(cfg):
    """Synthetic parameters (flat, in the library's layout and the config's
    dtype) and token ids or block-stack inputs, on the GPU.  Drawn once per
    model shape: the layout does not depend on the block architecture or the
    schedule, so every leg of the bench reuses the same device copies."""
    import torch

    from paper_2510_14614_amd import fal, synth
    key = (cfg.n_layer, cfg.d_model, cfg.n_head, cfg.head_dim, cfg.d_ff, cfg.vocab, cfg.seq_len, cfg.batch,
           cfg.dtype, cfg.has_embed_head, cfg.n_kv_head)
    if key not in _INPUTS:
        g, blocks = synth.make_params(cfg, seed=0, mode="throughput")
        flat = torch.from_numpy(fal.flatten_params(cfg, g, blocks))
        del g, blocks
        pdtype = torch.bfloat16 if cfg.dtype == 1 else torch.float32
        ent = {"params": flat.to(pdtype).cuda()}
        del flat
        if cfg.has_embed_head:
            ent["tok"] = torch.from_numpy(synth.make_tokens(cfg, seed=1)).cuda()
        else:
            x1, gout = synth.make_stack_inputs(cfg, seed=2)
            ent["x1"] = torch.from_numpy(x1).cuda()
            ent["dy"] = torch.from_numpy(gout).cuda()
        _INPUTS[key] = ent
    return _INPUTS[key]


class Runner:
    def __init__(self, cfg, single_stream=False, optimizer=False, forward_only=False, graph=False):
        import torch

        from paper_2510_14614_amd import fal
        self.torch = torch
        self.cfg = cfg
        self.optimizer = optimizer
        self.forward_only = forward_only
        self.hp = fal.ADAMW_PAPER
        # a graph is captured on a stream of its own, which the context must use
        main = torch.cuda.Stream() if graph else torch.cuda.current_stream()
        self.F = fal.Fal(cfg, stream_main=main, stream_aux=main if single_stream else None)
        self.graph = None
        inp = device_inputs(cfg)
        self.F.params.copy_(inp["params"])
        if cfg.has_embed_head:
            self.tok = inp["tok"]
        else:
            self.x1 = inp["x1"]
            self.dy = inp["dy"]
            self.dx = torch.empty_like(self.x1)
        if optimizer:
            self.F.init_optimizer()
        if graph:
            self.capture()

    def capture(self):
        """Records one whole step (every launch of both streams) as a HIP graph
        and replays it from then on: the same kernels, without the per-launch
        host work and dispatch gaps."""
        torch = self.torch
        with torch.cuda.stream(self.F.stream_main):
            for _ in range(2):
                self.launch()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=self.F.stream_main):
            self.launch()
        torch.cuda.synchronize()
        self.graph = g

    def step(self):
        if self.graph is not None:
            self.graph.replay()
            return
        self.launch()

    def launch(self):
        if self.forward_only:
            if self.cfg.has_embed_head:
                self.F.model_forward(self.tok)
            else:
                self.F.stack_forward(self.x1)
            return
        if self.cfg.has_embed_head:
            self.F.model_step(self.tok)
        else:
            self.F.stack_step(self.x1, self.dy, self.dx)
        if self.optimizer:
            self.F.adamw_step(**self.hp)

    def time(self, steps, warmup):
        torch = self.torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        s = self.F.stream_main if self.graph is None else torch.cuda.current_stream()
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


def measured_peaks():
    """Sustained dense bf16 MFMA rate (register-only MFMA chains on every
    SIMD, libfal_probe.so) and HBM copy rate (1 GiB read + 1 GiB written by
    one elementwise kernel), both timed with HIP events."""
    import ctypes

    import torch
    path = os.path.join(ROOT, "paper_2510_14614_amd", "libfal_probe.so")
    L = ctypes.CDLL(path)
    L.fal_probe_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    blocks, iters = 8 * 256, 4096
    out = torch.empty(blocks * 256, device="cuda", dtype=torch.float32)
    s = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for rep in range(2):  # first launch warms up
        e0.record(s)
        assert L.fal_probe_mfma_bf16(blocks, iters, ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(s.cuda_stream)) == 0
        e1.record(s)
        torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    flops = blocks * 4.0 * iters * L.fal_probe_mfma_chains() * 2 * 16 * 16 * 32
    n = (1 << 30) // 4
    src = torch.ones(n, device="cuda", dtype=torch.float32)
    dst = torch.empty_like(src)
    for rep in range(3):
        e0.record(s)
        torch.mul(src, 2.0, out=dst)
        e1.record(s)
        torch.cuda.synchronize()
    cms = e0.elapsed_time(e1)
    return {"mfma_bf16_tflops": flops / (ms / 1e3) / 1e12, "hbm_copy_gbs": 2.0 * n * 4 / (cms / 1e3) / 1e9}


def cpu_baseline(cfg):
    """Time the fp64 oracle on a bounded sample of the workload: one training
    step of one sequence through the full-width model (full vocabulary) with
    one block and with two blocks.  The full-depth step time of one sequence
    is extrapolated linearly in the block count, t1 + (L - 1) (t2 - t1), and
    reported as tokens/s."""
    import threadpoolctl

    import oracle
    from paper_2510_14614_amd import synth
    threads = max((p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()), default=1)
    times = []
    for nl in (1, 2):
        sc = cfg.replace(batch=1, dtype=0, n_layer=nl)
        g, blocks = synth.make_params(sc, seed=0, mode="throughput")
        if sc.has_embed_head:
            tok = synth.make_tokens(sc, seed=1)
            t0 = time.perf_counter()
            oracle.train_step(sc, g, blocks, tok)
        else:
            x1, gout = synth.make_stack_inputs(sc, seed=2)
            t0 = time.perf_counter()
            oracle.stack_step(sc, blocks, x1, gout)
        times.append(time.perf_counter() - t0)
    t1, t2 = times
    per_block = max(t2 - t1, 0.0)
    est = t1 + (cfg.n_layer - 1) * per_block
    return {"value": cfg.seq_len / est, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"one fwd+bwd step of one sequence ({cfg.seq_len} tokens), numpy float64, full width "
                      f"and vocabulary, with 1 block ({t1:.1f} s) and 2 blocks ({t2:.1f} s); the "
                      f"{cfg.n_layer}-block step extrapolated linearly in the block count: {est:.1f} s",
            "host_cpus": os.cpu_count()}


def sources_hash():
    h = hashlib.sha256()
    for rel in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(config, arch):
    """Bytes per GEMM call from the committed counter summary of this config
    and architecture, or None when it is missing or was taken on different
    kernel sources."""
    try:
        lines = open(traffic_file(config, arch)).read().splitlines()
    except OSError:
        return None
    kv = {}
    for ln in lines:
        if ln.startswith("- `") and "`: " in ln:
            k, v = ln[3:].split("`: ", 1)
            kv[k] = v.strip()
    if kv.get("gemm_sources_sha256") != sources_hash():
        return None
    try:
        return float(kv["traffic_bytes_per_call"])
    except (KeyError, ValueError):
        return None


def summarize_stats(stats_csv, out_md, cmds, label):
    rows = list(csv.DictReader(open(stats_csv)))
    tot = sum(float(r["TotalDurationNs"]) for r in rows)
    lines = [f"# Kernel time, {label} training step (serialized launches)", "",
             "Command (repository root on the GPU host, `TMPDIR=/tmp`):", ""]
    lines += ["```", *cmds, "```", "",
              f"All dispatches of the run; total GPU kernel time {tot / 1e6:.2f} ms.", "",
              "| kernel | calls | avg us | total ms | % |", "|---|---|---|---|---|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        ms = float(r["TotalDurationNs"]) / 1e6
        if ms < 0.05:
            continue
        name = r["Name"].replace("|", "/")[:110]
        lines.append(f"| `{name}` | {int(r['Calls'])} | {float(r['AverageNs']) / 1e3:.1f} | {ms:.2f} | "
                     f"{float(r['Percentage']):.1f} |")
    gm = [r for r in rows if "gemm_bf16_" in r["Name"]]
    red = [r for r in rows if "splitk_reduce" in r["Name"]]
    n = sum(int(r["Calls"]) for r in gm)
    tg = sum(float(r["TotalDurationNs"]) for r in gm)
    tr = sum(float(r["TotalDurationNs"]) for r in red)
    lines += ["", f"bf16 GEMM kernels (all instantiations): {n} calls, average {tg / n / 1e3:.1f} us per call; "
              f"with the split-K reduces they launch, {(tg + tr) / n / 1e3:.1f} us per call (the span bench.py "
              f"times as one GEMM call)."]
    open(out_md, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines[-3:]))


def summarize_traffic(fetch_csv, write_csv, probe_mib, out_md, cmds, label):
    probe_bytes = int(probe_mib) * (1 << 20)

    def load(path, counter):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        probe = [r for r in rows if "MulFunctor" in r["Kernel_Name"]]
        assert probe, "no copy-probe dispatch in " + path
        calib = probe_bytes / (float(probe[-1]["Counter_Value"]) * 1024.0)
        g = [float(r["Counter_Value"]) * 1024.0 for r in rows if "gemm_bf16_" in r["Kernel_Name"]]
        red = [float(r["Counter_Value"]) * 1024.0 for r in rows if "splitk_reduce" in r["Kernel_Name"]]
        return calib, probe_bytes, float(probe[-1]["Counter_Value"]) * 1024.0, g, red, len(rows)
    cf, pbf, rawf, gf, rf, _ = load(fetch_csv, "FETCH_SIZE")
    cw, pbw, raww, gw, rw, _ = load(write_csv, "WRITE_SIZE")
    n = len(gf)
    assert n == len(gw) and n > 0
    fetch = (sum(gf) + sum(rf)) * cf / n
    write = (sum(gw) + sum(rw)) * cw / n
    lines = [f"# HBM traffic of the bf16 GEMM kernels, {label} training step", "",
             "Commands (repository root on the GPU host, `TMPDIR=/tmp`), one counter per run:", "",
             "```", *cmds, "```", "",
             "Each run ends with a plain elementwise copy (`--copy-probe`) that reads and writes a known number",
             "of bytes; its counter reading calibrates the counter for this part:", "",
             f"- FETCH_SIZE: copy of {pbf / 2**20:.0f} MiB read {rawf / 2**20:.1f} MiB -> factor {cf:.4f}",
             f"- WRITE_SIZE: copy of {pbw / 2**20:.0f} MiB wrote {raww / 2**20:.1f} MiB -> factor {cw:.4f}", "",
             f"Over {n} GEMM calls (each call = one bf16 GEMM dispatch plus the split-K reduce it may launch):", "",
             f"- `fetch_bytes_per_call`: {fetch:.0f}",
             f"- `write_bytes_per_call`: {write:.0f}",
             f"- `traffic_bytes_per_call`: {fetch + write:.0f}",
             f"- `gemm_sources_sha256`: {sources_hash()}", "",
             "bench.py reports `traffic_bytes_per_call` as roofline.traffic while the kernel sources hash to the",
             "value above, and null otherwise."]
    open(out_md, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


N_SIMD = 256 * 4  # MI355X: 256 compute units of 4 SIMDs
CLOCK_GHZ = 2.4   # MI355X peak engine clock


def summarize_mfma(pmc_csv, trace_csv, out_md, cmds):
    """MFMA work and busy time per kernel class from per-dispatch counters.

    Executed bf16 MFMA FLOPs = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512; busy
    fraction = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x duration x 2.4 GHz),
    the duration taken from the kernel trace of the same run.  At 1024 bf16
    FLOPs per SIMD per cycle the two agree when every busy cycle does dense
    bf16 work.
    """
    dur = {}
    for r in csv.DictReader(open(trace_csv)):
        dur[r["Dispatch_Id"]] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
    per = {}
    for r in csv.DictReader(open(pmc_csv)):
        d = per.setdefault(r["Dispatch_Id"], {"name": r["Kernel_Name"]})
        d[r["Counter_Name"]] = float(r["Counter_Value"])
    classes = [("bf16 GEMMs (gemm_bf16_*)", "gemm_bf16_"), ("attention forward (attn_fwd_mfma)", "attn_fwd_mfma"),
               ("attention backward dK/dV (attn_bwd_dkdv_mfma)", "attn_bwd_dkdv_mfma"),
               ("attention backward dQ (attn_bwd_dq_mfma)", "attn_bwd_dq_mfma")]
    lines = ["# MFMA utilisation of the FAL training step (serialized launches; workload as in the command)", "",
             "Commands (repository root on the GPU host, `TMPDIR=/tmp`):", "",
             "```", *cmds, "```", "",
             "Per kernel class, summed over its dispatches: executed bf16 MFMA FLOPs =",
             "SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 over the traced kernel time (dense bf16 peak 2500 TFLOP/s);",
             "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x traced time x 2.4 GHz).  Executed FLOPs",
             "include work the algorithmic count leaves out (zero-padded edge tiles, the masked half of",
             "diagonal attention tiles, the recomputed scores of the backward).", "",
             "| class | dispatches | total ms | executed TFLOP/s | of 2500 | MFMA busy |",
             "|---|---|---|---|---|---|"]
    for label, key in classes:
        ds = [(k, v) for k, v in per.items() if key in v["name"] and k in dur
              and "SQ_VALU_MFMA_BUSY_CYCLES" in v and "SQ_INSTS_VALU_MFMA_MOPS_BF16" in v]
        if not ds:
            continue
        t = sum(dur[k] for k, _ in ds)
        flops = sum(v["SQ_INSTS_VALU_MFMA_MOPS_BF16"] for _, v in ds) * 512
        busy = sum(v["SQ_VALU_MFMA_BUSY_CYCLES"] for _, v in ds)
        tf = flops / t / 1e12
        lines.append(f"| {label} | {len(ds)} | {t * 1e3:.2f} | {tf:.0f} | {tf / 2500:.3f} | "
                     f"{100 * busy / (N_SIMD * t * CLOCK_GHZ * 1e9):.1f}% |")
    open(out_md, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))

HBM_CLASSES = [("bf16 GEMMs + split-K reduces", ("gemm_bf16_", "splitk_reduce")),
               ("attention (MFMA kernels)", ("attn_fwd_mfma", "attn_bwd_")),
               ("LayerNorm fwd / bwd / parameter sums", ("ln_fwd", "ln_bwd", "ln_param_partials",
                                                         "col_reduce_multi", "norm_bwd")),
               ("cross-entropy rows", ("ce_rows",)),
               ("bias-gradient column sums", ("col_sum_batch_partials", "col_reduce_batch")),
               ("embedding fwd / bwd", ("embed_", "wpe_grad")),
               ("AdamW update", ("adamw",))]


def summarize_hbm(fetch_csv, write_csv, probe_mib, out_md, cmds):
    """HBM bytes and achieved GB/s per kernel class from FETCH_SIZE / WRITE_SIZE.

    Each counter is read per dispatch (KiB) and scaled by the factor that
    makes the run's plain copy of PROBE_MIB MiB read and write exactly that
    many bytes; durations come from the dispatch timestamps in the same
    file.  Achieved GB/s = (fetched + written bytes) / kernel time.
    """
    probe_bytes = int(probe_mib) * (1 << 20)

    def load(path, counter):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        probe = [r for r in rows if "MulFunctor" in r["Kernel_Name"]]
        assert probe, "no copy-probe dispatch in " + path
        calib = probe_bytes / (float(probe[-1]["Counter_Value"]) * 1024.0)
        return calib, rows
    cf, fr = load(fetch_csv, "FETCH_SIZE")
    cw, wr = load(write_csv, "WRITE_SIZE")
    lines = ["# HBM traffic per kernel class of the FAL training step (serialized launches; workload as in the "
             "command)", "",
             "Commands (repository root on the GPU host, `TMPDIR=/tmp`), one counter per run:", "",
             "```", *cmds, "```", "",
             f"Counter calibration by the run's plain copy of {int(probe_mib)} MiB: FETCH_SIZE x {cf:.4f}, "
             f"WRITE_SIZE x {cw:.4f}.", "Kernel time is the FETCH_SIZE run's dispatch time; HBM peak 8000 GB/s.", "",
             "| class | dispatches | kernel ms | fetched MB | written MB | GB/s | of 8 TB/s |",
             "|---|---|---|---|---|---|---|"]
    for label, keys in HBM_CLASSES:
        f = [r for r in fr if any(k in r["Kernel_Name"] for k in keys)]
        w = [r for r in wr if any(k in r["Kernel_Name"] for k in keys)]
        if not f or not w:
            continue
        fb = sum(float(r["Counter_Value"]) for r in f) * 1024.0 * cf
        wb = sum(float(r["Counter_Value"]) for r in w) * 1024.0 * cw
        t = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in f) * 1e-9
        gbs = (fb + wb) / t / 1e9
        lines.append(f"| {label} | {len(f)} | {t * 1e3:.2f} | {fb / 1e6:.0f} | {wb / 1e6:.0f} | {gbs:.0f} | "
                     f"{gbs / 8000:.2f} |")
    open(out_md, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    args = parse()
    if args.summarize_stats:
        summarize_stats(*args.summarize_stats, args.cmd, args.label)
        return
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic, args.cmd, args.label)
        return
    if args.summarize_mfma:
        summarize_mfma(*args.summarize_mfma, args.cmd)
        return
    if args.summarize_hbm:
        summarize_hbm(*args.summarize_hbm, args.cmd)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported: the training step "
              f"runs on a single GPU (multi-GPU sharding is not implemented).", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2510_14614_amd import get_config
    from paper_2510_14614_amd.config import ARCH_NAMES, SCHED_NAMES, SCHED_SEQ

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    arch = ARCH_NAMES[args.arch]
    sched = SCHED_NAMES[args.sched]
    cfg = get_config(args.config, arch=arch, sched=sched, dtype=1)

    r = Runner(cfg, single_stream=args.single_stream, graph=args.graph)
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
    peaks = measured_peaks()

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
            "kernel": "gemm_bf16_dbl / gemm_bf16_pipe (all bf16 GEMM launches of the step, with the split-K "
                      "reduces they launch)",
            "achieved": gemm_tflops,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": gemm_tflops / PEAK_BF16_TFLOPS,
            "traffic": measured_traffic(args.config, args.arch),
            "traffic_unit": "HBM bytes per GEMM call (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "avg_launch_ms": gemm_avg_ms,
            "avg_launch_gflop": g["flops"] / max(g["launches"], 1) / 1e9,
            "avg_launch_alg_bytes": g["bytes"] / max(g["launches"], 1),
            "measured_peak": peaks["mfma_bf16_tflops"],
            "frac_of_measured_peak": gemm_tflops / peaks["mfma_bf16_tflops"],
        },
        "measured_peaks": peaks,
        "kernels": kernels,
        "wall_s_timed": wall,
    }

    if not args.no_compare:
        comp = {}
        for name, a, s in (("gpt_seq", "gpt", SCHED_SEQ), ("falplus_seq", "falplus", SCHED_SEQ),
                           ("parallel", "parallel", sched)):
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

    if not args.no_optimizer:
        # the same step followed by the AdamW update of every parameter
        # (fp32 master weights and moments, bf16 weight copy; the paper's
        # lr 1e-4, weight decay 0.001, clip 1)
        ro = Runner(cfg, single_stream=args.single_stream, optimizer=True)
        ms_o, _ = ro.time(args.steps, args.warmup)
        po = ro.profile(args.steps)["optimizer"]
        n_params = ro.F.layout["total"]
        ro.close()
        opt_ms = po["ms"] / max(po["launches"], 1)
        out["training_with_optimizer"] = {
            "tokens_per_s": cfg.tokens / (ms_o / 1000.0),
            "ms_per_step": ms_o,
            "optimizer_ms": opt_ms,
            "parameters": n_params,
            "optimizer_alg_bytes": po["bytes"] / max(po["launches"], 1),
            "optimizer_GB/s": po["bytes"] / max(po["ms"], 1e-9) / 1e6,
            "optimizer_frac_hbm_peak": po["bytes"] / max(po["ms"], 1e-9) / 1e6 / PEAK_HBM_GBS,
        }

    if not args.no_forward:
        # forward step without gradients (the paper's inference measurement),
        # this architecture and the same-kernel sequential GPT
        fo = {}
        for name, c2 in (("this", cfg), ("gpt_seq", cfg.replace(arch=ARCH_NAMES["gpt"], sched=SCHED_SEQ))):
            rf = Runner(c2, single_stream=args.single_stream, forward_only=True)
            ms_f, _ = rf.time(args.steps, args.warmup)
            rf.close()
            fo[name] = {"tokens_per_s": c2.tokens / (ms_f / 1000.0), "ms_per_forward": ms_f}
        fo["speedup_over_gpt_same_kernels"] = fo["gpt_seq"]["ms_per_forward"] / fo["this"]["ms_per_forward"]
        out["forward_only"] = fo

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg)

    if args.copy_probe > 0:
        out["copy_probe_bytes"] = copy_probe(args.copy_probe)

    print(json.dumps(out), flush=True)


def copy_probe(mib):
    """One elementwise kernel that reads and writes mib MiB each (a plain
    copy with a scale, so it is a shader dispatch the counters see)."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, device="cuda", dtype=torch.float32)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.mul(src, 2.0, out=dst)
    torch.cuda.synchronize()
    return n * 4


if __name__ == "__main__":
    main()
