"""Host-only checks of bench.py's offline rocprofv3 summaries (no GPU)."""
import csv
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def test_summarize_mfma_known_counts(tmp_path):
    # two GEMM dispatches (100 us and 50 us), one attention forward (40 us) and
    # one unrelated kernel that must be ignored
    trace = tmp_path / "trace.csv"
    _write(trace, ["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"], [
        [1, "void fal::gemm_bf16_dbl<1, 1, 128, 128, 2>(fal::GemmGroup, int)", 1000, 101000],
        [2, "void fal::gemm_bf16_pipe<1, 0, 256, 256, 1, 4>(fal::GemmGroup, int)", 200000, 250000],
        [3, "void fal::attn_fwd_mfma<64, true>(bf16 const*, int, int, bf16*, float*)", 300000, 340000],
        [4, "fal::zero_kernel(float*, long)", 400000, 401000],
    ])
    # GEMMs: 150 us in all; 1.5e11 FLOPs -> 1000 TFLOP/s = 0.4 of 2500;
    # busy cycles for 40% of 1024 SIMDs x 150 us x 2.4 GHz
    mops_g = [1.0e11 / 512, 0.5e11 / 512]
    busy_g = [0.4 * 1024 * 100e-6 * 2.4e9, 0.4 * 1024 * 50e-6 * 2.4e9]
    # attention: 40 us, 2e10 FLOPs -> 500 TFLOP/s = 0.2; busy 20%
    rows = []
    for d, (m, b) in enumerate(zip(mops_g, busy_g), start=1):
        rows.append([d, "gemm_bf16_x", "SQ_INSTS_VALU_MFMA_MOPS_BF16", m])
        rows.append([d, "gemm_bf16_x", "SQ_VALU_MFMA_BUSY_CYCLES", b])
    rows.append([3, "attn_fwd_mfma", "SQ_INSTS_VALU_MFMA_MOPS_BF16", 2e10 / 512])
    rows.append([3, "attn_fwd_mfma", "SQ_VALU_MFMA_BUSY_CYCLES", 0.2 * 1024 * 40e-6 * 2.4e9])
    rows.append([4, "zero_kernel", "SQ_INSTS_VALU_MFMA_MOPS_BF16", 0])
    rows.append([4, "zero_kernel", "SQ_VALU_MFMA_BUSY_CYCLES", 0])
    pmc = tmp_path / "pmc.csv"
    _write(pmc, ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], rows)
    out = tmp_path / "out.md"
    bench.summarize_mfma(str(pmc), str(trace), str(out), ["cmd"])
    text = out.read_text()
    gemm = next(l for l in text.splitlines() if l.startswith("| bf16 GEMMs"))
    attn = next(l for l in text.splitlines() if l.startswith("| attention forward"))
    assert gemm.split("|")[2:7] == [" 2 ", " 0.15 ", " 1000 ", " 0.400 ", " 40.0% "]
    assert attn.split("|")[2:7] == [" 1 ", " 0.04 ", " 500 ", " 0.200 ", " 20.0% "]
    assert "zero_kernel" not in text
    assert "attention backward" not in text  # classes with no dispatches are left out


def test_summarize_hbm_calibrated_rates(tmp_path):
    # counters read half the copy's bytes on fetch (factor 2) and all on write
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    probe = "void at::native::vectorized_elementwise_kernel<4, at::native::MulFunctor<float> >(int)"
    ln = "void fal::ln_bwd_v4<bf16, 3>(fal::LnBwdArgs)"
    ce = "void fal::ce_rows_x8<7>(bf16 const*, int const*, int, int, float, bf16*, float*)"
    mib = 1 << 20
    fetch = [[1, ln, "FETCH_SIZE", 50 * mib / 1024 / 2, 0, 20000],        # 50 MiB in 20 us
             [2, ce, "FETCH_SIZE", 100 * mib / 1024 / 2, 30000, 80000],   # 100 MiB in 50 us
             [3, probe, "FETCH_SIZE", 1024 * mib / 1024 / 2, 90000, 99000]]
    write = [[1, ln, "WRITE_SIZE", 30 * mib / 1024, 0, 21000],
             [2, ce, "WRITE_SIZE", 100 * mib / 1024, 30000, 81000],
             [3, probe, "WRITE_SIZE", 1024 * mib / 1024, 90000, 99000]]
    _write(tmp_path / "f.csv", hdr, fetch)
    _write(tmp_path / "w.csv", hdr, write)
    out = tmp_path / "out.md"
    bench.summarize_hbm(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), 1024, str(out), ["cmd"])
    lines = out.read_text().splitlines()
    assert "FETCH_SIZE x 2.0000, WRITE_SIZE x 1.0000" in "\n".join(lines)
    lnl = next(l for l in lines if l.startswith("| LayerNorm")).split("|")
    cel = next(l for l in lines if l.startswith("| cross-entropy")).split("|")
    # kernel time from the fetch run's timestamps
    assert lnl[2:5] == [" 1 ", " 0.02 ", f" {50 * mib / 1e6:.0f} "]
    assert lnl[5].strip() == f"{30 * mib / 1e6:.0f}"
    assert lnl[6].strip() == f"{80 * mib / 20e-6 / 1e9:.0f}"
    assert cel[6].strip() == f"{200 * mib / 50e-6 / 1e9:.0f}"
    assert not any(l.startswith("| bf16 GEMMs") for l in lines)
