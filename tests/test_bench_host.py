"""Host-side arithmetic of bench.py: the algorithmic FLOPs per UNet row
(a topology walk that must give the SD-1.5 and SDXL figures the roofline is
quoted against) and the split of that total into GEMM-class, attention and
output-conv work."""
import math
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from fixtures import get_config  # noqa: E402


def test_flops_per_row_of_the_published_shapes():
    assert math.isclose(bench.unet_flops_per_row(get_config("c3_sd15_mixed32")["unet"]), 803.27344128e9, rel_tol=1e-12)
    assert math.isclose(bench.unet_flops_per_row(get_config("c4_sdxl_cfg8")["unet"]), 6761.23639808e9, rel_tol=1e-12)


def test_non_gemm_split():
    u = get_config("c3_sd15_mixed32")["unet"]
    attn, out = bench.non_gemm_flops_per_row(u)
    # self-attention 4 N^2 C and cross-attention 4 N 77 C summed over the 16 Transformer blocks
    assert math.isclose(attn, 126.05227008e9, rel_tol=1e-12)
    assert out == 2.0 * 64 * 64 * 9 * 320 * 4


def _write_csv(path, header, rows):
    import csv
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def test_counter_summary_arithmetic(tmp_path):
    """The summary of synthetic rocprofv3 CSVs: calibration scale, bytes per
    GEMM launch (the split-K reduction charged to its launch), per-class
    bandwidth and the cycle-weighted busy fractions."""
    d = str(tmp_path)
    gemm = "void sd::gemm_bf16_dma_kernel<256>(sd::GemmArgs)"
    red = "sd::splitk_reduce_kernel(sd::GemmArgs)"
    gn = "_ZN2sd17gn_partial_kernelIDF16bEEvPKT_"
    copy = "void at::native::elementwise_kernel<128, 4>(int)"
    _write_csv(f"{d}/stats/p_kernel_stats.csv", ["Name", "Calls", "TotalDurationNs"],
               [[gemm, 2, 400000], [red, 1, 20000], [gn, 4, 40000]])
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    # the copy moves 1 MiB each way; FETCH reads half the bytes in KiB (scale 2), WRITE exact
    _write_csv(f"{d}/fetch/p_counter_collection.csv", hdr,
               [[1, copy, "FETCH_SIZE", 512], [2, gemm, "FETCH_SIZE", 100], [3, red, "FETCH_SIZE", 10],
                [4, gemm, "FETCH_SIZE", 100], [5, gn, "FETCH_SIZE", 8], [6, gn, "FETCH_SIZE", 8],
                [7, gn, "FETCH_SIZE", 8], [8, gn, "FETCH_SIZE", 8]])
    _write_csv(f"{d}/write/p_counter_collection.csv", hdr,
               [[1, copy, "WRITE_SIZE", 1024], [2, gemm, "WRITE_SIZE", 50], [3, red, "WRITE_SIZE", 0],
                [4, gemm, "WRITE_SIZE", 50], [5, gn, "WRITE_SIZE", 1], [6, gn, "WRITE_SIZE", 1],
                [7, gn, "WRITE_SIZE", 1], [8, gn, "WRITE_SIZE", 1]])
    _write_csv(f"{d}/sq/p_counter_collection.csv", hdr,
               [[2, gemm, "MfmaUtil", 40.0], [2, gemm, "VALUBusy", 10.0], [2, gemm, "GRBM_GUI_ACTIVE", 100],
                [4, gemm, "MfmaUtil", 70.0], [4, gemm, "VALUBusy", 20.0], [4, gemm, "GRBM_GUI_ACTIVE", 300],
                [4, gemm, "SQ_LDS_BANK_CONFLICT", 5], [4, gemm, "SQ_INSTS_LDS", 20]])
    txt = bench.summarize(f"{d}/stats", f"{d}/fetch", f"{d}/write", 2**20, f"{d}/sq")
    tables = [[[c.strip() for c in l.split("|")[1:-1]] for l in block.splitlines() if l.startswith("|")]
              for block in txt.split("\n\n")]
    by_head = {t[0][-1]: {r[0]: r[1:] for r in t[2:]} for t in tables if t}
    q = by_head["value"]
    assert q["fetch scale"] == ["2.0000"] and q["write scale"] == ["1.0000"]
    assert q["GEMM launches"] == ["2"]
    # (2 x 100 + 10) KiB x 2 fetched + 100 KiB written over 2 launches
    assert float(q["traffic_bytes_per_launch"][0]) == (210 * 2 + 100) * 1024 / 2
    bw = by_head["GB/s"]
    # GEMM class: 420 us over 2 launches = 210 us; GroupNorm: 10 us per launch, 17 KiB per launch
    assert bw["gemm"][-1] == f"{(210 * 2 + 100) * 1024 / 2 / 210e-6 / 1e9:.0f}"
    assert bw["groupnorm"][-1] == f"{17 * 1024 / 10e-6 / 1e9:.0f}"
    # cycle-weighted: (40 x 100 + 70 x 300) / 400 = 62.5; (10 x 100 + 20 x 300) / 400 = 17.5
    sq = by_head["LDS bank-conflict cycles per LDS instruction"]
    assert sq["gemm"] == ["2", "62.5", "17.5", "0.250"]
