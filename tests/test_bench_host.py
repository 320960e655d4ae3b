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
