"""The GroupNorm-statistics entry point that allocates nothing
(synerdiff_op_groupnorm_stats_noalloc) against the entry point that takes a
caller-allocated partial-sum buffer: same outputs, bit for bit, on two calls
in a row with the second on a smaller input (the library's device array
keeps the first call's partials), and a clear error past its capacity."""
import ctypes

import numpy as np
import pytest

from fixtures import bf16_round

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _case(rng, n, H, W, c0, c1, dt):
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    x0 = rng.standard_normal((n, H, W, c0)).astype(np.float32) * 2 + 0.5
    x1 = rng.standard_normal((n, H, W, c1)).astype(np.float32) if c1 else None
    if dt == "bf16":
        x0 = bf16_round(x0)
        x1 = bf16_round(x1) if c1 else None
    g = (1 + 0.1 * rng.standard_normal(c0 + c1)).astype(np.float32)
    b = (0.1 * rng.standard_normal(c0 + c1)).astype(np.float32)
    dev = lambda a, t=None: torch.from_numpy(np.ascontiguousarray(a)).cuda().to(t) if t else \
        torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return dev(x0, tdt), (dev(x1, tdt) if c1 else None), dev(g), dev(b)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_noalloc_matches_the_allocating_entry_point_twice(dt):
    from paper_2605_08835_amd import ops
    rng = np.random.default_rng(11)
    # first call: 16 images at 64x64 x 320 (215k partial floats); second: smaller, with a concat
    for (n, H, W, c0, c1, G) in [(16, 64, 64, 320, 0, 32), (3, 8, 8, 64, 32, 8)]:
        x0, x1, g, b = _case(rng, n, H, W, c0, c1, dt)
        ref_sc, ref_sh = ops.groupnorm_stats(x0, G, 1e-5, g, b, x1=x1)
        sc, sh = ops.groupnorm_stats_noalloc(x0, G, 1e-5, g, b, x1=x1)
        torch.cuda.synchronize()
        print(f"noalloc groupnorm {dt} {(n, H, W, c0, c1, G)}: max |diff| "
              f"{(sc - ref_sc).abs().max().item():.3e} {(sh - ref_sh).abs().max().item():.3e}", flush=True)
        assert torch.equal(sc, ref_sc) and torch.equal(sh, ref_sh)


def test_noalloc_rejects_more_than_its_scratch():
    from paper_2605_08835_amd import lib, ops
    from paper_2605_08835_amd.binding import SynerDiffError
    # 9 images of 64x64 x 4096 channels need 9 * 64 * 4096 * 2 = 4.7M partial floats > 4M
    x = torch.zeros(9, 64, 64, 4096, device="cuda", dtype=torch.bfloat16)
    g = torch.ones(4096, device="cuda")
    need = lib().synerdiff_op_groupnorm_scratch_floats(9, 64 * 64, 4096)
    assert need > (1 << 22)
    with pytest.raises(SynerDiffError, match="exceed"):
        ops.groupnorm_stats_noalloc(x, 32, 1e-5, g, g)
    torch.cuda.synchronize()
