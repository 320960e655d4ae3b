"""The step-level continuous-batching loop on the GPU (SD-1.5 shape, 64x64):
requests join and leave between steps; sampled requests of one iteration
are replayed through the oracle."""
import math

import numpy as np
import pytest

import oracle
from fixtures import get_config, serve_null_context
from tests.gpu_util import log, rel_l2

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def test_serving_loop_and_oracle_replay(weights_cache):
    from paper_2605_08835_amd import serve
    wl = "c5_sd15_serve"
    res, snaps = serve.run(wl, iterations=14, weights=weights_cache(wl), snapshot_at={13}, log=log)
    log(f"serving loop: {res}")
    assert res["steps_run"] == 14 and res["mean_rows"] > 0
    snap = snaps[13]
    inp = snap["inputs"]
    unet = get_config(wl)["unet"]
    null = serve_null_context(wl)
    abar = oracle.alphas_cumprod(oracle.betas(unet["schedule"]))
    on = np.flatnonzero(inp["cfg_on"] == 1)
    picks = [int(on[0])] if len(on) else [0]
    for i in picks:
        ref = oracle.unet_step_request(unet, weights_cache(wl), snap["before"][i], int(inp["t"][i]),
                                       int(inp["t_prev"][i]), bool(inp["cfg_on"][i]), float(inp["guidance"][i]),
                                       snap["ctx"][i], null, abar)
        err = rel_l2(snap["after"][i], ref)
        log(f"  replay request {inp['ids'][i]} t={inp['t'][i]} cfg={inp['cfg_on'][i]}: rel L2 {err:.3e}")
        assert err <= 2e-2
