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


def test_serving_loop_with_vae_chunking_and_controller():
    """The loop with finished requests decoded in chunks on a second stream
    beside the UNet steps, and the feedback controller moving the Skip-CFG
    threshold and c: every decoded image is bit-identical to a plain decode
    of the same latents on one stream."""
    from fixtures.vae import VAE_CONFIGS, make_vae_weights
    from paper_2605_08835_amd import VAE, serve
    from paper_2605_08835_amd.control import FeedbackController
    ctl = FeedbackController(c0=2, c_max=3, window=2, grow=0.1, shrink=0.1)
    res, snaps = serve.run("t_serve_tiny", iterations=30, log=log, vae="vae_t16", vae_batch=2, chunks=2,
                           controller=ctl, keep_images=True)
    log(f"serving loop with VAE: {res}")
    assert res["finished"] > 0 and res["images_decoded"] > 0 and res["vae_chunk_rounds"] >= 2
    assert 0.3 - 1e-9 <= res["controller"]["final_skip_after"] <= 0.6 + 1e-9
    assert 2 <= res["controller"]["final_c"] <= 3
    jobs = snaps["images"]
    assert sum(len(ids) for ids, _, _ in jobs) == res["images_decoded"]
    v = VAE(VAE_CONFIGS["vae_t16"]["vae"], max_images=2)
    v.load_weights(make_vae_weights("vae_t16"))
    for ids, z, img in jobs:
        ref = v.decode(torch.from_numpy(z).cuda())
        torch.cuda.synchronize()
        assert np.array_equal(ref.cpu().numpy(), img), f"job {ids}"
    v.close()


def test_planned_windows_decode_every_finished_request():
    """The loop driven by the stage planner on a synthetic lookup table
    (latency growing with the requests, the decodes and fewer skips): each
    policy runs, decodes the finished requests, and the exact planner never
    leaves a window without a plan."""
    from paper_2605_08835_amd import serve
    grid = dict(m_grid=[1, 4], n_grid=[0, 2], k_fracs=[0.0, 1.0],
                tau=[[[2.0, 1.5], [4.0, 3.5]], [[5.0, 3.0], [7.0, 5.0]]],
                delta=[[[0.0, 0.0], [3.0, 3.0]], [[0.0, 0.0], [4.0, 4.0]]])
    for policy in ("single", "alg1", "exact"):
        res = serve.run_planned("t_serve_tiny", iterations=24, lut=grid, policy=policy, vae="vae_t16", nmax=2,
                                log=log)
        log(f"planned serving ({policy}): {res}")
        assert res["images_decoded"] > 0 and res["stages"] >= 24
        assert res["decode_wait_ms_mean"] is not None and res["decode_wait_ms_mean"] >= 0
        if policy == "exact":
            assert res["fallbacks"] == 0
