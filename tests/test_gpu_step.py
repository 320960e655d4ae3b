"""Whole-step parity on the GPU: the HIP UNet step against the oracle on the
same seeded inputs, per request (relative L2 of x' and of the guided eps),
plus the step's invariants."""
import numpy as np
import pytest

import oracle
from fixtures import get_config, make_requests
from tests.gpu_util import gpu_step, log, rel_l2, to_dev

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

# Tolerances.  Latents: as stated for the two precisions.  The raw UNet
# output of a row (eps_c, from a Skip-CFG pass) is gated too, because
# x' = A x + B eps is dominated by the exactly shared A x.  The guided
# eps_u + w (eps_c - eps_u) inherits the branch errors scaled by the
# combine: |err| <= tol * (|1 - w| |eps_u| + |w| |eps_c|).
TOL_LAT = {"f32": 1e-4, "bf16": 2e-2}
TOL_EPS = {"f32": 1e-4, "bf16": 3e-2}

_MODELS = {}


def model_for(workload, weights_cache, max_requests=None):
    from paper_2605_08835_amd import UNet
    key = (workload, max_requests)
    if key not in _MODELS:
        unet = get_config(workload)["unet"]
        R = max_requests or get_config(workload)["requests"]
        m = UNet(unet, max_requests=R)
        m.load_weights(weights_cache(workload))
        _MODELS[key] = m
    return _MODELS[key]


def check(workload, weights_cache, only=None, req=None):
    unet = get_config(workload)["unet"]
    dt = unet["dtype"]
    req = req or make_requests(workload)
    m = model_for(workload, weights_cache)
    log(f"{workload}: GPU step, {len(req['timesteps'])} requests, cfg_on={list(req['cfg_on'])}")
    out, eps = gpu_step(m, req)
    _, eps_c = gpu_step(m, dict(req, cfg_on=np.zeros_like(req["cfg_on"])))
    idx = list(range(len(req["timesteps"])) if only is None else only)
    parts = {}
    ref, ref_eps = oracle.unet_step(unet, weights_cache(workload), req, only=idx, want_eps=True, parts=parts)
    worst = 0.0
    for r in idx:
        ec, eu = parts[r]["eps_c"], parts[r]["eps_u"]
        el, eg, er = rel_l2(out[r], ref[r]), rel_l2(eps[r], ref_eps[r]), rel_l2(eps_c[r], ec)
        w = float(req["guidance"][r])
        amp = 1.0 if eu is None else (abs(1 - w) * np.linalg.norm(eu) + abs(w) * np.linalg.norm(ec)) / np.linalg.norm(ref_eps[r])
        log(f"  request {r} t={req['timesteps'][r]} cfg={req['cfg_on'][r]}: rel L2 latents {el:.3e} "
            f"eps_c {er:.3e} guided eps {eg:.3e} (combine gain {amp:.1f})")
        assert np.isfinite(out[r]).all()
        assert el <= TOL_LAT[dt] and er <= TOL_EPS[dt] and eg <= TOL_EPS[dt] * amp, (r, el, er, eg, amp)
        worst = max(worst, el)
    return worst


def test_tiny_f32_step(weights_cache):
    check("c1_tiny_f32", weights_cache)


def test_tiny_f32_ragged_step(weights_cache):
    check("t_tiny_f32_ragged", weights_cache)


def test_tiny_bf16_step(weights_cache):
    check("t_tiny_bf16", weights_cache)


def test_sd15_shape_16px_step(weights_cache):
    check("t_sd15_16", weights_cache)


def test_sdxl_shape_16px_step(weights_cache):
    check("t_sdxl_16", weights_cache)


def test_c2_full_size_sampled(weights_cache):
    check("c2_sd15_cfg8", weights_cache, only=[0, 5])


def test_c3_full_size_sampled(weights_cache):
    req = make_requests("c3_sd15_mixed32")
    on = int(np.flatnonzero(req["cfg_on"])[0])
    off = int(np.flatnonzero(req["cfg_on"] == 0)[-1])
    check("c3_sd15_mixed32", weights_cache, only=[on, off], req=req)


def test_c4_sdxl_full_size_sampled(weights_cache):
    """SDXL-like UNet at 128x128 (8 requests with CFG, 16 rows): the full
    batch runs on the GPU; request 3 is recomputed by the oracle."""
    check("c4_sdxl_cfg8", weights_cache, only=[3])


def test_batch_permutation_is_bitwise_invariant(weights_cache):
    wl = "t_sd15_16"
    req = make_requests(wl)
    m = model_for(wl, weights_cache)
    a, ea = gpu_step(m, req)
    perm = [2, 0, 1]
    rp = dict(req)
    for k in ("latents", "ctx_cond", "timesteps", "t_prev", "cfg_on", "guidance"):
        rp[k] = req[k][perm]
    b, eb = gpu_step(m, rp)
    for i, r in enumerate(perm):
        assert np.array_equal(a[r], b[i]) and np.array_equal(ea[r], eb[i]), r


def test_batch_mates_do_not_change_a_request(weights_cache):
    wl = "t_sd15_16"
    req = make_requests(wl)
    m = model_for(wl, weights_cache)
    a, _ = gpu_step(m, req)
    one = {k: (v[1:2] if isinstance(v, np.ndarray) and v.ndim and v.shape[0] == 3 and k != "ctx_uncond" else v)
           for k, v in req.items()}
    b, _ = gpu_step(m, one)
    assert np.array_equal(a[1], b[0])


def test_guidance_one_equals_skip_cfg(weights_cache):
    wl = "t_sd15_16"
    req = make_requests(wl)
    m = model_for(wl, weights_cache)
    r1 = dict(req, guidance=np.ones(3, np.float32), cfg_on=np.array([1, 1, 1], np.uint8))
    r0 = dict(req, cfg_on=np.array([0, 0, 0], np.uint8))
    a, ea = gpu_step(m, r1)
    b, eb = gpu_step(m, r0)
    assert rel_l2(ea, eb) < 1e-6 and rel_l2(a, b) < 1e-6


def test_in_place_and_empty_batch(weights_cache):
    wl = "t_tiny_bf16"
    req = make_requests(wl)
    m = model_for(wl, weights_cache)
    a, _ = gpu_step(m, req)
    b, _ = gpu_step(m, req, out_inplace=True)
    assert np.array_equal(a, b)
    u = get_config(wl)["unet"]
    lat = torch.zeros(0, 4, 12, 12, device="cuda")
    ctx = torch.zeros(0, u["ctx_len"], u["ctx_dim"], device="cuda", dtype=m.act_dtype)
    unc = torch.zeros(u["ctx_len"], u["ctx_dim"], device="cuda", dtype=m.act_dtype)
    m.step(lat, np.zeros(0, np.int32), np.zeros(0, np.uint8), np.zeros(0, np.float32), ctx, unc,
           np.zeros((0, 2), np.float32), out=lat)


def test_ten_chained_steps(weights_cache):
    """Each side feeds its own outputs back for 10 steps; requests whose
    t_prev < 0 finish and leave the chain."""
    wl = "t_sd15_16"
    unet = get_config(wl)["unet"]
    req = make_requests(wl)
    req["timesteps"] = np.array([999, 180, 560])
    req["t_prev"] = req["timesteps"] - 20
    m = model_for(wl, weights_cache)
    g = dict(req)
    o = dict(req)
    for step in range(10):
        live = np.flatnonzero(g["timesteps"] >= 0)
        sub = {k: (v[live] if isinstance(v, np.ndarray) and v.ndim and v.shape[0] == 3 and k != "ctx_uncond" else v)
               for k, v in g.items()}
        gl, _ = gpu_step(m, sub)
        osub = dict(sub, latents=o["latents"][live])
        ol = oracle.unet_step(unet, weights_cache(wl), osub)
        g["latents"] = g["latents"].copy()
        o["latents"] = o["latents"].copy()
        for j, r in enumerate(live):
            g["latents"][r] = gl[j].astype(np.float32)
            o["latents"][r] = ol[j].astype(np.float32)
        g["timesteps"] = g["timesteps"] - 20
        g["t_prev"] = g["t_prev"] - 20
        errs = [rel_l2(g["latents"][r], o["latents"][r]) for r in range(3)]
        log(f"  chained step {step}: rel L2 {['%.2e' % e for e in errs]}")
    assert max(errs) <= 5e-2


def test_v_prediction_tiny_f32_step(weights_cache):
    """v-prediction (SD-2.x): the same kernels with the v-form (A, B)."""
    check("t_tiny_f32_v", weights_cache)


def test_sd21_shape_16px_step(weights_cache):
    """SD-2.1 layout (64-wide heads, 1024-wide context, v-prediction) at 16x16."""
    check("t_sd21_16", weights_cache)


def test_c6_sd21_768px_sampled(weights_cache):
    """SD-2.1 at 768 px (96x96 latents), 8 requests with CFG: request 2
    recomputed by the oracle."""
    check("c6_sd21_v", weights_cache, only=[2])


def test_mixed_resolutions_share_weights(weights_cache):
    """Requests at 16x16 and 24x24 latents in one step through handles that
    share one weight copy: each request matches the oracle, and the 16x16
    group is bit-identical to a standalone handle."""
    from paper_2605_08835_amd import MultiResolutionUNet
    wl = "t_sd15_16"
    unet = get_config(wl)["unet"]
    W = weights_cache(wl)
    mr = MultiResolutionUNet(unet, {(16, 16): 3, (24, 24): 2})
    mr.load_weights(W)
    base = make_requests(wl)
    rng = np.random.default_rng(3)
    big = dict(base, latents=rng.standard_normal((2, 4, 24, 24)).astype(np.float32),
               timesteps=np.array([640, 90]), t_prev=np.array([620, 70]), cfg_on=np.array([1, 0], np.uint8),
               guidance=np.array([6.5, 6.5], np.float32), ctx_cond=base["ctx_cond"][:2])
    act = mr.act_dtype
    unc = to_dev(base["ctx_uncond"], act)
    groups = {}
    for size, r in (((16, 16), base), ((24, 24), big)):
        groups[size] = dict(latents=to_dev(r["latents"], torch.float32), timesteps=r["timesteps"], cfg_on=r["cfg_on"],
                            guidance=r["guidance"], ctx_cond=to_dev(r["ctx_cond"], act),
                            coef=mr.coefficients(r["schedule"], r["timesteps"], r["t_prev"]))
    outs = mr.step(groups, unc)
    torch.cuda.synchronize()
    for size, r in (((16, 16), base), ((24, 24), big)):
        cfg = dict(unet, latent_h=size[0], latent_w=size[1])
        ref = oracle.unet_step(cfg, W, r)
        got = outs[size].cpu().double().numpy()
        for i in range(len(r["timesteps"])):
            err = rel_l2(got[i], ref[i])
            log(f"  mixed resolution {size} request {i}: rel L2 {err:.3e}")
            assert err <= TOL_LAT["bf16"], (size, i, err)
    alone, _ = gpu_step(model_for(wl, weights_cache), base, eps=False)
    assert np.array_equal(outs[(16, 16)].cpu().double().numpy(), alone)
    mr.close()
