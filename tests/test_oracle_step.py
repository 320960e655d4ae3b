"""Pins of the oracle's sampler, guidance and whole-step composition.  CPU only."""
import math

import numpy as np
import pytest

import oracle
from fixtures import get_config, make_requests, make_weights, manifest, param_count
from fixtures.configs import SD21, SD15, SDXL, TINY
from oracle import sampler
from oracle.unet import Weights, unet_eps

rng = np.random.default_rng(11)


# ---- schedules and DDIM -------------------------------------------------------

def test_beta_schedule_endpoints_and_shape():
    lin = sampler.betas("linear")
    assert lin[0] == pytest.approx(1e-4, abs=1e-18) and lin[-1] == pytest.approx(0.02, abs=1e-17)
    assert np.allclose(np.diff(lin, 2), 0, atol=1e-17)  # linear in s
    sl = sampler.betas("scaled_linear")
    assert sl[0] == pytest.approx(0.00085, rel=1e-14) and sl[-1] == pytest.approx(0.012, rel=1e-14)
    assert np.allclose(np.diff(np.sqrt(sl), 2), 0, atol=1e-16)  # linear in sqrt(beta)


@pytest.mark.parametrize("schedule", ["linear", "scaled_linear"])
def test_alphas_cumprod_by_sum_of_logs(schedule):
    b = sampler.betas(schedule)
    ab = sampler.alphas_cumprod(b)
    for t in (0, 1, 500, 999):
        assert ab[t] == pytest.approx(math.exp(math.fsum(math.log1p(-x) for x in b[:t + 1])), rel=1e-12)
    assert np.all(np.diff(ab) < 0)


@pytest.mark.parametrize("a_t,a_prev", [(0.05, 0.07), (0.3, 0.9), (0.999, 1.0), (4e-5, 6e-5)])
def test_ddim_forward_consistency(a_t, a_prev):
    """If x was noised from x0 with eps at level a_t and the model predicts
    eps exactly, DDIM lands on x0 noised with the same eps at a_prev."""
    x0, eps = rng.standard_normal((4, 5, 5)), rng.standard_normal((4, 5, 5))
    x = math.sqrt(a_t) * x0 + math.sqrt(1 - a_t) * eps
    xn = sampler.ddim_step(x, eps, a_t, a_prev)
    assert np.allclose(xn, math.sqrt(a_prev) * x0 + math.sqrt(1 - a_prev) * eps, atol=1e-10)
    A, B = sampler.ddim_coefficients(a_t, a_prev)
    assert np.allclose(A * x + B * eps, xn, atol=1e-10)


@pytest.mark.parametrize("a_t,a_prev", [(0.05, 0.07), (0.3, 0.9), (0.999, 1.0), (4e-5, 6e-5)])
def test_ddim_v_forward_consistency(a_t, a_prev):
    """v-prediction: with x noised from x0 and eps at a_t and the model
    predicting v = sqrt(a_t) eps - sqrt(1 - a_t) x0 exactly, the update lands
    on x0 noised with the same eps at a_prev (and a_prev = a_t is the
    identity, a_prev = 1 returns x0)."""
    x0, eps = rng.standard_normal((4, 5, 5)), rng.standard_normal((4, 5, 5))
    x = math.sqrt(a_t) * x0 + math.sqrt(1 - a_t) * eps
    v = math.sqrt(a_t) * eps - math.sqrt(1 - a_t) * x0
    assert np.allclose(sampler.ddim_step_v(x, v, a_t, a_prev), math.sqrt(a_prev) * x0 + math.sqrt(1 - a_prev) * eps,
                       atol=1e-10)
    assert np.allclose(sampler.ddim_step_v(x, v, a_t, a_t), x, atol=1e-12)
    assert np.allclose(sampler.ddim_step_v(x, v, a_t, 1.0), x0, atol=1e-10)


def test_ddim_identity_and_final_step():
    x, eps = rng.standard_normal(10), rng.standard_normal(10)
    assert np.allclose(sampler.ddim_step(x, eps, 0.4, 0.4), x, atol=1e-14)
    ab = sampler.alphas_cumprod(sampler.betas("linear"))
    assert sampler.abar_at(ab, -10) == 1.0
    # final step (abar_prev = 1) returns the x0 prediction
    assert np.allclose(sampler.ddim_step(x, eps, 0.25, 1.0), (x - math.sqrt(0.75) * eps) / 0.5)


def test_cfg_combine_closed_forms():
    ec, eu = rng.standard_normal(8), rng.standard_normal(8)
    assert np.allclose(sampler.cfg_combine(ec, eu, 1.0), ec, rtol=0, atol=1e-15)
    assert np.array_equal(sampler.cfg_combine(ec, eu, 0.0), eu)
    e3 = [sampler.cfg_combine(ec, eu, w) for w in (2.0, 5.0, 8.0)]
    assert np.allclose(e3[1] - e3[0], e3[2] - e3[1])  # affine in w


# ---- topology ---------------------------------------------------------------

def test_public_parameter_counts():
    """The manifest reproduces the published UNet sizes: SD-1.5 859,520,964
    and SDXL 2,567,463,684 parameters."""
    assert param_count(SD15) == 859_520_964
    assert param_count(SDXL) == 2_567_463_684
    assert param_count(TINY) == 1_055_044
    # SD-2.x: 1024-wide text context, 64-wide heads (no parameters) and linear projections (same count)
    assert param_count(SD21) == 865_910_724


@pytest.fixture(scope="module")
def tiny():
    cfg = get_config("c1_tiny_f32")["unet"]
    return cfg, make_weights("c1_tiny_f32"), make_requests("c1_tiny_f32")


def test_every_parameter_is_consumed(tiny):
    cfg, w, req = tiny
    W = Weights(w)
    oracle.unet_step(cfg, W, req)
    assert W.used == {n for n, _, _ in manifest(cfg)}


def test_sdxl_shape_every_parameter_is_consumed():
    cfg = get_config("t_sdxl_16")["unet"]
    w = make_weights("t_sdxl_16")
    req = make_requests("t_sdxl_16")
    W = Weights(w)
    oracle.unet_step(cfg, W, req, only=[1])
    assert W.used == {n for n, _, _ in manifest(cfg)}


def test_each_tensor_changes_the_output(tiny):
    """Perturbing any one parameter tensor with noise moves eps (none is read
    and then dropped).  The noise is random rather than a constant because a
    shift common to a whole norm group is removed by the next normalisation.
    A seeded sample of tensors keeps the test short."""
    cfg, w, req = tiny
    base = unet_eps(cfg, w, req["latents"][0], 999, req["ctx_cond"][0])
    names = [n for n, _, _ in manifest(cfg)]
    pick = np.random.default_rng(3).choice(len(names), 40, replace=False)
    for i in sorted(pick):
        w2 = dict(w)
        w2[names[i]] = w[names[i]] + 0.05 * rng.standard_normal(w[names[i]].shape)
        e = unet_eps(cfg, w2, req["latents"][0], 999, req["ctx_cond"][0])
        assert np.abs(e - base).max() > 1e-9, names[i]


# ---- whole-step invariants -------------------------------------------------------

def test_zero_output_conv_gives_pure_A_x(tiny):
    """P2: zero conv_out weights and bias => eps = 0 => x' = A x."""
    cfg, _, req = tiny
    w = make_weights("c1_tiny_f32", zero=("out.conv.w", "out.conv.b"))
    out = oracle.unet_step(cfg, w, req)
    ab = sampler.alphas_cumprod(sampler.betas(req["schedule"]))
    for r in range(2):
        A, _ = sampler.ddim_coefficients(sampler.abar_at(ab, int(req["timesteps"][r])),
                                         sampler.abar_at(ab, int(req["t_prev"][r])))
        assert np.allclose(out[r], A * req["latents"][r], atol=1e-12)


def test_guidance_one_equals_cond_only(tiny):
    """w = 1 makes a CFG request equal to its Skip-CFG (cond-only) twin."""
    cfg, w, req = tiny
    r2 = dict(req, guidance=np.array([1.0, 1.0], np.float32))
    on = oracle.unet_step(cfg, w, r2, only=[0])[0]
    r3 = dict(r2, cfg_on=np.array([0, 0], np.uint8))
    off = oracle.unet_step(cfg, w, r3, only=[0])[0]
    assert np.allclose(on, off, atol=1e-12)


def test_skip_cfg_equals_cond_only_pass(tiny):
    """P4: a Skip-CFG request's x' is the DDIM update with eps_c alone."""
    cfg, w, req = tiny
    out = oracle.unet_step(cfg, w, req, only=[1])[1]
    ab = sampler.alphas_cumprod(sampler.betas(req["schedule"]))
    eps = unet_eps(cfg, w, req["latents"][1], 500, req["ctx_cond"][1])
    ref = sampler.ddim_step(req["latents"][1], eps, ab[500], ab[480])
    assert np.allclose(out, ref, atol=1e-14)


def test_batch_order_independence(tiny):
    """P5: a request's output does not depend on its batch-mates or order."""
    cfg, w, req = tiny
    a = oracle.unet_step(cfg, w, req)
    perm = [1, 0]
    rp = {k: (v[perm] if isinstance(v, np.ndarray) and v.ndim and v.shape[0] == 2 and k != "ctx_uncond" else v)
          for k, v in req.items()}
    b = oracle.unet_step(cfg, w, rp)
    assert np.array_equal(a[0], b[1]) and np.array_equal(a[1], b[0])


def test_null_context_equal_to_cond_makes_w_irrelevant(tiny):
    """P6: with c = c_null the two branches agree, so eps = eps_c for any w."""
    cfg, w, req = tiny
    r2 = dict(req, ctx_uncond=req["ctx_cond"][0])
    o1, e1 = oracle.unet_step(cfg, w, dict(r2, guidance=np.array([2.0, 2.0], np.float32)), only=[0], want_eps=True)
    o2, e2 = oracle.unet_step(cfg, w, dict(r2, guidance=np.array([9.0, 9.0], np.float32)), only=[0], want_eps=True)
    assert np.allclose(e1[0], e2[0], atol=1e-12) and np.allclose(o1[0], o2[0], atol=1e-12)
