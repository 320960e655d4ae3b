"""Beta schedules, DDIM update, classifier-free guidance and the whole step."""
import math

import numpy as np

from .ops import F
from .unet import Weights, unet_eps


def betas(schedule, T=1000):
    """Noise schedules of DDPM (linear, Ho et al. 2020) and latent diffusion
    (scaled linear: linear in sqrt(beta) from 0.00085 to 0.012)."""
    s = np.arange(T, dtype=F) / (T - 1)
    if schedule == "linear":
        return 1e-4 + (0.02 - 1e-4) * s
    if schedule == "scaled_linear":
        a, b = math.sqrt(0.00085), math.sqrt(0.012)
        return (a + (b - a) * s) ** 2
    raise ValueError(schedule)


def alphas_cumprod(beta):
    """abar_t = prod_{s <= t} (1 - beta_s)."""
    return np.cumprod(1.0 - np.asarray(beta, F))


def abar_at(abar, t):
    """abar_t, with abar_t := 1 for t < 0 (the step that ends at x_0)."""
    return 1.0 if t < 0 else float(abar[t])


def ddim_step(x, eps, a_t, a_prev):
    """Deterministic DDIM update (Song et al. 2021, eta = 0, eps-prediction):
    x0 = (x - sqrt(1 - a_t) eps) / sqrt(a_t);
    x' = sqrt(a_prev) x0 + sqrt(1 - a_prev) eps."""
    x0 = (np.asarray(x, F) - math.sqrt(1.0 - a_t) * eps) / math.sqrt(a_t)
    return math.sqrt(a_prev) * x0 + math.sqrt(1.0 - a_prev) * eps


def ddim_step_v(x, v, a_t, a_prev):
    """DDIM update (eta = 0) for a v-prediction model (Salimans & Ho 2022,
    as SD-2.x is trained): the network predicts v = sqrt(a_t) eps -
    sqrt(1 - a_t) x0, so x0 = sqrt(a_t) x - sqrt(1 - a_t) v and
    eps = sqrt(1 - a_t) x + sqrt(a_t) v; then
    x' = sqrt(a_prev) x0 + sqrt(1 - a_prev) eps."""
    x = np.asarray(x, F)
    x0 = math.sqrt(a_t) * x - math.sqrt(1.0 - a_t) * v
    eps = math.sqrt(1.0 - a_t) * x + math.sqrt(a_t) * v
    return math.sqrt(a_prev) * x0 + math.sqrt(1.0 - a_prev) * eps


def ddim_coefficients(a_t, a_prev):
    """(A, B) with DDIM's x' = A x + B eps, from expanding ddim_step."""
    A = math.sqrt(a_prev / a_t)
    B = math.sqrt(1.0 - a_prev) - math.sqrt(a_prev * (1.0 - a_t) / a_t)
    return A, B


def cfg_combine(eps_c, eps_u, w):
    """Classifier-free guidance (Ho & Salimans 2022): eps_u + w (eps_c - eps_u)."""
    return eps_u + w * (eps_c - eps_u)


def unet_step_request(cfg, W, x, t, t_prev, cfg_on, w, ctx, ctx_null, abar,
                      pooled=None, pooled_null=None, time_ids=None, want_eps=False, parts=None):
    """One request's step: returns x' (and the guided eps when asked).

    For a v-prediction UNet (cfg["prediction"] == "v") the network's output
    is v; guidance combines the two branches' v the same way, and the update
    is ddim_step_v.

    With CFG on both the conditional and the unconditional UNet evaluations
    run and are combined; with Skip-CFG only the conditional one runs and its
    output is used as is (the unconditional branch is bypassed, Sec. III-B).
    When `parts` is a dict it receives the raw branch outputs under "eps_c"
    and "eps_u" (None under Skip-CFG)."""
    eps_c = unet_eps(cfg, W, x, t, ctx, pooled, time_ids)
    eps_u = None
    if cfg_on:
        eps_u = unet_eps(cfg, W, x, t, ctx_null, pooled_null, time_ids)
        eps = cfg_combine(eps_c, eps_u, F(w))
    else:
        eps = eps_c
    if parts is not None:
        parts["eps_c"], parts["eps_u"] = eps_c, eps_u
    step = ddim_step_v if cfg.get("prediction", "eps") == "v" else ddim_step
    xn = step(x, eps, abar_at(abar, t), abar_at(abar, t_prev))
    return (xn, eps) if want_eps else xn


def unet_step(cfg, weights, req, only=None, want_eps=False, parts=None):
    """The step over a batch, request by request.  `req` holds latents
    (R, C, H, W), timesteps, t_prev, cfg_on, guidance, ctx_cond (R, L, D),
    ctx_uncond (L, D), schedule and, for SDXL-like configs, pooled_cond,
    pooled_uncond and time_ids.  `only` restricts the work to some requests.
    Returns {request index: x'} (and {index: eps} when want_eps); a dict
    passed as `parts` receives {index: {"eps_c": ..., "eps_u": ...}}."""
    W = weights if isinstance(weights, Weights) else Weights(weights)
    abar = alphas_cumprod(betas(req["schedule"]))
    idx = range(len(req["timesteps"])) if only is None else only
    outs, epss = {}, {}
    for r in idx:
        extra = {}
        if cfg["add_in"]:
            extra = dict(pooled=req["pooled_cond"][r], pooled_null=req["pooled_uncond"],
                         time_ids=req["time_ids"])
        p = {} if parts is not None else None
        xn, eps = unet_step_request(
            cfg, W, req["latents"][r], int(req["timesteps"][r]), int(req["t_prev"][r]),
            bool(req["cfg_on"][r]), float(req["guidance"][r]), req["ctx_cond"][r],
            req["ctx_uncond"], abar, want_eps=True, parts=p, **extra)
        if parts is not None:
            parts[r] = p
        outs[r], epss[r] = xn, eps
    return (outs, epss) if want_eps else outs
