"""Weights and request batches for a named workload.

Stream ids: weights 0, latents 1, cond context 2, uncond context 3,
timesteps 4, Skip-CFG choice 5, guidance 6, arrivals 7, step counts 8,
pooled embeddings 9.
"""
import math

import numpy as np

from .configs import CONFIGS
from .manifest import manifest
from .rng import Stream, bf16_round, normal_many

# SDXL-like micro-conditioning time ids: (orig h, orig w, crop top, crop left,
# target h, target w), the same for every request and both CFG branches.
TIME_IDS = (1024.0, 1024.0, 0.0, 0.0, 1024.0, 1024.0)


def schedule_name(workload):
    return CONFIGS[workload]["unet"]["schedule"]


def _maybe_bf16(x, unet):
    return bf16_round(x) if unet["dtype"] == "bf16" else x.astype(np.float32)


def make_weights(workload, zero=()):
    """Random-init weights {name: float32 array} for the workload's UNet.

    Weights and biases ~ N(0, 0.02); norm scales 1 + N(0, 0.02); norm shifts
    N(0, 0.02).  bf16 workloads round every value to bfloat16 so that both
    paths consume identical numbers.  Names listed in `zero` are all-zero.
    """
    unet = CONFIGS[workload]["unet"]
    man = [m for m in manifest(unet) if m[0] not in zero]
    bf = unet["dtype"] == "bf16"

    def post_w(v):
        v = (v * 0.02).astype(np.float32)
        return bf16_round(v) if bf else v

    def post_g(v):
        v = (v * 0.02).astype(np.float32) + np.float32(1.0)
        return bf16_round(v) if bf else v

    vals = normal_many([(Stream(workload, 0, name), int(np.prod(shape)),
                         post_g if kind == "g" else post_w) for name, shape, kind in man])
    out = {}
    for (name, shape, kind), v in zip(man, vals):
        out[name] = v.reshape(shape)
    for name, shape, _ in manifest(unet):
        if name in zero:
            out[name] = np.zeros(shape, np.float32)
    return {name: out[name] for name, _, _ in manifest(unet)}


def make_requests(workload, n_req=None):
    """Seeded request batch for a workload (see CONFIGS for the recipe)."""
    spec = CONFIGS[workload]
    unet = spec["unet"]
    R = n_req if n_req is not None else spec["requests"]
    C, H, W = unet["latent_c"], unet["latent_h"], unet["latent_w"]
    L, D = unet["ctx_len"], unet["ctx_dim"]
    lat = Stream(workload, 1).normal(R * C * H * W).reshape(R, C, H, W)
    ctx = _maybe_bf16(Stream(workload, 2).normal(R * L * D), unet).reshape(R, L, D)
    unc = _maybe_bf16(Stream(workload, 3).normal(L * D), unet).reshape(L, D)

    kind = spec["t"][0]
    if kind == "fixed":
        t = np.array(spec["t"][1][:R], np.int64)
    else:
        t = Stream(workload, 4).integers(0, 1000, R)

    kind = spec["cfg"][0]
    if kind == "fixed":
        cfg = np.array(spec["cfg"][1][:R], np.uint8)
    elif kind == "all":
        cfg = np.ones(R, np.uint8)
    else:  # "half": a seeded permutation picks exactly R // 2 requests to skip
        order = np.argsort(Stream(workload, 5).uniform(R), kind="stable")
        cfg = np.ones(R, np.uint8)
        cfg[order[:R // 2]] = 0

    g = spec["guidance"]
    if g[0] == "fixed":
        w = np.array(g[1][:R], np.float32)
    elif g[0] == "fixed_all":
        w = np.full(R, g[1], np.float32)
    else:
        w = (g[1] + (g[2] - g[1]) * Stream(workload, 6).uniform(R)).astype(np.float32)

    step = 1000 // unet["n_steps"]
    req = dict(latents=lat.astype(np.float32), ctx_cond=ctx, ctx_uncond=unc,
               timesteps=t, t_prev=t - step, cfg_on=cfg, guidance=w,
               schedule=unet["schedule"])
    if unet["add_in"]:
        P = unet["pooled_dim"]
        pooled = Stream(workload, 9).normal((R + 1) * P)
        req["pooled_cond"] = _maybe_bf16(pooled[:R * P], unet).reshape(R, P)
        req["pooled_uncond"] = _maybe_bf16(pooled[R * P:], unet).reshape(P)
        req["time_ids"] = np.array(TIME_IDS, np.float32)
    return req


def _poisson(u, lam):
    """Poisson(lam) sample by inversion of the CDF at the uniform u."""
    k, p = 0, math.exp(-lam)
    c = p
    while u > c and k < 1000:
        k += 1
        p *= lam / k
        c += p
    return k


def serve_arrivals(workload, iterations):
    """Arrival trace of the serving-loop workload: for each iteration the
    list of (request id, denoising steps S_r, guidance w_r) that arrive.
    Poisson(rate) arrivals per iteration, S_r uniform on the steps range,
    w_r uniform on the guidance range."""
    spec = CONFIGS[workload]
    lam = spec["arrival_rate"]
    lo, hi = spec["steps_range"]
    g = spec["guidance"]
    u = Stream(workload, 7).uniform(iterations)
    counts = [_poisson(float(x), lam) for x in u]
    total = sum(counts)
    steps = Stream(workload, 8).integers(lo, hi + 1, total)
    w = g[1] + (g[2] - g[1]) * Stream(workload, 6).uniform(total)
    out, rid = [], 0
    for c in counts:
        batch = []
        for _ in range(c):
            batch.append((rid, int(steps[rid]), float(w[rid])))
            rid += 1
        out.append(batch)
    return out


def serve_request_inputs(workload, rid):
    """Initial latent (C, H, W) and text context (L, D) of request `rid`."""
    unet = CONFIGS[workload]["unet"]
    C, H, W = unet["latent_c"], unet["latent_h"], unet["latent_w"]
    L, D = unet["ctx_len"], unet["ctx_dim"]
    lat = Stream(workload, 1, f"req{rid}").normal(C * H * W).reshape(C, H, W)
    ctx = _maybe_bf16(Stream(workload, 2, f"req{rid}").normal(L * D), unet).reshape(L, D)
    return lat.astype(np.float32), ctx


def serve_null_context(workload):
    unet = CONFIGS[workload]["unet"]
    return _maybe_bf16(Stream(workload, 3).normal(unet["ctx_len"] * unet["ctx_dim"]), unet).reshape(
        unet["ctx_len"], unet["ctx_dim"])
