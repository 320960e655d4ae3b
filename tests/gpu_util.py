"""Helpers for the GPU parity tests: run the HIP step through the binding and
compare with the oracle (relative L2 in float64)."""
import numpy as np


def rel_l2(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


def to_dev(x, dtype):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(dtype)


def gpu_step(model, req, only_n=None, out_inplace=False, eps=True):
    """One step of `model` (a paper_2605_08835_amd.UNet) on request batch
    `req`; returns (latents_out, eps) as float64 numpy arrays."""
    import torch
    act = model.act_dtype
    lat = to_dev(req["latents"], torch.float32)
    ctx = to_dev(req["ctx_cond"], act)
    unc = to_dev(req["ctx_uncond"], act)
    coef = model.coefficients(req["schedule"], req["timesteps"], req["t_prev"])
    e = torch.empty_like(lat) if eps else None
    kw = {}
    if "pooled_cond" in req:
        kw = dict(pooled_cond=to_dev(req["pooled_cond"], torch.float32),
                  pooled_uncond=to_dev(req["pooled_uncond"], torch.float32), time_ids=req["time_ids"])
    out = model.step(lat, req["timesteps"], req["cfg_on"], req["guidance"], ctx, unc, coef,
                     out=lat if out_inplace else None, eps_out=e, **kw)
    torch.cuda.synchronize()
    return out.cpu().double().numpy(), (e.cpu().double().numpy() if eps else None)


def log(msg):
    print(msg, flush=True)
