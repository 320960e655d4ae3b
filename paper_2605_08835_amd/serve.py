"""Step-level continuous batching around the UNet step (SynerDiff, Sec. I and
Sec. III-A): requests join the running batch at any denoising step, every
iteration runs one UNet step for all of them, finished requests leave right
away and the batch refills from the queue.  Adaptive Skip-CFG (Sec. III-B)
drops a request's unconditional branch once it has passed a fraction of its
steps (quality threshold: early steps are CFG-sensitive, late ones are not).

The batch lives in device buffers of capacity `cap`; the active requests
occupy a contiguous prefix, so a retiring request is replaced by the last
active one (two device-to-device copies).  All denoising work is the C-ABI
step; this module only keeps per-request bookkeeping on the host.

    python -m paper_2605_08835_amd.serve --iterations 1000
prints one JSON line with rows*steps/s and the per-step device-time
p50 / p99 of the SD-1.5-shaped serving workload.
"""
import argparse
import json
import math
import os
import sys
import time
from collections import deque

import numpy as np

from .binding import UNet, alphas_cumprod, ddim_coef


class ContinuousBatcher:
    def __init__(self, model, cap, schedule, skip_after=0.6, device="cuda"):
        import torch
        self.torch = torch
        self.m = model
        u = model.unet
        self.cap = cap
        self.skip_after = skip_after
        self.abar = alphas_cumprod(schedule)
        dev = torch.device(device)
        self.lat = torch.empty(cap, u["latent_c"], u["latent_h"], u["latent_w"], device=dev)
        self.ctx = torch.empty(cap, u["ctx_len"], u["ctx_dim"], device=dev, dtype=model.act_dtype)
        self.ids = [None] * cap
        self.k = np.zeros(cap, np.int64)
        self.S = np.zeros(cap, np.int64)
        self.w = np.zeros(cap, np.float32)
        self.n = 0
        self.null_ctx = None
        self.coef_cache = {}

    def set_null_context(self, ctx):
        self.null_ctx = ctx

    def admit(self, rid, latent, ctx, n_steps, guidance):
        """Place a request (device latent (C, H, W), context (L, D)) in the batch."""
        i = self.n
        self.lat[i].copy_(latent)
        self.ctx[i].copy_(ctx)
        self.ids[i], self.k[i], self.S[i], self.w[i] = rid, 0, n_steps, guidance
        self.n += 1

    def plan(self):
        """Per-request timestep, previous timestep and Skip-CFG flag of the
        coming step: S_r steps of size floor(1000 / S_r), t_k = (S_r-1-k) step,
        CFG kept while k < ceil(skip_after * S_r)."""
        n = self.n
        S, k = self.S[:n], self.k[:n]
        step = 1000 // S
        t = (S - 1 - k) * step
        tp = t - step
        cfg = (k < np.ceil(self.skip_after * S)).astype(np.uint8)
        return t.astype(np.int32), tp.astype(np.int32), cfg

    def coefficients(self, t, tp):
        out = np.empty((len(t), 2), np.float32)
        for i, (a, b) in enumerate(zip(t, tp)):
            key = (int(a), int(b))
            if key not in self.coef_cache:
                self.coef_cache[key] = ddim_coef(self.abar, a, b)
            out[i] = self.coef_cache[key]
        return out

    def step(self, eps_out=None, stream=None):
        """One UNet step for every active request (in place).  Returns the
        step inputs (for replay) and the list of retired (id, slot) pairs;
        retired slots are refilled from the end of the batch."""
        n = self.n
        t, tp, cfg = self.plan()
        coef = self.coefficients(t, tp)
        inputs = dict(t=t, t_prev=tp, cfg_on=cfg, guidance=self.w[:n].copy(), coef=coef,
                      ids=list(self.ids[:n]), n=n)
        self.m.step(self.lat[:n], t, cfg, self.w[:n], self.ctx[:n], self.null_ctx, coef, out=self.lat[:n],
                    eps_out=eps_out, stream=stream)
        self.k[:n] += 1
        return inputs

    def retire(self):
        """Remove finished requests; returns their ids and final latents."""
        done = []
        i = 0
        while i < self.n:
            if self.k[i] >= self.S[i]:
                done.append((self.ids[i], self.lat[i].clone()))
                last = self.n - 1
                if i != last:
                    self.lat[i].copy_(self.lat[last])
                    self.ctx[i].copy_(self.ctx[last])
                    self.ids[i], self.k[i], self.S[i], self.w[i] = \
                        self.ids[last], self.k[last], self.S[last], self.w[last]
                self.n -= 1
            else:
                i += 1
        return done


def run(workload="c5_sd15_serve", iterations=1000, weights=None, log=None, snapshot_at=()):
    """Serve the workload's arrival trace for `iterations` iterations.
    Returns a result dict (and the snapshots requested by iteration index:
    the step inputs, the latents before and after the step)."""
    import torch

    from fixtures import (get_config, make_weights, serve_arrivals, serve_null_context,
                          serve_request_inputs)
    spec = get_config(workload)
    unet = spec["unet"]
    cap = spec["requests"]
    if weights is None:
        weights = make_weights(workload)
    m = UNet(unet, max_requests=cap)
    m.load_weights(weights)
    dev = torch.device("cuda")
    act = m.act_dtype
    b = ContinuousBatcher(m, cap, unet["schedule"], spec["skip_after"])
    b.set_null_context(torch.from_numpy(serve_null_context(workload)).to(dev).to(act))
    arrivals = serve_arrivals(workload, iterations)
    queue = deque()
    stream = torch.cuda.current_stream(dev)
    ev = []
    rows_total, req_steps, finished = 0, 0, 0
    host_ms = []
    snaps = {}
    for it in range(iterations):
        for rid, S, w in arrivals[it]:
            queue.append((rid, S, w))
        while queue and b.n < cap:
            rid, S, w = queue.popleft()
            lat, ctx = serve_request_inputs(workload, rid)
            b.admit(rid, torch.from_numpy(lat).to(dev), torch.from_numpy(ctx).to(dev).to(act), S, w)
        if b.n == 0:
            continue
        before = b.lat[:b.n].clone() if it in snapshot_at else None
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        h0 = time.perf_counter()
        e0.record(stream)
        inp = b.step(stream=stream)
        e1.record(stream)
        host_ms.append(1e3 * (time.perf_counter() - h0))
        ev.append((e0, e1))
        rows_total += int(inp["n"] + inp["cfg_on"].sum())
        req_steps += inp["n"]
        if before is not None:
            snaps[it] = dict(inputs=inp, before=before.cpu().numpy(), after=b.lat[:b.n].cpu().numpy(),
                             ctx=b.ctx[:b.n].float().cpu().numpy())
        finished += len(b.retire())
        if log and it % 100 == 0:
            log(f"iteration {it}: active {b.n}, queued {len(queue)}, finished {finished}")
    torch.cuda.synchronize()
    dev_ms = np.array([a.elapsed_time(c) for a, c in ev])
    m.close()
    res = {
        "workload": "SD-1.5-shaped UNet, 64x64 latents, bf16; Poisson(4) arrivals per iteration, "
                    "20-50 steps per request, batch cap 32, Skip-CFG after 60% of a request's steps",
        "iterations": iterations, "steps_run": len(dev_ms), "finished": finished, "queued_at_end": len(queue),
        "rows_steps_per_s": rows_total / (dev_ms.sum() / 1e3),
        "request_steps_per_s": req_steps / (dev_ms.sum() / 1e3),
        "mean_rows": rows_total / max(len(dev_ms), 1),
        "step_ms_p50": float(np.percentile(dev_ms, 50)), "step_ms_p99": float(np.percentile(dev_ms, 99)),
        "host_ms_p50": float(np.percentile(host_ms, 50)), "host_ms_p99": float(np.percentile(host_ms, 99)),
    }
    return res, snaps


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--iterations", type=int, default=1000)
    ap.add_argument("--workload", default="c5_sd15_serve")
    args = ap.parse_args()
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    res, _ = run(args.workload, args.iterations, log=lambda s: print(s, file=sys.stderr, flush=True))
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
