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

With VAE Chunking (Sec. III-B) finished latents queue for decoding; a
decode job of up to `vae_batch` images runs in c chunks on a second stream,
one chunk beside each UNet step, and both streams join at the end of every
iteration (one concurrent round).  The load-adaptive feedback controller
(Sec. III-D) sets the Skip-CFG threshold and c from the queue length.

    python -m paper_2605_08835_amd.serve --iterations 1000 [--vae vae_sd15
        --chunks C --controller --c-max CMAX]
prints one JSON line with rows*steps/s (device time and wall clock), the
per-iteration device-time p50 / p99, request latencies in iterations and,
with a VAE, images decoded per second.
"""
import argparse
import json
import math
import os
import sys
import time
from collections import deque

import numpy as np

from .binding import VAE, UNet, alphas_cumprod, ddim_coef, vae_chunk_plan
from .control import FeedbackController


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

    def permute(self, order):
        """Reorder the active prefix: slot i takes the request in slot order[i]."""
        n = self.n
        idx = self.torch.as_tensor(np.asarray(order, np.int64), device=self.lat.device)
        self.lat[:n] = self.lat[:n].index_select(0, idx)
        self.ctx[:n] = self.ctx[:n].index_select(0, idx)
        o = np.asarray(order)
        self.ids[:n] = [self.ids[i] for i in order]
        self.k[:n], self.S[:n], self.w[:n] = self.k[:n][o], self.S[:n][o], self.w[:n][o]

    def step_range(self, lo, hi, cfg, stream=None):
        """One UNet step for the requests in slots [lo, hi) with the given
        CFG flags (a request past its threshold may still run with CFG)."""
        t, tp, _ = self.plan()
        t, tp = t[lo:hi], tp[lo:hi]
        coef = self.coefficients(t, tp)
        self.m.step(self.lat[lo:hi], t, np.asarray(cfg, np.uint8), self.w[lo:hi], self.ctx[lo:hi], self.null_ctx,
                    coef, out=self.lat[lo:hi], stream=stream)
        self.k[lo:hi] += 1

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


def _stage_ms(vae, z, stream, reps=3):
    """Solo milliseconds of every decoder stage for the batch z (median of reps)."""
    import torch
    ns = len(vae.stages)
    acc = np.zeros((reps, ns))
    img = torch.empty(vae.image_shape(z.shape[0]), device=z.device)
    for r in range(reps + 1):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(ns)]
        for i in range(ns):
            evs[i][0].record(stream)
            vae.run(z, i, i + 1, image=img, stream=stream)
            evs[i][1].record(stream)
        torch.cuda.synchronize()
        if r:  # the first pass warms up
            acc[r - 1] = [a.elapsed_time(b) for a, b in evs]
    return np.median(acc, axis=0)


class VaeChunker:
    """VAE Chunking in the serving loop (Sec. III-B): finished latents queue
    for decoding; a decode job of up to `batch` images runs in c chunks of
    about equal solo time, one chunk per iteration on its own stream,
    concurrently with that iteration's UNet step."""

    def __init__(self, vae, batch, stream, keep=False):
        import torch
        self.torch = torch
        self.v = vae
        self.batch = batch
        self.stream = stream
        self.keep = keep
        self.kept = []           # with keep: (ids, latents, images) of every finished job
        self.z = None
        self.img = None
        self.pending = deque()  # (request id, latent [C, H, W] device tensor)
        self.job = None          # dict(ids, n, bounds, next)
        self.stage_cost = None
        self.plans = {}
        self.done = []           # (request id, iteration the decode finished)

    def setup(self, latent_shape, device):
        torch = self.torch
        self.z = torch.zeros((self.batch,) + tuple(latent_shape), device=device)
        self.img = torch.empty(self.v.image_shape(self.batch), device=device)
        self.stage_cost = _stage_ms(self.v, self.z[:1], self.stream)

    def bounds(self, c):
        c = max(1, min(c, len(self.v.stages)))
        if c not in self.plans:
            self.plans[c] = vae_chunk_plan(self.stage_cost, c)
        return self.plans[c]

    def start_job(self, c, stream):
        """Take up to `batch` pending latents (copied on `stream`, the UNet's,
        after the step that finished them) as the next decode job."""
        if self.job is not None or not self.pending:
            return
        ids = []
        while self.pending and len(ids) < self.batch:
            rid, lat = self.pending.popleft()
            with self.torch.cuda.stream(stream):
                self.z[len(ids)].copy_(lat)
            ids.append(rid)
        self.job = dict(ids=ids, n=len(ids), bounds=self.bounds(c), next=0)

    def run_chunk(self, it):
        """Enqueue the job's next chunk on the VAE stream; returns True if one ran."""
        j = self.job
        if j is None:
            return False
        b, e = j["bounds"][j["next"]], j["bounds"][j["next"] + 1]
        self.v.run(self.z[:j["n"]], b, e, image=self.img[:j["n"]], stream=self.stream)
        j["next"] += 1
        if j["next"] == len(j["bounds"]) - 1:
            self.done += [(rid, it) for rid in j["ids"]]
            if self.keep:
                with self.torch.cuda.stream(self.stream):
                    self.kept.append((j["ids"], self.z[:j["n"]].clone(), self.img[:j["n"]].clone()))
            self.job = None
        return True


def run(workload="c5_sd15_serve", iterations=1000, weights=None, log=None, snapshot_at=(), vae=None,
        vae_batch=4, chunks=1, controller=None, keep_images=False):
    """Serve the workload's arrival trace for `iterations` iterations.
    Returns a result dict (and the snapshots requested by iteration index:
    the step inputs, the latents before and after the step).

    vae: a VAE-decoder configuration name (fixtures.vae) to decode finished
    requests with VAE Chunking on a second stream, `chunks` chunks per decode
    job of up to `vae_batch` images; controller: a FeedbackController that
    sets the Skip-CFG threshold and the chunk count from the queue length
    every iteration (Sec. III-D); keep_images: return every decode job's
    latents and images under snaps["images"]."""
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
    vz = None
    if vae is not None:
        from fixtures.vae import VAE_CONFIGS, make_vae_weights
        vcfg = dict(VAE_CONFIGS[vae]["vae"])
        vh = VAE(vcfg, max_images=vae_batch, device=dev)
        vh.load_weights(make_vae_weights(vae))
        vz = VaeChunker(vh, vae_batch, torch.cuda.Stream(device=dev), keep=keep_images)  # default priority
        vz.setup((unet["latent_c"], unet["latent_h"], unet["latent_w"]), dev)
    if controller is not None:
        b.skip_after = controller.skip_after
        chunks = controller.c
    ev = []
    rows_total, req_steps, finished = 0, 0, 0
    host_ms = []
    snaps = {}
    arrived_at = {}
    finished_at = {}
    vae_rounds = 0
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for it in range(iterations):
        for rid, S, w in arrivals[it]:
            queue.append((rid, S, w))
            arrived_at[rid] = it
        if controller is not None:
            b.skip_after, chunks = controller.update(len(queue))
        while queue and b.n < cap:
            rid, S, w = queue.popleft()
            lat, ctx = serve_request_inputs(workload, rid)
            b.admit(rid, torch.from_numpy(lat).to(dev), torch.from_numpy(ctx).to(dev).to(act), S, w)
        if b.n == 0 and (vz is None or vz.job is None):
            continue
        before = b.lat[:b.n].clone() if it in snapshot_at else None
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        h0 = time.perf_counter()
        if vz is not None:
            # one concurrent round: both streams start after both finished
            # the previous round (and the VAE stream after the latent copies)
            stream.wait_stream(vz.stream)
            vz.stream.wait_stream(stream)
        e0.record(stream)
        inp = None
        if b.n:
            inp = b.step(stream=stream)
        if vz is not None:
            vae_rounds += int(vz.run_chunk(it))
            stream.wait_stream(vz.stream)
        e1.record(stream)
        host_ms.append(1e3 * (time.perf_counter() - h0))
        ev.append((e0, e1))
        if inp is not None:
            rows_total += int(inp["n"] + inp["cfg_on"].sum())
            req_steps += inp["n"]
            if before is not None:
                snaps[it] = dict(inputs=inp, before=before.cpu().numpy(), after=b.lat[:b.n].cpu().numpy(),
                                 ctx=b.ctx[:b.n].float().cpu().numpy())
        done = b.retire()
        finished += len(done)
        for rid, lat in done:
            finished_at[rid] = it
            if vz is not None:
                vz.pending.append((rid, lat))
        if vz is not None:
            vz.start_job(chunks, stream)
        if log and it % 100 == 0:
            extra = f", decode queue {len(vz.pending)}" if vz is not None else ""
            ctl = f", skip_after {b.skip_after:.2f}, c {chunks}" if controller is not None else ""
            log(f"iteration {it}: active {b.n}, queued {len(queue)}, finished {finished}{extra}{ctl}")
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - wall0
    dev_ms = np.array([a.elapsed_time(c) for a, c in ev])
    m.close()
    lo, hi = spec["steps_range"]
    desc = (f"{workload}: {unet['dtype']} UNet, {unet['latent_h']}x{unet['latent_w']} latents, widths {unet['ch']}; "
            f"Poisson({spec['arrival_rate']:g}) arrivals per iteration, {lo}-{hi} steps per request, batch cap {cap}, "
            f"Skip-CFG after {100 * spec['skip_after']:.0f}% of a request's steps")
    if vz is not None:
        desc += f"; VAE decoder {vae} on a second stream, jobs of up to {vae_batch} images"
    if controller is not None:
        desc += "; feedback controller on the queue length"
    res = {
        "workload": desc,
        "iterations": iterations, "steps_run": len(dev_ms), "finished": finished, "queued_at_end": len(queue),
        "rows_steps_per_s": rows_total / (dev_ms.sum() / 1e3),
        "request_steps_per_s": req_steps / (dev_ms.sum() / 1e3),
        "rows_steps_per_s_wall": rows_total / wall_s, "wall_s": wall_s,
        "mean_rows": rows_total / max(len(dev_ms), 1),
        "step_ms_p50": float(np.percentile(dev_ms, 50)), "step_ms_p99": float(np.percentile(dev_ms, 99)),
        "host_ms_p50": float(np.percentile(host_ms, 50)), "host_ms_p99": float(np.percentile(host_ms, 99)),
    }
    lat_it = [finished_at[r] - arrived_at[r] + 1 for r in finished_at]
    if lat_it:
        res["denoise_latency_iterations_p50"] = float(np.percentile(lat_it, 50))
        res["denoise_latency_iterations_p99"] = float(np.percentile(lat_it, 99))
    if vz is not None:
        img_it = [it - arrived_at[r] + 1 for r, it in vz.done]
        res.update(images_decoded=len(vz.done), vae_chunk_rounds=vae_rounds,
                   images_per_s=len(vz.done) / (dev_ms.sum() / 1e3),
                   decode_queue_at_end=len(vz.pending) + (vz.job["n"] if vz.job else 0),
                   chunk_bounds={str(c): bb for c, bb in vz.plans.items()},
                   stage_ms=[round(float(x), 4) for x in vz.stage_cost])
        if img_it:
            res["image_latency_iterations_p50"] = float(np.percentile(img_it, 50))
            res["image_latency_iterations_p99"] = float(np.percentile(img_it, 99))
        if keep_images:
            torch.cuda.synchronize()
            snaps["images"] = [(ids, z.cpu().numpy(), im.cpu().numpy()) for ids, z, im in vz.kept]
        vz.v.close()
    if controller is not None:
        res["controller"] = dict(final_skip_after=controller.skip_after, final_c=controller.c,
                                 changes=controller.log[:50], n_changes=len(controller.log))
    return res, snaps


def assign_stages(seq, cfg):
    """Slot order and CFG flags for a stage sequence [(m, n, k)] (Problem P,
    Sec. III-D) over the requests of one window: stage t takes k_t requests
    past their Skip-CFG threshold (cfg 0), which run without CFG, then
    m_t - k_t others with CFG (requests still under their threshold first;
    past-threshold ones fill in when those run out).  Returns (order, flags,
    stage bounds)."""
    elig = [i for i in range(len(cfg)) if cfg[i] == 0]
    rest = [i for i in range(len(cfg)) if cfg[i] != 0]
    order, flags, bounds = [], [], [0]
    for m, _, k in seq:
        take = [elig.pop(0) for _ in range(k)]
        flags += [0] * k
        for _ in range(m - k):
            take.append(rest.pop(0) if rest else elig.pop(0))
            flags.append(1)
        order += take
        bounds.append(len(order))
    if elig or rest or len(order) != len(cfg):
        raise ValueError("stage sequence does not cover the window's requests")
    return order, flags, bounds


def run_planned(workload="c5_sd15_serve", iterations=300, lut=None, policy="exact", vae="vae_sd15", nmax=4,
                alpha=0.1, saturate=True, log=None):
    """The serving loop driven by the inter-concurrency scheduler (Sec.
    III-D): every window gives each active request one step; the M steps, the
    N finished images waiting for decoding (at most nmax) and the K requests
    past their Skip-CFG threshold are split into concurrent stages (m_t, n_t,
    k_t) by the planner on the offline lookup table (`lut`: the profiler's
    lookup grid), each stage one UNet step over m_t requests beside one
    whole decode of n_t images on a second stream.  policy: "single" (one
    stage: every step and every decode together), "alg1" (Alg. 1) or
    "exact" (the optimum of Problem P).  T_lim = (1 + alpha) tau(M, N, K).
    The objective counts only the decodes' completion times, so where no
    decode is waiting every stage split ties and the planner returns its
    first (fewest skips); with saturate, every request past its threshold
    skips CFG in whichever stage it lands, which only shortens the stages
    (the latency cap still holds) and keeps the Skip-CFG rule of the other
    loops."""
    import torch

    from fixtures import (get_config, make_weights, serve_arrivals, serve_null_context,
                          serve_request_inputs)
    from fixtures.vae import VAE_CONFIGS, make_vae_weights

    from .binding import SynerDiffError, plan_sequence
    from .profiler import dense_table
    spec = get_config(workload)
    unet = spec["unet"]
    cap = spec["requests"]
    m = UNet(unet, max_requests=cap)
    m.load_weights(make_weights(workload))
    dev = torch.device("cuda")
    act = m.act_dtype
    b = ContinuousBatcher(m, cap, unet["schedule"], spec["skip_after"])
    b.set_null_context(torch.from_numpy(serve_null_context(workload)).to(dev).to(act))
    vh = VAE(dict(VAE_CONFIGS[vae]["vae"]), max_images=nmax, device=dev)
    vh.load_weights(make_vae_weights(vae))
    ns = len(vh.stages)
    z = torch.zeros((nmax, unet["latent_c"], unet["latent_h"], unet["latent_w"]), device=dev)
    img = torch.empty(vh.image_shape(nmax), device=dev)
    tau, delta = dense_table(lut, cap)
    arrivals = serve_arrivals(workload, iterations)
    queue, pending = deque(), deque()  # pending: (request id, latent, index of the stage that finished it)
    us, vs = torch.cuda.current_stream(dev), torch.cuda.Stream(device=dev)  # default priorities
    stages = []  # (start event, end event)
    finished_at, decoded_at = {}, {}
    plans, fallbacks, rows_total, req_steps = 0, 0, 0, 0
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for it in range(iterations):
        for rid, S, w in arrivals[it]:
            queue.append((rid, S, w))
        while queue and b.n < cap:
            rid, S, w = queue.popleft()
            lat, ctx = serve_request_inputs(workload, rid)
            b.admit(rid, torch.from_numpy(lat).to(dev), torch.from_numpy(ctx).to(dev).to(act), S, w)
        M = b.n
        N = min(len(pending), nmax, max(M, 1))
        if M == 0 and N == 0:
            continue
        _, _, cfg = b.plan()
        K = int((cfg == 0).sum())
        if M == 0:
            seq = [(0, N, 0)]  # no request to step: a decode-only stage
        elif policy == "single":
            seq = [(M, N, K)]
        else:
            try:
                seq, _, _ = plan_sequence(M, N, K, tau, delta, (1 + alpha) * tau[M, N, K], exact=policy == "exact")
                plans += 1
            except SynerDiffError:
                seq = [(M, N, K)]
                fallbacks += 1
        order, flags, bounds = assign_stages(seq, cfg) if M else ([], [], [0, 0])
        if M:
            b.permute(order)
            if saturate:
                flags = [int(cfg[o]) for o in order]
        for si, (mt, nt, kt) in enumerate(seq):
            vs.wait_stream(us)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(us)
            job = []
            for j in range(nt):
                rid, lat, _ = pending.popleft()
                with torch.cuda.stream(us):
                    z[j].copy_(lat)
                job.append(rid)
            if nt:
                vs.wait_stream(us)
                vh.run(z[:nt], 0, ns, image=img[:nt], stream=vs)
            lo, hi = bounds[si], bounds[si + 1]
            if hi > lo:
                b.step_range(lo, hi, flags[lo:hi], stream=us)
            rows_total += (hi - lo) + int(sum(flags[lo:hi]))
            req_steps += hi - lo
            us.wait_stream(vs)
            e1.record(us)
            stages.append((e0, e1))
            for rid in job:
                decoded_at[rid] = len(stages) - 1
            for i in range(lo, hi):
                if b.k[i] >= b.S[i]:
                    finished_at[b.ids[i]] = len(stages) - 1
        for rid, lat in b.retire():
            pending.append((rid, lat, finished_at[rid]))
        if log and it % 50 == 0:
            log(f"window {it}: active {b.n}, queued {len(queue)}, decode queue {len(pending)}, stages {len(seq)}")
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - wall0
    dur = np.array([a.elapsed_time(c) for a, c in stages])
    end = np.cumsum(dur)
    waits = [end[decoded_at[r]] - end[finished_at[r]] for r in decoded_at]
    m.close()
    vh.close()
    res = {
        "workload": workload, "policy": policy, "windows": iterations, "stages": len(stages),
        "plans": plans, "fallbacks": fallbacks, "device_ms": float(dur.sum()), "wall_s": wall_s,
        "rows_steps_per_s": rows_total / dur.sum() * 1e3, "request_steps_per_s": req_steps / dur.sum() * 1e3,
        "images_decoded": len(decoded_at), "images_per_s": len(decoded_at) / dur.sum() * 1e3,
        "decode_wait_ms_mean": float(np.mean(waits)) if waits else None,
        "decode_wait_ms_p50": float(np.percentile(waits, 50)) if waits else None,
        "decode_wait_ms_p99": float(np.percentile(waits, 99)) if waits else None,
    }
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--iterations", type=int, default=1000)
    ap.add_argument("--workload", default="c5_sd15_serve")
    ap.add_argument("--vae", default="", help="decode finished requests with this VAE (e.g. vae_sd15)")
    ap.add_argument("--vae-batch", type=int, default=4)
    ap.add_argument("--chunks", type=int, default=1, help="VAE Chunking granularity c")
    ap.add_argument("--controller", action="store_true", help="load-adaptive feedback controller")
    ap.add_argument("--c-max", type=int, default=4)
    ap.add_argument("--planner", choices=["single", "alg1", "exact"], default=None,
                    help="windows planned by the inter-concurrency scheduler on --lut")
    ap.add_argument("--lut", default="", help="offline profile JSON (paper_2605_08835_amd.profiler --out)")
    args = ap.parse_args()
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    if args.planner:
        with open(args.lut) as f:
            grid = json.load(f)["lookup_grid"]
        res = run_planned(args.workload, args.iterations, lut=grid, policy=args.planner, vae=args.vae or "vae_sd15",
                          nmax=args.vae_batch, log=lambda s: print(s, file=sys.stderr, flush=True))
        print(json.dumps(res), flush=True)
        return
    ctl = FeedbackController(c0=args.chunks, c_max=max(args.c_max, args.chunks)) if args.controller else None
    res, _ = run(args.workload, args.iterations, log=lambda s: print(s, file=sys.stderr, flush=True),
                 vae=args.vae or None, vae_batch=args.vae_batch, chunks=args.chunks, controller=ctl)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
