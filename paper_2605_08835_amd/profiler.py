"""Offline profiler (Sec. III-A component A, Sec. III-C): micro-benchmarks of
the UNet step and the VAE decoder on this GPU that fix the static
configuration the scheduler works with.

* VAE Chunking granularity: for c = 1..C_max the decoder is split into c
  chunks of about equal solo time at ResNet-block boundaries, and each chunk
  runs on its own stream concurrently with one UNet step (one concurrent
  round).  From the per-round latencies t_u^i (UNet) and t_v^i (VAE chunk),
  Eq. (2) gives the cumulative latencies T_u(c), T_v(c) and Eq. (1) the cost
  L(c) against the solo latencies; the chosen c minimises L.
* The concurrent-latency lookup table T^c(m, n, k): tau = latency of a round
  with m UNet requests (k of them under Skip-CFG) and the first chunk of a
  c-chunk decode of n images, delta = that chunk's latency.
* B_max: the request count beyond which a step's throughput stops growing.

Readings (the paper leaves them open): T_u0 is c solo UNet steps and T_v0
one solo decode, so L(c) compares the same work with and without
concurrency; C_max is the smallest c whose UNet overhead
(T_u(c) - T_u0) / T_u0 is within 5 % (finer chunking no longer helps the
UNet and only lengthens the decode), capped at the stage count; B_max is the
smallest batch whose throughput is within 5 % of the largest measured.  The
table is measured on a grid of (m, n, k / m) and filled in between by
multilinear interpolation, since a dense table would take hours of GPU time
for a 32-request batch.

All GPU work is the library's (synerdiff_unet_step, synerdiff_vae_run);
this module only times it with HIP events and does the bookkeeping.

    python -m paper_2605_08835_amd.profiler --out profile.json
profiles the SD-1.5-shaped UNet (32 requests) beside the SD-1.5 VAE decoder
and writes the chunking table, the lookup-table grid, B_max and a planned
stage sequence as JSON.
"""
import argparse
import json
import os
import sys

import numpy as np

from .binding import chunk_cost, plan_sequence, vae_chunk_plan


def _events(torch):
    return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)


class Profiler:
    def __init__(self, unet_model, unet_inputs, vae_model, vae_latents):
        """unet_inputs: dict(latents, timesteps, cfg_on, guidance, ctx_cond,
        ctx_uncond, coef) of a full batch (device tensors / host arrays);
        vae_latents: fp32 device tensor [n, C, H, W]."""
        import torch
        self.torch = torch
        self.m = unet_model
        self.u = unet_inputs
        self.v = vae_model
        self.z = vae_latents
        self.sa = torch.cuda.Stream()  # default priority
        self.sb = torch.cuda.Stream()
        self.out = torch.empty_like(unet_inputs["latents"])
        self.img = torch.empty(vae_model.image_shape(vae_latents.shape[0]), device=vae_latents.device)
        self.n_stages = len(vae_model.stages)

    # ------------------------------------------------------------ launches
    def _unet(self, n=None, skip=None, stream=None):
        """One step of the first n requests; with skip = k, the first k run
        without CFG and the rest with it."""
        u = self.u
        n = len(u["timesteps"]) if n is None else n
        cfg = np.array(u["cfg_on"][:n], np.uint8)
        if skip is not None:
            cfg[:] = 1
            cfg[:skip] = 0
        self.m.step(u["latents"][:n], u["timesteps"][:n], cfg, u["guidance"][:n], u["ctx_cond"][:n],
                    u["ctx_uncond"], u["coef"][:n], out=self.out[:n], stream=stream)

    def _vae(self, b, e, n=None, stream=None):
        n = self.z.shape[0] if n is None else n
        self.v.run(self.z[:n], b, e, image=self.img[:n], stream=stream)

    def _time(self, fn, stream, reps=3):
        torch = self.torch
        ts = []
        for _ in range(reps):
            e0, e1 = _events(torch)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    # ---------------------------------------------------------- solo costs
    def stage_times(self, reps=3, n=None):
        """Solo milliseconds of every decoder stage (one full decode per rep)."""
        torch = self.torch
        ns = self.n_stages
        acc = np.zeros((reps, ns))
        for r in range(reps):
            evs = [_events(torch) for _ in range(ns)]
            for i in range(ns):
                evs[i][0].record(self.sb)
                self._vae(i, i + 1, n, stream=self.sb)
                evs[i][1].record(self.sb)
            torch.cuda.synchronize()
            acc[r] = [a.elapsed_time(b) for a, b in evs]
        return np.median(acc, axis=0)

    def solo(self, reps=5):
        """Solo milliseconds of one full-batch UNet step and one decode."""
        ns = self.n_stages
        self._unet(stream=self.sa)
        self._vae(0, ns, stream=self.sb)
        self.torch.cuda.synchronize()
        t_u = self._time(lambda: self._unet(stream=self.sa), self.sa, reps)
        t_v = self._time(lambda: self._vae(0, ns, stream=self.sb), self.sb, reps)
        return t_u, t_v

    # ------------------------------------------------------- concurrency
    def rounds(self, bounds, n_unet=None, skip=None, n_vae=None):
        """One decode in len(bounds) - 1 chunks, chunk i concurrent with UNet
        step i on the other stream; returns per-round (t_u, t_v) in ms.  The
        chunks cover the stage range [bounds[0], bounds[-1])."""
        torch = self.torch
        res = []
        for b, e in zip(bounds[:-1], bounds[1:]):
            ua, ub = _events(torch)
            va, vb = _events(torch)
            torch.cuda.synchronize()
            ua.record(self.sa)
            va.record(self.sb)
            self._unet(n_unet, skip, stream=self.sa)
            self._vae(b, e, n_vae, stream=self.sb)
            ub.record(self.sa)
            vb.record(self.sb)
            torch.cuda.synchronize()
            res.append((ua.elapsed_time(ub), va.elapsed_time(vb)))
        return res

    def choose_chunking(self, lam=0.5, c_limit=None, reps=3, overhead=0.05):
        """Eq. (1)-(2) over c = 1..C_max; returns a dict with every c's
        T_u, T_v, L, the chunk bounds, C_max and the chosen c."""
        ns = self.n_stages
        st = self.stage_times()
        t_u, t_v = self.solo()
        c_limit = min(c_limit or ns, ns)
        table = []
        c_max = c_limit
        for c in range(1, c_limit + 1):
            bounds = vae_chunk_plan(st, c)
            per = np.median(np.array([self.rounds(bounds) for _ in range(reps)]), axis=0)
            Tu, Tv, L = chunk_cost(per[:, 0], per[:, 1], c * t_u, t_v, lam)
            table.append(dict(c=c, bounds=bounds, t_u=per[:, 0].tolist(), t_v=per[:, 1].tolist(),
                              T_u=Tu, T_v=Tv, T_u0=c * t_u, T_v0=t_v, L=L,
                              unet_overhead=(Tu - c * t_u) / (c * t_u), vae_overhead=(Tv - t_v) / t_v))
            if (Tu - c * t_u) / (c * t_u) <= overhead:
                c_max = c
                break
        best = min(table, key=lambda r: r["L"])
        return dict(stage_ms=st.tolist(), stages=list(self.v.stages), t_u_solo=t_u, t_v_solo=t_v, lam=lam,
                    overhead_limit=overhead, C_max=c_max, chosen_c=best["c"], rounds=table)

    def lookup_grid(self, c, m_grid, n_grid, k_fracs=(0.0, 0.5, 1.0), reps=2):
        """tau and delta (ms) on the grid: m requests (k = round(f m) of them
        under Skip-CFG), the first chunk of a c-chunk decode of n images
        (n = 0: the step alone, delta = 0).  Returns a dict with the grid and
        arrays [len(m_grid)][len(n_grid)][len(k_fracs)]."""
        ns = self.n_stages
        bounds = vae_chunk_plan(self.stage_times(reps=1), c)
        first = bounds[:2]
        tau = np.zeros((len(m_grid), len(n_grid), len(k_fracs)))
        delta = np.zeros_like(tau)
        for a, m in enumerate(m_grid):
            for b, n in enumerate(n_grid):
                for f, kf in enumerate(k_fracs):
                    k = int(round(kf * m))
                    vals = []
                    for _ in range(reps):
                        if n:
                            r = self.rounds(first, n_unet=m, skip=k, n_vae=n)[0]
                            if first[1] < ns:  # finish the decode
                                self._vae(first[1], ns, n, stream=self.sb)
                                self.torch.cuda.synchronize()
                        else:
                            r = (self._time(lambda: self._unet(m, k, stream=self.sa), self.sa, 1), 0.0)
                        vals.append(r)
                    t = np.median(np.array(vals), axis=0)
                    tau[a, b, f] = max(t[0], t[1])
                    delta[a, b, f] = t[1]
        return dict(c=c, first_chunk=first, m_grid=list(m_grid), n_grid=list(n_grid), k_fracs=list(k_fracs),
                    tau=tau.tolist(), delta=delta.tolist())

    def saturation_batch(self, counts, reps=3, tol=0.05):
        """Step throughput (requests / s) per request count; B_max is the
        smallest count within tol of the best."""
        thr = {}
        for n in counts:
            t = self._time(lambda: self._unet(n, stream=self.sa), self.sa, reps)
            thr[n] = n * 1e3 / t
        best = max(thr.values())
        bmax = min(n for n in counts if thr[n] >= (1 - tol) * best)
        return bmax, thr


def _interp1(grid, x):
    """Bracketing indices and weight of x on a sorted grid (clamped at the ends)."""
    g = np.asarray(grid, np.float64)
    if x <= g[0]:
        return 0, 0, 0.0
    if x >= g[-1]:
        return len(g) - 1, len(g) - 1, 0.0
    j = int(np.searchsorted(g, x, side="right"))
    i = j - 1
    return i, j, float((x - g[i]) / (g[j] - g[i]))


def dense_table(grid, bmax):
    """The planner's tau[m][n][k], delta[m][n][k] ((bmax + 1)^3, 1 <= m <=
    bmax, n, k <= m) from a lookup grid by multilinear interpolation in m,
    n and k / m; n beyond the grid takes its largest n."""
    t = np.asarray(grid["tau"], np.float64)
    d = np.asarray(grid["delta"], np.float64)
    B = bmax + 1
    tau = np.zeros((B, B, B))
    delta = np.zeros((B, B, B))
    for m in range(1, B):
        im, jm, wm = _interp1(grid["m_grid"], m)
        for n in range(m + 1):
            i_n, j_n, wn = _interp1(grid["n_grid"], n)
            for k in range(m + 1):
                ik, jk, wk = _interp1(grid["k_fracs"], k / m)
                for arr, out in ((t, tau), (d, delta)):
                    acc = 0.0
                    for (a, wa) in ((im, 1 - wm), (jm, wm)):
                        for (b, wb) in ((i_n, 1 - wn), (j_n, wn)):
                            for (c, wc) in ((ik, 1 - wk), (jk, wk)):
                                acc += wa * wb * wc * arr[a, b, c]
                    out[m, n, k] = acc
    return tau, delta


def main():
    ap = argparse.ArgumentParser(description="offline profile: VAE chunking, lookup table, B_max")
    ap.add_argument("--workload", default="c3_sd15_mixed32")
    ap.add_argument("--vae", default="vae_sd15")
    ap.add_argument("--images", type=int, default=4, help="VAE images available to a chunk")
    ap.add_argument("--chunk-images", type=int, default=1, help="images per decode in the chunking sweep")
    ap.add_argument("--c-limit", type=int, default=0)
    ap.add_argument("--out", default="")
    args = ap.parse_args()
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import torch

    from fixtures import get_config, make_requests, make_weights
    from fixtures.vae import VAE_CONFIGS, make_vae_latents, make_vae_weights

    from .binding import VAE, UNet

    def log(s):
        print(s, file=sys.stderr, flush=True)

    spec = get_config(args.workload)
    unet = spec["unet"]
    req = make_requests(args.workload)
    R = len(req["timesteps"])
    dev = torch.device("cuda:0")
    m = UNet(unet, max_requests=R, device=dev)
    m.load_weights(make_weights(args.workload))
    act = m.act_dtype
    inputs = dict(latents=torch.from_numpy(req["latents"]).to(dev), timesteps=req["timesteps"],
                  cfg_on=req["cfg_on"], guidance=req["guidance"],
                  ctx_cond=torch.from_numpy(req["ctx_cond"]).to(dev).to(act),
                  ctx_uncond=torch.from_numpy(req["ctx_uncond"]).to(dev).to(act),
                  coef=m.coefficients(req["schedule"], req["timesteps"], req["t_prev"]))
    vspec = VAE_CONFIGS[args.vae]
    v = VAE(vspec["vae"], max_images=args.images, device=dev)
    v.load_weights(make_vae_weights(args.vae))
    z = torch.from_numpy(make_vae_latents(args.vae, args.images)).to(dev)
    log(f"profiling {args.workload} ({R} requests) beside {args.vae} ({len(v.stages)} stages)")

    P = Profiler(m, inputs, v, z[:args.chunk_images])
    chunking = P.choose_chunking(c_limit=args.c_limit or None)
    log(f"chunking: C_max {chunking['C_max']}, chosen c {chunking['chosen_c']}")
    counts = sorted({1, 2, 4, 8, 12, 16, 20, 24, 28, R} & set(range(1, R + 1)))
    bmax, thr = P.saturation_batch(counts)
    log(f"B_max {bmax}")
    P2 = Profiler(m, inputs, v, z)
    m_grid = sorted({1, 8, 16, 24, R} & set(range(1, R + 1)))
    n_grid = sorted({0, 1, 2, args.images})
    grid = P2.lookup_grid(chunking["chosen_c"], m_grid, n_grid)
    log("lookup grid done")
    tau, delta = dense_table(grid, R)
    # one planning instance on the measured table: every request of the batch
    # has a step to run, `images` decodes are pending, half the requests are
    # past the Skip-CFG threshold, and the total latency may exceed one round
    # of the lot by 10 % (T_lim = (1 + alpha) tau(M, N, K), alpha = 0.1)
    M, N, K = R, args.images, R // 2
    T_lim = 1.1 * tau[M, N, K]
    plans = {}
    for exact in (False, True):
        try:
            seq, cost, tm = plan_sequence(M, N, K, tau, delta, T_lim, exact=exact)
            plans["exact" if exact else "alg1"] = dict(sequence=seq, cost_ms=cost, time_ms=tm)
        except Exception as e:  # no sequence under the cap
            plans["exact" if exact else "alg1"] = dict(error=str(e))
    res = dict(workload=args.workload, vae=args.vae, chunk_images=args.chunk_images, chunking=chunking,
               saturation=dict(B_max=bmax, requests_per_s={str(k): v_ for k, v_ in thr.items()}),
               lookup_grid=grid, plan=dict(M=M, N=N, K=K, T_lim_ms=T_lim, **plans))
    txt = json.dumps(res)
    if args.out:
        with open(args.out, "w") as f:
            f.write(txt)
    print(txt, flush=True)
    m.close()
    v.close()


if __name__ == "__main__":
    main()
