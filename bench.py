"""Benchmark of the step-level continuous-batching UNet step on one MI355X.

Workload: SD-1.5-shaped UNet (latent 4x64x64, channels 320/640/1280/1280),
bf16, a continuous batch of 32 requests at seeded timesteps in [0, 999],
half of them under Skip-CFG (48 packed rows), per-request guidance in [5, 9]
and text contexts, one UNet evaluation + CFG combine + DDIM update per step.
Random-init weights and synthetic inputs (the step's cost is independent of
the values).

Prints ONE JSON line: rows*steps/s (value), the fraction of the bf16 MFMA
peak the whole step reaches, the roofline of the dominant kernel class
(the MFMA implicit-GEMM convolution/linear kernel) measured with HIP events
on the launch stream, and the CPU oracle timed on a bounded sample.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = "c3_sd15_mixed32"


def unet_flops_per_row(u):
    """Algorithmic FLOPs of one UNet row: 2 x MACs of every convolution and
    linear at full size (the upsampling convs as 3x3 convs on the upsampled
    grid, the context K/V per row), the attention products Q K^T and P V,
    and the time MLP with every ResBlock's time projection.  803.27 GFLOP for
    SD-1.5 at 64x64, 6761.24 for the SDXL shape at 128x128."""
    H, W = u["latent_h"], u["latent_w"]
    lc, ch, nl = u["latent_c"], u["ch"], len(u["ch"])
    td, L, D = u["temb_dim"], u["ctx_len"], u["ctx_dim"]
    f = 2.0 * (u["temb_in"] * td + td * td)
    if u["add_in"]:
        f += 2.0 * (u["add_in"] * td + td * td)

    def res(hw, ci, co):
        return 2.0 * hw * co * 9 * (ci + co) + (2.0 * hw * co * ci if ci != co else 0.0) + 2.0 * td * co

    def tx(n, C, depth):
        g = 4.0 * n * C * C  # proj_in, proj_out
        for _ in range(depth):
            g += 8.0 * n * C * C + 4.0 * n * n * C                       # Q/K/V/O, self-attention
            g += 4.0 * n * C * C + 4.0 * L * D * C + 4.0 * n * L * C     # Q/O, context K/V, cross-attention
            g += 24.0 * n * C * C                                        # GEGLU FF (8C up, 4C down)
        return g

    hw = H * W
    f += 2.0 * hw * ch[0] * 9 * lc
    skips, cur = [ch[0]], ch[0]
    for lv in range(nl):
        for _ in range(u["n_res"]):
            f += res(hw, cur, ch[lv])
            cur = ch[lv]
            if u["tx_depth"][lv]:
                f += tx(hw, cur, u["tx_depth"][lv])
            skips.append(cur)
        if lv != nl - 1:
            hw //= 4
            f += 2.0 * hw * cur * 9 * cur
            skips.append(cur)
    f += 2 * res(hw, cur, cur)
    if u["mid_tx_depth"]:
        f += tx(hw, cur, u["mid_tx_depth"])
    for lv in reversed(range(nl)):
        for _ in range(u["n_res"] + 1):
            f += res(hw, cur + skips.pop(), ch[lv])
            cur = ch[lv]
            if u["tx_depth"][lv]:
                f += tx(hw, cur, u["tx_depth"][lv])
        if lv != 0:
            hw *= 4
            f += 2.0 * hw * cur * 9 * cur
    return f + 2.0 * hw * lc * 9 * ch[0]


# Other single-GPU workloads bench.py can time with --workload (the default
# line is the one above): algorithmic FLOPs per UNet row and a description.
WORKLOADS = {
    "c3_sd15_mixed32": (None, "SD-1.5-shaped UNet, latent 4x64x64, bf16; 32 requests at seeded timesteps, "
                                  "16 under Skip-CFG -> 48 packed rows; guidance U[5,9]; 77x768 contexts; "
                                  "UNet + CFG combine + DDIM per step"),
    "c2_sd15_cfg8": (None, "SD-1.5-shaped UNet, latent 4x64x64, bf16; 8 requests, all with CFG -> 16 rows; "
                               "guidance 7.5; 77x768 contexts; UNet + CFG combine + DDIM per step"),
    "c4_sdxl_cfg8": (None, "SDXL-shaped UNet, latent 4x128x128, bf16, channels 320/640/1280, "
                                "transformer depths 0/2/10, 64-wide heads; 8 requests, all with CFG -> 16 rows; "
                                "77x2048 contexts, pooled 1280 + 6 time ids; UNet + CFG combine + DDIM per step"),
    "c6_sd21_v": (None, "SD-2.1-shaped UNet, latent 4x96x96 (768 px), bf16, 64-wide heads, 77x1024 contexts, "
                        "v-prediction; 8 requests, all with CFG -> 16 rows; guidance 7.5; UNet + CFG combine + "
                        "DDIM per step"),
}
METRIC = "UNet rows·steps/sec + % bf16 MFMA peak, SD-1.5-shape, 32-req mixed-CFG batch"
PEAK_BF16 = 2.5166e15  # dense bf16 MFMA, 256 CU x 4096 FLOP/clk x 2.4 GHz
PEAK_HBM = 8.0e12


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_sd15_48rows_traffic.md")
GEMM_SOURCE = os.path.join(ROOT, "paper_2605_08835_amd", "csrc", "gemm.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_class(name):
    """Kernel class of a device kernel name (the classes of the step's profile)."""
    for key, cls in (("gemm_bf16", "gemm"), ("gemm_f32", "gemm"), ("splitk_reduce", "gemm"),
                     ("attn_", "attention"), ("gn_apply", "groupnorm apply"), ("gn_", "groupnorm"),
                     ("layernorm", "layernorm"), ("geglu", "geglu"), ("linear_smallm", "time_mlp"),
                     ("time_inputs", "time_mlp"), ("pack_latents", "pack"), ("out_cfg_ddim", "out_cfg_ddim"),
                     ("cfg_ddim", "cfg_ddim")):
        if key in name:
            return cls
    return None


def non_gemm_flops_per_row(unet):
    """Algorithmic FLOPs per UNet row that are not GEMM-class work: the
    attention cores (Q K^T and P V: 4 N_q N_k C per Transformer block, self-
    and cross-attention) and the output conv (3x3, C0 -> latent channels),
    which the fused output kernel computes.  The rest of the per-row total is
    the convolutions and linears the GEMM kernel runs."""
    H, W = unet["latent_h"], unet["latent_w"]
    L = unet["ctx_len"]
    f = 0.0
    for l, C in enumerate(unet["ch"]):
        n = (H >> l) * (W >> l)
        blocks = (2 * unet["n_res"] + 1) * unet["tx_depth"][l]  # down: n_res, up: n_res + 1
        f += blocks * 4.0 * n * (n + L) * C
    n = (H >> (len(unet["ch"]) - 1)) * (W >> (len(unet["ch"]) - 1))
    f += unet["mid_tx_depth"] * 4.0 * n * (n + L) * unet["ch"][-1]
    out_conv = 2.0 * H * W * 9 * unet["ch"][0] * unet["latent_c"]
    return f, out_conv


def cpu_description():
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return os.cpu_count(), model


def source_digest(path):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def stored_traffic():
    """HBM bytes per GEMM launch from the committed counter summary, if it was
    taken on the GEMM source as it is now (else None)."""
    import re
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    mb = re.search(r"traffic_bytes_per_launch\s*\|\s*([0-9.eE+]+)", text)
    md = re.search(r"gemm\.hip sha256\s*\|\s*([0-9a-f]{64})", text)
    if not mb or not md or md.group(1) != source_digest(GEMM_SOURCE):
        return None
    return float(mb.group(1))


def _per_dispatch(d, counters):
    """{dispatch id: (kernel name, {counter: value})} from a --pmc run's CSV."""
    import csv
    import glob
    f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
    out = {}
    for r in csv.DictReader(open(f)):
        if r["Counter_Name"] in counters:
            name, vals = out.setdefault(r["Dispatch_Id"], (r["Kernel_Name"], {}))
            vals[r["Counter_Name"]] = vals.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return out


def summarize(stats_dir=None, fetch_dir=None, write_dir=None, copy_bytes=None, sq_dir=None):
    """Markdown summary of rocprofv3 output: per-kernel statistics (from a
    --kernel-trace --stats run); from two --pmc runs, the HBM bytes per
    GEMM launch calibrated on the plain copy kernel of copy_bytes each way,
    and with the statistics run as well, every kernel class's bytes per
    launch and bandwidth; from a --pmc run of MfmaUtil, VALUBusy,
    GRBM_GUI_ACTIVE (and LDS counters), each class's MFMA and VALU busy
    fractions weighted by the dispatches' active cycles."""
    import csv
    import glob
    out = []
    class_us = {}
    if stats_dir:
        f = glob.glob(os.path.join(stats_dir, "**", "*kernel_stats.csv"), recursive=True)[0]
        rows = list(csv.DictReader(open(f)))
        out.append("| kernel | class | calls | total ms | avg us |")
        out.append("|---|---|---|---|---|")
        tot = {}
        for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
            cls = kernel_class(r["Name"])
            calls, ns = int(r["Calls"]), float(r["TotalDurationNs"])
            out.append(f"| `{r['Name'][:90]}` | {cls} | {calls} | {ns / 1e6:.3f} | {ns / calls / 1e3:.1f} |")
            if cls:
                t = tot.setdefault(cls, [0, 0.0])
                t[0] += 0 if ("splitk_reduce" in r["Name"] or "gn_finalize" in r["Name"]) else calls
                t[1] += ns
        out.append("")
        out.append("| class | launches | total ms | avg us per launch |")
        out.append("|---|---|---|---|")
        for cls, (calls, ns) in sorted(tot.items(), key=lambda kv: -kv[1][1]):
            out.append(f"| {cls} | {calls} | {ns / 1e6:.3f} | {ns / max(calls, 1) / 1e3:.1f} |")
            class_us[cls] = ns / max(calls, 1) / 1e3
    if fetch_dir and write_dir:
        def per_dispatch(d, counter):
            f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
            vals = {}
            for r in csv.DictReader(open(f)):
                if r["Counter_Name"] == counter:
                    vals[r["Dispatch_Id"]] = (r["Kernel_Name"], vals.get(r["Dispatch_Id"], ("", 0.0))[1]
                                              + float(r["Counter_Value"]))
            return list(vals.values())
        fetch, write = per_dispatch(fetch_dir, "FETCH_SIZE"), per_dispatch(write_dir, "WRITE_SIZE")
        cal_f = max(v for n, v in fetch if "elementwise" in n)
        cal_w = max(v for n, v in write if "elementwise" in n)
        kf, kw = copy_bytes / (cal_f * 1024), copy_bytes / (cal_w * 1024)
        g_f = sum(v for n, v in fetch if kernel_class(n) == "gemm")
        g_w = sum(v for n, v in write if kernel_class(n) == "gemm")
        launches = sum(1 for n, _ in fetch if kernel_class(n) == "gemm" and "splitk_reduce" not in n)
        per = (g_f * 1024 * kf + g_w * 1024 * kw) / launches
        out.append("")
        out.append("| quantity | value |")
        out.append("|---|---|")
        out.append(f"| copy kernel bytes each way | {copy_bytes} |")
        out.append(f"| FETCH_SIZE of the copy (KiB) | {cal_f:.0f} |")
        out.append(f"| WRITE_SIZE of the copy (KiB) | {cal_w:.0f} |")
        out.append(f"| fetch scale | {kf:.4f} |")
        out.append(f"| write scale | {kw:.4f} |")
        out.append(f"| GEMM launches | {launches} |")
        out.append(f"| GEMM fetch bytes (scaled) | {g_f * 1024 * kf:.4e} |")
        out.append(f"| GEMM write bytes (scaled) | {g_w * 1024 * kw:.4e} |")
        out.append(f"| traffic_bytes_per_launch | {per:.4e} |")
        out.append(f"| gemm.hip sha256 | {source_digest(GEMM_SOURCE)} |")
        if class_us:
            # every class: scaled bytes per launch (a split-K reduction and a
            # GroupNorm finalize are charged to their launch, as in the timings)
            byc = {}
            for lst, k in ((fetch, kf), (write, kw)):
                for n, v in lst:
                    cls = kernel_class(n)
                    if cls:
                        b = byc.setdefault(cls, [0.0, 0])
                        b[0] += v * 1024 * k
            for n, _ in fetch:
                cls = kernel_class(n)
                if cls and "splitk_reduce" not in n and "gn_finalize" not in n:
                    byc[cls][1] += 1
            out.append("")
            out.append("| class | launches | HBM bytes per launch (fetch + write) | avg us per launch | GB/s |")
            out.append("|---|---|---|---|---|")
            for cls, (b, nl) in sorted(byc.items(), key=lambda kv: -kv[1][0]):
                if nl and cls in class_us:
                    per_l = b / nl
                    out.append(f"| {cls} | {nl} | {per_l:.4e} | {class_us[cls]:.1f} | "
                               f"{per_l / (class_us[cls] * 1e-6) / 1e9:.0f} |")
    if sq_dir:
        names = ("MfmaUtil", "VALUBusy", "GRBM_GUI_ACTIVE", "SQ_LDS_BANK_CONFLICT", "SQ_INSTS_LDS")
        acc = {}
        for _, (n, v) in _per_dispatch(sq_dir, names).items():
            cls = kernel_class(n)
            if not cls or "GRBM_GUI_ACTIVE" not in v:
                continue
            a = acc.setdefault(cls, [0.0, 0.0, 0.0, 0.0, 0.0, 0])
            g = v["GRBM_GUI_ACTIVE"]
            a[0] += g
            a[1] += v.get("MfmaUtil", 0.0) * g
            a[2] += v.get("VALUBusy", 0.0) * g
            a[3] += v.get("SQ_LDS_BANK_CONFLICT", 0.0)
            a[4] += v.get("SQ_INSTS_LDS", 0.0)
            a[5] += 1
        out.append("")
        out.append("| class | dispatches | MfmaUtil % | VALUBusy % | LDS bank-conflict cycles per LDS instruction |")
        out.append("|---|---|---|---|---|")
        for cls, a in sorted(acc.items(), key=lambda kv: -kv[1][0]):
            out.append(f"| {cls} | {a[5]} | {a[1] / a[0]:.1f} | {a[2] / a[0]:.1f} | {a[3] / max(a[4], 1):.3f} |")
    return "\n".join(out)


def cpu_baseline(unet, weights, req, budget_s=25.0):
    """The oracle, as it is, on a bounded sample: whole requests (one
    Skip-CFG request = 1 row, one CFG request = 2 rows) until ~budget_s."""
    import oracle
    from oracle.unet import Weights
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count()
    W = Weights(weights)
    for name in weights:  # one-off fp64 conversion of the parameters (setup)
        W(name)
    order = list(np.flatnonzero(req["cfg_on"] == 0)) + list(np.flatnonzero(req["cfg_on"] == 1))
    rows, t0 = 0, time.perf_counter()
    done = []
    for r in order:
        oracle.unet_step(unet, W, req, only=[int(r)])
        rows += 1 + int(req["cfg_on"][r])
        done.append(int(r))
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    ncpu, model = cpu_description()
    return {"value": rows / el, "unit": "rows·steps/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{len(done)} requests ({rows} UNet rows) of the same {len(req['cfg_on'])}-request batch, "
                      f"one full float64 step each, {el:.1f} s",
            "host_cpu_count": ncpu, "host_cpu_model": model,
            "cores_note": "cores = BLAS threads the oracle's float64 products ran on"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--layers", default=None, help="write a per-layer device-time table to this file")
    ap.add_argument("--workload", default=WORKLOAD, choices=sorted(WORKLOADS),
                    help="batch to time (the default is the metric's workload)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="run a plain copy kernel of MIB MiB each way first (counter calibration)")
    ap.add_argument("--summarize", nargs="*", metavar="DIR",
                    help="print a markdown summary of rocprofv3 output: STATS_DIR [FETCH_DIR WRITE_DIR [SQ_DIR]] "
                         "(the copy size comes from --calibrate-copy)")
    args = ap.parse_args()
    if args.summarize is not None:
        d = [x or None for x in args.summarize] + [None] * 4
        print(summarize(d[0], d[1], d[2], args.calibrate_copy * 2**20, d[3]))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the step shards by request with no collective, "
              f"and each process drives a single MI355X (got --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch

    from fixtures import get_config, make_requests, make_weights
    from paper_2605_08835_amd import UNet

    wl = args.workload
    _, description = WORKLOADS[wl]
    spec = get_config(wl)
    unet = spec["unet"]
    flop_per_row = unet_flops_per_row(unet)
    t0 = time.time()
    weights = make_weights(wl)
    req = make_requests(wl)
    log(f"inputs ready in {time.time() - t0:.1f} s")
    R = len(req["timesteps"])
    rows = int(R + req["cfg_on"].sum())
    m = UNet(unet, max_requests=R, device="cuda:0")
    m.load_weights(weights)
    dev = torch.device("cuda:0")
    act = m.act_dtype
    lat = torch.from_numpy(req["latents"]).to(dev)
    ctx = torch.from_numpy(req["ctx_cond"]).to(dev).to(act)
    unc = torch.from_numpy(req["ctx_uncond"]).to(dev).to(act)
    coef = m.coefficients(req["schedule"], req["timesteps"], req["t_prev"])
    out = torch.empty_like(lat)
    stream = torch.cuda.current_stream(dev)
    if args.calibrate_copy:
        n = args.calibrate_copy * 2**20 // 4
        src, dst = torch.ones(n, device=dev), torch.empty(n, device=dev)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    extra = {}
    if "pooled_cond" in req:  # SDXL-style added conditioning
        extra = dict(pooled_cond=torch.from_numpy(np.asarray(req["pooled_cond"], np.float32)).to(dev),
                     pooled_uncond=torch.from_numpy(np.asarray(req["pooled_uncond"], np.float32)).to(dev),
                     time_ids=req["time_ids"])

    def step():
        m.step(lat, req["timesteps"], req["cfg_on"], req["guidance"], ctx, unc, coef, out=out, stream=stream,
               **extra)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")
    # one event between consecutive steps: the mean over the whole run is the
    # metric, the per-step spread (median, min, max) comes from the same events
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for i in range(args.steps):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    log(f"timed {args.steps} steps: {ms:.3f} ms/step")

    # Per-kernel-class split: the same steps again with an event after every launch.
    m.profile(True)
    m.profile_read(reset=True)
    m.profile_read_layers(reset=True)
    for _ in range(args.steps):
        step()
        m.profile_read(reset=False)
    prof = m.profile_read(reset=True)
    layers = m.profile_read_layers(reset=True)
    m.profile(False)
    if args.layers:
        with open(args.layers, "w") as f:
            f.write(f"{'layer':44s} {'launches':>8s} {'ms/step':>8s} {'us/launch':>10s} {'TFLOP/s':>8s} {'GB/s':>8s}\n")
            for k, v in sorted(layers.items(), key=lambda kv: -kv[1]["ms"]):
                n = v["launches"]
                f.write(f"{k:44s} {n / args.steps:8.1f} {v['ms'] / args.steps:8.3f} {1e3 * v['ms'] / n:10.1f} "
                        f"{v['flop'] / max(v['ms'], 1e-9) / 1e9:8.1f} {v['bytes'] / max(v['ms'], 1e-9) / 1e6:8.1f}\n")
    kernels = {}
    for k, v in prof.items():
        n = v["launches"]
        kernels[k] = {"launches_per_step": n / args.steps, "ms_per_step": v["ms"] / args.steps,
                      "avg_launch_us": 1e3 * v["ms"] / max(n, 1),
                      "tflops": v["flop"] / max(v["ms"], 1e-9) / 1e9,
                      "gbps": v["bytes"] / max(v["ms"], 1e-9) / 1e6}
    g = prof.get("gemm", {"launches": 1, "ms": 1.0, "flop": 0.0, "bytes": 0.0})
    g_launches = g["launches"] / args.steps
    avg_s = g["ms"] / max(g["launches"], 1) / 1e3
    # Algorithmic FLOPs of the GEMM class: every conv and linear of the
    # model at its full size (each upsampling conv as a 3x3 on the upsampled
    # grid, every row's CFG prefix), i.e. the per-row total less the
    # attention cores and the output conv, times the rows, per launch.
    attn_row, out_row = non_gemm_flops_per_row(unet)
    gemm_row = flop_per_row - attn_row - out_row
    flop_per_launch = rows * gemm_row / max(g_launches, 1e-9)
    achieved = flop_per_launch / avg_s / 1e12
    exec_per_launch = g["flop"] / max(g["launches"], 1)
    roof = {"kernel": "gemm_bf16_dma_kernel (implicit-GEMM conv / linear, MFMA 32x32x16 bf16)",
            "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16 / 1e12, "unit": "TFLOP/s",
            "frac": round(achieved * 1e12 / PEAK_BF16, 4), "traffic": stored_traffic() if wl == WORKLOAD else None,
            "flop_per_launch": flop_per_launch, "gemm_flop_per_row": gemm_row, "launches_per_step": g_launches,
            "avg_launch_us": round(avg_s * 1e6, 2),
            "executed_flop_per_launch": exec_per_launch,
            "executed_frac": round(exec_per_launch / avg_s / PEAK_BF16, 4)}

    value = rows * 1e3 / ms
    res = {
        "metric": METRIC, "value": round(value, 2), "unit": "rows·steps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 3),
        "step_ms": {"mean": round(ms, 3), "median": round(float(np.median(per_step)), 3),
                    "min": round(float(per_step.min()), 3), "max": round(float(per_step.max()), 3)},
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) latents and contexts, random-init N(0,0.02) weights)",
        "config": {"workload": description, "name": wl, "requests": R, "rows": rows,
                   "latent": [unet["latent_c"], unet["latent_h"], unet["latent_w"]]},
        "requests_steps_per_s": round(R * 1e3 / ms, 2),
        "pct_bf16_peak": round(100 * value * flop_per_row / PEAK_BF16, 2),
        "roofline": roof,
        "kernels": kernels,
    }
    if wl != WORKLOAD:
        res["metric"] = METRIC.replace("SD-1.5-shape, 32-req mixed-CFG batch", wl)
    if not args.no_cpu_baseline and wl == WORKLOAD:
        log("timing the CPU oracle on a bounded sample ...")
        res["cpu_baseline"] = cpu_baseline(unet, weights, req)
    m.close()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
