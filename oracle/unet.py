"""The latent-diffusion UNet noise predictor eps_theta(x, t, c), float64.

The paper serves SD-v1.5 (Sec. IV-A) and describes none of the UNet's
internals, so the layers follow the published latent-diffusion UNet
(Rombach et al. 2022) as configured for SD-1.5 and SDXL:

  time:   tau = W2 SiLU(W1 e + b1) + b2 with e the sinusoidal embedding of t;
          SDXL-like configs add W4 SiLU(W3 a + b3) + b4, where a is the pooled
          text embedding followed by the sinusoidal embeddings of six time ids.
  ResBlock(h): u = Conv3(SiLU(GN(h))) + Wt SiLU(tau) + bt (per channel)
               u = Conv3(SiLU(GN(u)))
               return u + (Conv1(h) if the width changes else h)
  Transformer2D(h, c): z = Lin_in(GN_eps=1e-6(h)) per pixel, then per block
               z += SelfAttn(LN1 z); z += CrossAttn(LN2 z, c);
               z += W2 (a * GELU(g)) + b2 with [a | g] = W1 LN3 z + b1;
               return Lin_out(z) + h
  Attn(x, kv): heads of Q = x Wq, K = kv Wk, V = kv Wv (no bias), output
               projection with bias.
  Topology: conv_in; down levels of n_res x (ResBlock, Transformer2D if the
            level has one), each output pushed on a skip stack (conv_in's
            output first), strided 3x3 conv between levels (also pushed);
            mid ResBlock, Transformer2D, ResBlock; up levels of (n_res + 1) x
            (ResBlock on [h | popped skip], Transformer2D), nearest-2x + 3x3
            conv between levels; out = Conv3(SiLU(GN(h))).
GroupNorm eps is 1e-5 except inside Transformer2D (1e-6); LayerNorm eps 1e-5.
"""
import numpy as np

from .ops import (F, attention, conv2d, gelu, group_norm, layer_norm, linear,
                  silu, timestep_embedding, upsample_nearest2x)


class Weights:
    """Read-only view of a {name: array} weight dict that records which
    parameters were read (the composition tests check that every parameter
    is consumed)."""

    def __init__(self, d):
        self.d = d
        self.used = set()
        self._f64 = {}

    def __call__(self, name):
        self.used.add(name)
        if name not in self._f64:
            self._f64[name] = np.asarray(self.d[name], F)
        return self._f64[name]


def heads_at(cfg, c):
    if cfg["heads"]:
        return cfg["heads"]
    return c // cfg["head_dim"]


def time_embedding(cfg, W, t, pooled=None, time_ids=None):
    e = timestep_embedding(t, cfg["temb_in"])
    tau = linear(silu(linear(e, W("time.lin1.w"), W("time.lin1.b"))),
                 W("time.lin2.w"), W("time.lin2.b"))
    if cfg["add_in"]:
        ids = np.concatenate([timestep_embedding(v, cfg["time_id_dim"]) for v in time_ids])
        a = np.concatenate([np.asarray(pooled, F), ids])
        tau = tau + linear(silu(linear(a, W("add.lin1.w"), W("add.lin1.b"))),
                           W("add.lin2.w"), W("add.lin2.b"))
    return tau


def resblock(cfg, W, p, h, tau):
    G = cfg["gn_groups"]
    u = conv2d(silu(group_norm(h, G, W(f"{p}.norm1.g"), W(f"{p}.norm1.b"), 1e-5)),
               W(f"{p}.conv1.w"), W(f"{p}.conv1.b"))
    u = u + linear(silu(tau), W(f"{p}.temb.w"), W(f"{p}.temb.b"))
    u = conv2d(silu(group_norm(u, G, W(f"{p}.norm2.g"), W(f"{p}.norm2.b"), 1e-5)),
               W(f"{p}.conv2.w"), W(f"{p}.conv2.b"))
    if f"{p}.skip.w" in W.d:
        return u + linear(h, W(f"{p}.skip.w"), W(f"{p}.skip.b"))
    return u + h


def transformer(cfg, W, p, h, ctx, depth):
    H, Wd, C = h.shape
    heads = heads_at(cfg, C)
    z = group_norm(h, cfg["gn_groups"], W(f"{p}.norm.g"), W(f"{p}.norm.b"), 1e-6)
    z = linear(z.reshape(H * Wd, C), W(f"{p}.proj_in.w"), W(f"{p}.proj_in.b"))
    for j in range(depth):
        b = f"{p}.blk{j}"
        x = layer_norm(z, W(f"{b}.ln1.g"), W(f"{b}.ln1.b"))
        a = attention(linear(x, W(f"{b}.attn1.q.w")), linear(x, W(f"{b}.attn1.k.w")),
                      linear(x, W(f"{b}.attn1.v.w")), heads)
        z = z + linear(a, W(f"{b}.attn1.o.w"), W(f"{b}.attn1.o.b"))
        x = layer_norm(z, W(f"{b}.ln2.g"), W(f"{b}.ln2.b"))
        a = attention(linear(x, W(f"{b}.attn2.q.w")), linear(ctx, W(f"{b}.attn2.k.w")),
                      linear(ctx, W(f"{b}.attn2.v.w")), heads)
        z = z + linear(a, W(f"{b}.attn2.o.w"), W(f"{b}.attn2.o.b"))
        x = layer_norm(z, W(f"{b}.ln3.g"), W(f"{b}.ln3.b"))
        ag = linear(x, W(f"{b}.ff.w1"), W(f"{b}.ff.b1"))
        n = ag.shape[1] // 2
        z = z + linear(ag[:, :n] * gelu(ag[:, n:]), W(f"{b}.ff.w2"), W(f"{b}.ff.b2"))
    z = linear(z, W(f"{p}.proj_out.w"), W(f"{p}.proj_out.b"))
    return z.reshape(H, Wd, C) + h


def unet_eps(cfg, W, x, t, ctx, pooled=None, time_ids=None):
    """eps_theta for one latent x of shape (C, H, W); returns (C, H, W)."""
    if not isinstance(W, Weights):
        W = Weights(W)
    ctx = np.asarray(ctx, F)
    tau = time_embedding(cfg, W, t, pooled, time_ids)
    ch, nl = cfg["ch"], len(cfg["ch"])
    h = conv2d(np.asarray(x, F).transpose(1, 2, 0), W("conv_in.w"), W("conv_in.b"))
    skips = [h]
    for lvl in range(nl):
        for i in range(cfg["n_res"]):
            h = resblock(cfg, W, f"down{lvl}.res{i}", h, tau)
            if cfg["tx_depth"][lvl]:
                h = transformer(cfg, W, f"down{lvl}.tx{i}", h, ctx, cfg["tx_depth"][lvl])
            skips.append(h)
        if lvl != nl - 1:
            h = conv2d(h, W(f"down{lvl}.down.w"), W(f"down{lvl}.down.b"), stride=2)
            skips.append(h)
    h = resblock(cfg, W, "mid.res0", h, tau)
    if cfg["mid_tx_depth"]:
        h = transformer(cfg, W, "mid.tx", h, ctx, cfg["mid_tx_depth"])
    h = resblock(cfg, W, "mid.res1", h, tau)
    for lvl in reversed(range(nl)):
        for i in range(cfg["n_res"] + 1):
            h = np.concatenate([h, skips.pop()], axis=2)
            h = resblock(cfg, W, f"up{lvl}.res{i}", h, tau)
            if cfg["tx_depth"][lvl]:
                h = transformer(cfg, W, f"up{lvl}.tx{i}", h, ctx, cfg["tx_depth"][lvl])
        if lvl != 0:
            h = conv2d(upsample_nearest2x(h), W(f"up{lvl}.up.w"), W(f"up{lvl}.up.b"))
    h = silu(group_norm(h, cfg["gn_groups"], W("out.norm.g"), W("out.norm.b"), 1e-5))
    out = conv2d(h, W("out.conv.w"), W("out.conv.b"))
    return out.transpose(2, 0, 1)
