"""Parameter names and shapes of a UNet configuration.

Names follow the module structure of the latent-diffusion UNet: a timestep
MLP (and, for SDXL-like configs, an added-embedding MLP), conv_in, down
levels of ResBlocks and Transformer2D blocks with strided-conv downsampling,
a mid block, up levels consuming the skip stack with nearest-2x upsampling,
and the output GroupNorm + conv.  Shapes use the (out, in[, kh, kw]) order.
Each entry is (name, shape, kind) where kind selects the init recipe:
  "w"  weight ~ N(0, 0.02)   "b" bias ~ N(0, 0.02)
  "g"  norm scale ~ 1 + N(0, 0.02)   "beta" norm shift ~ N(0, 0.02)
"""


def _resblock(P, name, cin, cout, tdim):
    P += [(f"{name}.norm1.g", (cin,), "g"), (f"{name}.norm1.b", (cin,), "beta"),
          (f"{name}.conv1.w", (cout, cin, 3, 3), "w"), (f"{name}.conv1.b", (cout,), "b"),
          (f"{name}.temb.w", (cout, tdim), "w"), (f"{name}.temb.b", (cout,), "b"),
          (f"{name}.norm2.g", (cout,), "g"), (f"{name}.norm2.b", (cout,), "beta"),
          (f"{name}.conv2.w", (cout, cout, 3, 3), "w"), (f"{name}.conv2.b", (cout,), "b")]
    if cin != cout:
        P += [(f"{name}.skip.w", (cout, cin), "w"), (f"{name}.skip.b", (cout,), "b")]


def _transformer(P, name, c, depth, ctx_dim):
    P += [(f"{name}.norm.g", (c,), "g"), (f"{name}.norm.b", (c,), "beta"),
          (f"{name}.proj_in.w", (c, c), "w"), (f"{name}.proj_in.b", (c,), "b")]
    for j in range(depth):
        p = f"{name}.blk{j}"
        P += [(f"{p}.ln1.g", (c,), "g"), (f"{p}.ln1.b", (c,), "beta"),
              (f"{p}.attn1.q.w", (c, c), "w"), (f"{p}.attn1.k.w", (c, c), "w"),
              (f"{p}.attn1.v.w", (c, c), "w"),
              (f"{p}.attn1.o.w", (c, c), "w"), (f"{p}.attn1.o.b", (c,), "b"),
              (f"{p}.ln2.g", (c,), "g"), (f"{p}.ln2.b", (c,), "beta"),
              (f"{p}.attn2.q.w", (c, c), "w"), (f"{p}.attn2.k.w", (c, ctx_dim), "w"),
              (f"{p}.attn2.v.w", (c, ctx_dim), "w"),
              (f"{p}.attn2.o.w", (c, c), "w"), (f"{p}.attn2.o.b", (c,), "b"),
              (f"{p}.ln3.g", (c,), "g"), (f"{p}.ln3.b", (c,), "beta"),
              (f"{p}.ff.w1", (8 * c, c), "w"), (f"{p}.ff.b1", (8 * c,), "b"),
              (f"{p}.ff.w2", (c, 4 * c), "w"), (f"{p}.ff.b2", (c,), "b")]
    P += [(f"{name}.proj_out.w", (c, c), "w"), (f"{name}.proj_out.b", (c,), "b")]


def manifest(unet):
    """Ordered list of (name, shape, kind) for every UNet parameter."""
    P = []
    ti, td = unet["temb_in"], unet["temb_dim"]
    P += [("time.lin1.w", (td, ti), "w"), ("time.lin1.b", (td,), "b"),
          ("time.lin2.w", (td, td), "w"), ("time.lin2.b", (td,), "b")]
    if unet["add_in"]:
        P += [("add.lin1.w", (td, unet["add_in"]), "w"), ("add.lin1.b", (td,), "b"),
              ("add.lin2.w", (td, td), "w"), ("add.lin2.b", (td,), "b")]
    ch, nl = unet["ch"], len(unet["ch"])
    lc = unet["latent_c"]
    P += [("conv_in.w", (ch[0], lc, 3, 3), "w"), ("conv_in.b", (ch[0],), "b")]
    skips = [ch[0]]
    cur = ch[0]
    for lvl in range(nl):
        for i in range(unet["n_res"]):
            _resblock(P, f"down{lvl}.res{i}", cur, ch[lvl], td)
            cur = ch[lvl]
            if unet["tx_depth"][lvl]:
                _transformer(P, f"down{lvl}.tx{i}", cur, unet["tx_depth"][lvl], unet["ctx_dim"])
            skips.append(cur)
        if lvl != nl - 1:
            P += [(f"down{lvl}.down.w", (cur, cur, 3, 3), "w"), (f"down{lvl}.down.b", (cur,), "b")]
            skips.append(cur)
    _resblock(P, "mid.res0", cur, cur, td)
    if unet["mid_tx_depth"]:
        _transformer(P, "mid.tx", cur, unet["mid_tx_depth"], unet["ctx_dim"])
    _resblock(P, "mid.res1", cur, cur, td)
    for lvl in reversed(range(nl)):
        for i in range(unet["n_res"] + 1):
            s = skips.pop()
            _resblock(P, f"up{lvl}.res{i}", cur + s, ch[lvl], td)
            cur = ch[lvl]
            if unet["tx_depth"][lvl]:
                _transformer(P, f"up{lvl}.tx{i}", cur, unet["tx_depth"][lvl], unet["ctx_dim"])
        if lvl != 0:
            P += [(f"up{lvl}.up.w", (cur, cur, 3, 3), "w"), (f"up{lvl}.up.b", (cur,), "b")]
    P += [("out.norm.g", (ch[0],), "g"), ("out.norm.b", (ch[0],), "beta"),
          ("out.conv.w", (lc, ch[0], 3, 3), "w"), ("out.conv.b", (lc,), "b")]
    return P


def param_count(unet):
    n = 0
    for _, shape, _ in manifest(unet):
        k = 1
        for s in shape:
            k *= s
        n += k
    return n
