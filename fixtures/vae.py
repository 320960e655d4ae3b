"""VAE-decoder shapes, parameter names and seeded inputs.

The decoder is the one of the KL-regularised autoencoder the latent-diffusion
models use (Rombach et al. 2022): a 1x1 post-quantisation conv, conv_in, a
mid block (ResBlock, single-head spatial self-attention, ResBlock), up
levels of (n_res + 1) ResBlocks with nearest-2x + 3x3 conv upsampling
between them, and GroupNorm + SiLU + conv_out.  This module holds names,
shapes and seeded values only; the oracle and the HIP library each build the
decoder on their own.  Shapes use the (out, in[, kh, kw]) order; kinds as in
fixtures.manifest.
"""
import numpy as np

from .rng import Stream, bf16_round, normal_many

# SD-1.5's decoder: 4 latent channels, block widths (128, 256, 512, 512)
# listed from the output end, two ResBlocks per encoder level (three per
# decoder level), 32 GroupNorm groups, RGB output; latents are divided by
# the scaling factor 0.18215 before decoding.
VAE_SD = dict(latent_c=4, latent_h=64, latent_w=64, ch=(128, 256, 512, 512), n_res=2, gn_groups=32,
              out_c=3, scaling=0.18215, dtype="bf16")

VAE_CONFIGS = {
    # SD-1.5 decoder at 512 px (64x64 latents)
    "vae_sd15": dict(vae=VAE_SD, images=1),
    # the same layers on small latents (parity at oracle-friendly sizes)
    "vae_t16": dict(vae=dict(VAE_SD, latent_h=16, latent_w=16), images=2),
    "vae_t12x8": dict(vae=dict(VAE_SD, latent_h=12, latent_w=8), images=2),
    # narrow widths and fp32 storage
    "vae_tiny_f32": dict(vae=dict(VAE_SD, latent_h=8, latent_w=8, ch=(32, 64), gn_groups=8, dtype="f32"),
                         images=2),
}


def _res(P, name, cin, cout):
    P += [(f"{name}.norm1.g", (cin,), "g"), (f"{name}.norm1.b", (cin,), "beta"),
          (f"{name}.conv1.w", (cout, cin, 3, 3), "w"), (f"{name}.conv1.b", (cout,), "b"),
          (f"{name}.norm2.g", (cout,), "g"), (f"{name}.norm2.b", (cout,), "beta"),
          (f"{name}.conv2.w", (cout, cout, 3, 3), "w"), (f"{name}.conv2.b", (cout,), "b")]
    if cin != cout:
        P += [(f"{name}.skip.w", (cout, cin), "w"), (f"{name}.skip.b", (cout,), "b")]


def vae_manifest(vae):
    """Ordered (name, shape, kind) of every decoder parameter."""
    P = []
    lc, ch, nl = vae["latent_c"], vae["ch"], len(vae["ch"])
    P += [("post_quant.w", (lc, lc), "w"), ("post_quant.b", (lc,), "b")]
    top = ch[-1]
    P += [("conv_in.w", (top, lc, 3, 3), "w"), ("conv_in.b", (top,), "b")]
    _res(P, "mid.res0", top, top)
    P += [("mid.attn.norm.g", (top,), "g"), ("mid.attn.norm.b", (top,), "beta")]
    for p in ("q", "k", "v", "o"):
        P += [(f"mid.attn.{p}.w", (top, top), "w"), (f"mid.attn.{p}.b", (top,), "b")]
    _res(P, "mid.res1", top, top)
    cur = top
    for i, lvl in enumerate(reversed(range(nl))):
        for j in range(vae["n_res"] + 1):
            _res(P, f"up{i}.res{j}", cur, ch[lvl])
            cur = ch[lvl]
        if lvl != 0:
            P += [(f"up{i}.up.w", (cur, cur, 3, 3), "w"), (f"up{i}.up.b", (cur,), "b")]
    P += [("out.norm.g", (ch[0],), "g"), ("out.norm.b", (ch[0],), "beta"),
          ("out.conv.w", (vae["out_c"], ch[0], 3, 3), "w"), ("out.conv.b", (vae["out_c"],), "b")]
    return P


def vae_param_count(vae):
    return int(sum(int(np.prod(s)) for _, s, _ in vae_manifest(vae)))


def make_vae_weights(name):
    """Random-init decoder weights (N(0, 0.02) weights and biases, norm scales
    1 + N(0, 0.02), shifts N(0, 0.02)); bf16 configs round to bfloat16."""
    vae = VAE_CONFIGS[name]["vae"]
    bf = vae["dtype"] == "bf16"

    def post_w(v):
        v = (v * 0.02).astype(np.float32)
        return bf16_round(v) if bf else v

    def post_g(v):
        v = (v * 0.02).astype(np.float32) + np.float32(1.0)
        return bf16_round(v) if bf else v

    man = vae_manifest(vae)
    vals = normal_many([(Stream(name, 0, n), int(np.prod(s)), post_g if k == "g" else post_w) for n, s, k in man])
    return {n: v.reshape(s) for (n, s, _), v in zip(man, vals)}


def make_vae_latents(name, images=None):
    """Seeded N(0, 1) * 0.18215-scale latents [images, C, H, W] fp32, the
    magnitude of final SD latents (unit variance after the 1 / scaling
    division)."""
    spec = VAE_CONFIGS[name]
    vae = spec["vae"]
    n = spec["images"] if images is None else images
    shape = (n, vae["latent_c"], vae["latent_h"], vae["latent_w"])
    (v,) = normal_many([(Stream(name, 1, "latents"), int(np.prod(shape)), None)])
    return (v.reshape(shape) * np.float32(vae["scaling"])).astype(np.float32)
