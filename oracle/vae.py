"""The VAE decoder of the latent-diffusion models, float64, one image at a time.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper decodes finished latents with the diffusion model's VAE and notes
that its decoder is dominated by serial ResNet blocks (Sec. II-B, Fig. 5);
VAE Chunking splits it into sub-blocks at ResNet-block boundaries (Sec.
III-B).  The paper gives no layer list, so this follows the published
KL-regularised autoencoder decoder that SD uses (Rombach et al. 2022):

  z = latents / scaling;  h = Conv1x1_post(z);  h = Conv3(h)       (conv_in)
  mid:  h = Res(h);  h = h + Attn(GN(h));  h = Res(h)
  up levels from the widest: (n_res + 1) x Res, then nearest-2x + Conv3
        (all levels but the last)
  out:  Conv3(SiLU(GN(h)))
  Res(h): u = Conv3(SiLU(GN1(h))); u = Conv3(SiLU(GN2(u)));
          return u + (Conv1(h) if the width changes else h)
  Attn(x): single head over the H*W tokens, Q/K/V/O linear with biases,
          softmax(Q K^T / sqrt(C)) V.
GroupNorm eps is 1e-6 throughout.  There is no time embedding.

The decoder is also written as a list of stages (the ResNet-block-level
sub-blocks VAE Chunking partitions), so a chunked decode is checked against
the plain one stage by stage.
"""
import numpy as np

from .ops import F, attention, conv2d, group_norm, linear, silu, upsample_nearest2x

GN_EPS = 1e-6


def _res(W, p, h, groups):
    u = conv2d(silu(group_norm(h, groups, W(f"{p}.norm1.g"), W(f"{p}.norm1.b"), GN_EPS)),
               W(f"{p}.conv1.w"), W(f"{p}.conv1.b"))
    u = conv2d(silu(group_norm(u, groups, W(f"{p}.norm2.g"), W(f"{p}.norm2.b"), GN_EPS)),
               W(f"{p}.conv2.w"), W(f"{p}.conv2.b"))
    if u.shape[-1] != h.shape[-1]:
        h = linear(h, W(f"{p}.skip.w"), W(f"{p}.skip.b"))
    return u + h


def _attn(W, h, groups):
    H, Wd, C = h.shape
    x = group_norm(h, groups, W("mid.attn.norm.g"), W("mid.attn.norm.b"), GN_EPS).reshape(H * Wd, C)
    q = linear(x, W("mid.attn.q.w"), W("mid.attn.q.b"))
    k = linear(x, W("mid.attn.k.w"), W("mid.attn.k.b"))
    v = linear(x, W("mid.attn.v.w"), W("mid.attn.v.b"))
    o = attention(q, k, v, 1)  # one head: scale 1 / sqrt(C)
    return h + linear(o, W("mid.attn.o.w"), W("mid.attn.o.b")).reshape(H, Wd, C)


def stages(vae):
    """Names of the decoder's sub-blocks in execution order: the input convs,
    every ResBlock, the attention block, every upsampling conv, the output."""
    s = ["in", "mid.res0", "mid.attn", "mid.res1"]
    nl = len(vae["ch"])
    for i, lvl in enumerate(reversed(range(nl))):
        s += [f"up{i}.res{j}" for j in range(vae["n_res"] + 1)]
        if lvl != 0:
            s.append(f"up{i}.up")
    return s + ["out"]


def run_stage(vae, W, name, h):
    """Apply one stage to h (the latent (C, H, W) for "in", else an H x W x C
    activation); "out" returns the image (out_c, 8H, 8W)."""
    g = vae["gn_groups"]
    if name == "in":
        z = np.asarray(h, F).transpose(1, 2, 0) / vae["scaling"]  # (H, W, C)
        z = linear(z, W("post_quant.w"), W("post_quant.b"))
        return conv2d(z, W("conv_in.w"), W("conv_in.b"))
    if name == "mid.attn":
        return _attn(W, h, g)
    if name.endswith(".up"):
        return conv2d(upsample_nearest2x(h), W(f"{name}.w"), W(f"{name}.b"))
    if name == "out":
        y = conv2d(silu(group_norm(h, g, W("out.norm.g"), W("out.norm.b"), GN_EPS)), W("out.conv.w"),
                   W("out.conv.b"))
        return y.transpose(2, 0, 1)
    return _res(W, name, h, g)


def decode(vae, W, z, begin=0, end=None, h=None):
    """Decode one latent z (C, H, W): stages [begin, end) applied in order,
    starting from z (begin = 0) or from the activation h.  With the default
    range the result is the image (out_c, 8H, 8W) in float64."""
    names = stages(vae)
    end = len(names) if end is None else end
    x = z if begin == 0 else h
    for name in names[begin:end]:
        x = run_stage(vae, W, name, x)
    return x
