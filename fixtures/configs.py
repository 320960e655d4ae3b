"""UNet shapes and request-batch recipes of the five workloads.

A configuration is a plain dict.  Keys:
  latent_c, latent_h, latent_w : latent tensor per request (C, H, W)
  ch        : channel width per resolution level
  n_res     : ResBlocks per down level (up levels use n_res + 1)
  tx_depth  : transformer blocks per Transformer2D at each level (0 = none)
  mid_tx_depth : transformer blocks in the mid Transformer2D
  heads / head_dim : exactly one is non-zero; the other follows from C
  gn_groups : GroupNorm group count
  ctx_len, ctx_dim : text-context tokens and width
  temb_in, temb_dim : sinusoid width and time-embedding width
  add_in    : width of the added (pooled + time-id) embedding input, 0 = none
  pooled_dim, time_id_dim, n_time_ids : pieces of add_in (SDXL-like only)
  dtype     : "f32" or "bf16" (the HIP path's compute/storage type)
  schedule  : beta schedule name, "linear" or "scaled_linear"
  n_steps   : DDIM steps per request (step size 1000 // n_steps)
"""
import copy

SD15 = dict(
    latent_c=4, latent_h=64, latent_w=64, ch=(320, 640, 1280, 1280), n_res=2,
    tx_depth=(1, 1, 1, 0), mid_tx_depth=1, heads=8, head_dim=0, gn_groups=32,
    ctx_len=77, ctx_dim=768, temb_in=320, temb_dim=1280, add_in=0,
    pooled_dim=0, time_id_dim=0, n_time_ids=0, dtype="bf16",
    schedule="scaled_linear", n_steps=50,
)

SDXL = dict(
    latent_c=4, latent_h=128, latent_w=128, ch=(320, 640, 1280), n_res=2,
    tx_depth=(0, 2, 10), mid_tx_depth=10, heads=0, head_dim=64, gn_groups=32,
    ctx_len=77, ctx_dim=2048, temb_in=320, temb_dim=1280, add_in=2816,
    pooled_dim=1280, time_id_dim=256, n_time_ids=6, dtype="bf16",
    schedule="scaled_linear", n_steps=50,
)

# SD-2.1 (768 px): the SD-1.5 layout with 64-wide heads (5/10/20/20 heads),
# linear proj_in/proj_out (the per-pixel linear both shapes use here), a
# 1024-wide text context and v-prediction; 96x96 latents.
SD21 = dict(SD15, latent_h=96, latent_w=96, heads=0, head_dim=64, ctx_dim=1024, prediction="v")

TINY = dict(
    latent_c=4, latent_h=16, latent_w=16, ch=(32, 64), n_res=1,
    tx_depth=(1, 1), mid_tx_depth=1, heads=4, head_dim=0, gn_groups=8,
    ctx_len=8, ctx_dim=32, temb_in=32, temb_dim=128, add_in=0,
    pooled_dim=0, time_id_dim=0, n_time_ids=0, dtype="f32",
    schedule="linear", n_steps=50,
)


def _with(base, **kw):
    c = copy.deepcopy(base)
    c.update(kw)
    return c


# Batch recipes.  "requests" is the request count; "cfg" how Skip-CFG flags
# are drawn; "guidance" how scales are drawn; "t" how timesteps are drawn.
CONFIGS = {
    # Tiny fp32 UNet: two requests at t = 999 and 500, request 0 CFG (w=7.5),
    # request 1 skips CFG; one DDIM step, linear betas.
    "c1_tiny_f32": dict(unet=TINY, requests=2, t=("fixed", (999, 500)),
                        cfg=("fixed", (1, 0)), guidance=("fixed", (7.5, 7.5))),
    # SD-1.5 shape, 8 requests all with CFG (16 rows), w = 7.5.
    "c2_sd15_cfg8": dict(unet=SD15, requests=8, t=("uniform",),
                         cfg=("all",), guidance=("fixed_all", 7.5)),
    # SD-1.5 shape, 32 requests, a seeded half skip CFG (48 rows), w ~ U[5, 9].
    "c3_sd15_mixed32": dict(unet=SD15, requests=32, t=("uniform",),
                            cfg=("half",), guidance=("uniform", 5.0, 9.0)),
    # SDXL-like, 8 requests with CFG (16 rows).
    "c4_sdxl_cfg8": dict(unet=SDXL, requests=8, t=("uniform",),
                         cfg=("all",), guidance=("fixed_all", 7.5)),
    # Serving loop: Poisson(4) arrivals per iteration, 20..50 steps, cap 32,
    # Skip-CFG from 60% of a request's steps on.
    "c5_sd15_serve": dict(unet=SD15, requests=32, iterations=1000,
                          arrival_rate=4.0, steps_range=(20, 50),
                          skip_after=0.6, guidance=("uniform", 5.0, 9.0)),
    # A small serving loop for tests: a narrow bf16 UNet on 16x16 latents
    # (the 16x16 VAE test decoder's input), 2-4 steps per request, cap 4.
    "t_serve_tiny": dict(unet=_with(TINY, dtype="bf16", ch=(64, 128), heads=2, gn_groups=32, ctx_len=11,
                                    ctx_dim=64, schedule="scaled_linear"),
                         requests=4, iterations=30, arrival_rate=1.5, steps_range=(2, 4), skip_after=0.6,
                         guidance=("uniform", 5.0, 9.0)),
    # Smaller parity workloads with the same kernels' shapes and tails.
    "t_tiny_bf16": dict(unet=_with(TINY, dtype="bf16", ch=(64, 128), heads=2,
                                   gn_groups=32, ctx_len=11, ctx_dim=64,
                                   latent_h=12, latent_w=12, schedule="scaled_linear"),
                        requests=3, t=("uniform",), cfg=("fixed", (1, 0, 1)),
                        guidance=("uniform", 5.0, 9.0)),
    "t_sd15_16": dict(unet=_with(SD15, latent_h=16, latent_w=16),
                      requests=3, t=("uniform",), cfg=("fixed", (1, 0, 1)),
                      guidance=("uniform", 5.0, 9.0)),
    "t_sdxl_16": dict(unet=_with(SDXL, latent_h=16, latent_w=16, tx_depth=(0, 1, 2),
                                 mid_tx_depth=2),
                      requests=2, t=("uniform",), cfg=("fixed", (1, 0)),
                      guidance=("uniform", 5.0, 9.0)),
    # SD-2.1 shape (v-prediction, 64-wide heads, 1024-wide context): 8 requests
    # with CFG at 768 px, and the same layers at 16x16 for parity.
    "c6_sd21_v": dict(unet=SD21, requests=8, t=("uniform",), cfg=("all",), guidance=("fixed_all", 7.5)),
    "t_sd21_16": dict(unet=_with(SD21, latent_h=16, latent_w=16), requests=3, t=("uniform",),
                      cfg=("fixed", (1, 0, 1)), guidance=("uniform", 5.0, 9.0)),
    "t_tiny_f32_v": dict(unet=_with(TINY, prediction="v", schedule="scaled_linear"), requests=2,
                         t=("uniform",), cfg=("fixed", (1, 0)), guidance=("uniform", 5.0, 9.0)),
    "t_tiny_f32_ragged": dict(unet=_with(TINY, latent_h=12, latent_w=20),
                              requests=3, t=("uniform",), cfg=("fixed", (0, 1, 1)),
                              guidance=("uniform", 5.0, 9.0)),
}


def get_config(name):
    return CONFIGS[name]


def heads_of(unet, c):
    """Attention heads and head width at channel width c."""
    if unet["heads"]:
        return unet["heads"], c // unet["heads"]
    return c // unet["head_dim"], unet["head_dim"]
