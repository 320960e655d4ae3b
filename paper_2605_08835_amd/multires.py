"""Requests of several resolutions in one step (the paper serves 512, 768
and 1024 px requests side by side, Sec. IV-A).

One UNet architecture, one packed copy of its weights, and a handle per
latent size that shares it (synerdiff_unet_create_shared).  A step takes
each size's ragged batch (its own timesteps, Skip-CFG flags, guidance and
contexts) and enqueues the per-size UNet steps back to back on one stream;
every request is still independent of its batch-mates.
"""
from .binding import UNet


class MultiResolutionUNet:
    def __init__(self, unet, sizes, device=None):
        """sizes: {(latent_h, latent_w): max_requests}."""
        if not sizes:
            raise ValueError("at least one latent size")
        self.unet = unet
        self.handles = {}
        first = None
        for (H, W), cap in sizes.items():
            cfg = dict(unet, latent_h=H, latent_w=W)
            h = UNet(cfg, max_requests=cap, device=device, share_weights_with=first)
            first = first or h
            self.handles[(H, W)] = h
        self.first = first
        self.act_dtype = first.act_dtype

    def load_weights(self, weights):
        self.first.load_weights(weights)

    def coefficients(self, schedule, timesteps, t_prev):
        return self.first.coefficients(schedule, timesteps, t_prev)

    def step(self, groups, ctx_uncond, stream=None):
        """groups: {(H, W): dict(latents, timesteps, cfg_on, guidance,
        ctx_cond, coef[, out, eps_out])}; returns {(H, W): out}."""
        res = {}
        for size, g in groups.items():
            if size not in self.handles:
                raise ValueError(f"no handle for latent size {size}")
            res[size] = self.handles[size].step(g["latents"], g["timesteps"], g["cfg_on"], g["guidance"],
                                                g["ctx_cond"], ctx_uncond, g["coef"], out=g.get("out"),
                                                eps_out=g.get("eps_out"), stream=stream)
        return res

    def close(self):
        for h in self.handles.values():
            if h is not self.first:
                h.close()
        self.first.close()
