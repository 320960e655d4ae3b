"""CPU oracle of one step-level continuous-batching UNet denoising step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import or call this package.  The product
path (the HIP library and its Python binding) never touches it, and it shares
no code with that path: the only common dependency is the seeded input
generator in `fixtures`, which holds none of the method's arithmetic.

The oracle writes out the plain per-request definition of the step in
float64, one request at a time, with no row packing:

  1. eps_c = UNet(x, t, c) and, when the request keeps CFG, eps_u = UNet(x, t, c_null)
     (Skip-CFG drops the unconditional evaluation: Sec. II-B, Sec. III-B);
  2. eps = eps_u + w (eps_c - eps_u) when CFG is on, else eps_c
     (classifier-free guidance, Ho & Salimans 2022);
  3. x' = DDIM(eta = 0) update of x with eps (Song et al. 2021).

The UNet is the latent-diffusion UNet (Rombach et al. 2022) that the paper
serves (SD-v1.5, Sec. IV-A); the paper gives none of its internals, so every
layer follows the published architecture; see `oracle.unet`.

Parity status: the per-op functions are pinned by brute force, closed forms
and library routines; the whole-UNet composition is pinned by the exact
public parameter counts, by consumption of every parameter, and by the
invariants of the step (w = 1, Skip-CFG = cond-only, batch independence,
zeroed output conv).  No printed value of the paper covers a UNet output, so
the whole step is "parity unpinned" by the paper itself.
"""
from . import ops, unet, sampler  # noqa: F401
from .sampler import unet_step, unet_step_request, betas, alphas_cumprod, ddim_coefficients  # noqa: F401
