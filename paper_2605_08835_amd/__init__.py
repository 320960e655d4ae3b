"""MI355X (gfx950) step-level continuous-batching UNet denoising step.

The compute path is the HIP library libsynerdiff.so (hand-written gfx950
kernels behind the C ABI declared in include/synerdiff.h); `binding` is a
thin ctypes layer over it that uses PyTorch only for device memory and
streams.  Importing the package does not load the library; the first call
that needs it does, and raises if it is missing.
"""
from .binding import (UNet, UNetConfig, alphas_cumprod, config_from_dict, ddim_coef,  # noqa: F401
                      lib, manifest, row_plan, SynerDiffError, VAE, VAEConfig, vae_config_from_dict, vae_manifest,
                      vae_chunk_plan, chunk_cost, plan_sequence)
from .multires import MultiResolutionUNet  # noqa: F401,E402
