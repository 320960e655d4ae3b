"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module generates inputs only: UNet configurations (shapes), random-init
weights, latents, text contexts, timesteps, Skip-CFG flags and guidance
scales.  It holds none of the denoising arithmetic; the oracle and the HIP
library each implement that on their own.

Random numbers come from a counter-based SplitMix64 (Steele, Lea & Flood,
"Fast splittable pseudorandom number generators", OOPSLA 2014; the finaliser
constants are Vigna's published ones), turned into 53-bit uniforms and then
into normals with the Box-Muller transform (Box & Muller 1958).  Every tensor
has its own stream keyed by (base seed, workload name, stream id, tensor
name), so values do not depend on generation order or on the NumPy version.
"""
from .rng import Stream, bf16_round  # noqa: F401
from .configs import CONFIGS, get_config, heads_of  # noqa: F401
from .manifest import manifest, param_count  # noqa: F401
from .synth import (make_weights, make_requests, schedule_name, serve_arrivals,  # noqa: F401
                    serve_request_inputs, serve_null_context)
