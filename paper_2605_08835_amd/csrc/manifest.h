// UNet parameter manifest (names, shapes, order) and config validation.
// Host-only C++; no HIP calls.
#pragma once
#include <stdint.h>

#include <string>
#include <vector>

#include "synerdiff.h"

namespace sd {

struct Param {
  std::string name;
  std::vector<int64_t> shape;
  size_t offset;  // in floats, within the concatenated fp32 parameter array
  size_t numel;
};

// Parameters in load order.  Shapes are (out, in[, kh, kw]); the walk is the
// latent-diffusion UNet topology: time MLP, optional added-embedding MLP,
// conv_in, down levels (ResBlocks, Transformer2D, strided conv), mid block,
// up levels over the skip stack (ResBlocks on the concat, Transformer2D,
// nearest-2x + conv), output GroupNorm + conv.
std::vector<Param> build_manifest(const sd_unet_config& c);

// Empty string if supported, else the reason.
std::string check_config(const sd_unet_config& c);

inline int heads_at(const sd_unet_config& c, int ch) { return c.heads ? c.heads : ch / c.head_dim; }

}  // namespace sd
