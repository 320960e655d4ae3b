/*
 * synerdiff_vae.h - C ABI of the VAE decoder and of VAE Chunking.
 *
 * The serving pipeline decodes every finished latent with the diffusion
 * model's VAE decoder (Sec. I, Sec. II-B).  The decoder is dominated by
 * serial ResNet blocks (Fig. 5); VAE Chunking splits it into sub-blocks at
 * ResNet-block boundaries that run interleaved with UNet steps, one chunk
 * per concurrent round (Sec. III-B).  This header exposes the decoder as a
 * list of such sub-blocks ("stages"): a call runs a contiguous range of
 * them, so a caller can decode in one call or in c chunks on a second
 * stream beside synerdiff_unet_step.  The layers follow the published
 * KL-autoencoder decoder the latent-diffusion models use (Rombach et al.
 * 2022): 1x1 post-quantisation conv of latents / scaling, conv_in, mid
 * block (ResBlock, single-head spatial attention, ResBlock), up levels of
 * n_res + 1 ResBlocks with nearest-2x + 3x3 conv upsampling, GroupNorm +
 * SiLU + conv_out.  GroupNorm eps 1e-6.
 *
 * Conventions as in synerdiff.h: caller-owned device buffers (the library
 * allocates no device memory), the caller's stream, validation before
 * enqueue, SD_ERR_HIP on a launch failure, one host thread per handle.
 */
#ifndef SYNERDIFF_VAE_H
#define SYNERDIFF_VAE_H

#include "synerdiff.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Decoder shape.  ch[] lists the block widths from the output end (SD:
 * 128, 256, 512, 512); the mid block and conv_in run at ch[n_levels - 1].
 * Supported: latent_c <= 8; ch[] multiples of 32 and of gn_groups, <= 1024;
 * n_levels 1..4; out_c 1..4; the mid-block attention's token count
 * latent_h * latent_w <= 8192. */
typedef struct {
  int32_t latent_c, latent_h, latent_w;
  int32_t n_levels;
  int32_t ch[4];
  int32_t n_res;      /* ResBlocks per encoder level; the decoder runs n_res + 1 per level */
  int32_t gn_groups;
  int32_t out_c;      /* image channels */
  int32_t max_images; /* images per call */
  int32_t dtype;      /* sd_dtype */
  float scaling;      /* latents are divided by this before decoding */
} sd_vae_config;

typedef struct sd_vae sd_vae; /* opaque, host-side handle */

sd_status synerdiff_vae_config_check(const sd_vae_config* cfg);
/* Parameter manifest (names and shapes in load order), as for the UNet. */
int64_t synerdiff_vae_param_count(const sd_vae_config* cfg);
sd_status synerdiff_vae_param_info(const sd_vae_config* cfg, int64_t i, char* name, size_t name_cap, int64_t shape[4],
                                   int32_t* ndim);
/* Device bytes for the packed weights and for the workspace (sized for
 * max_images); 0 on a bad config.  The workspace also carries a chunked
 * decode's state from one call to the next. */
size_t synerdiff_vae_weights_bytes(const sd_vae_config* cfg);
size_t synerdiff_vae_workspace_bytes(const sd_vae_config* cfg);
sd_status synerdiff_vae_create(const sd_vae_config* cfg, void* d_weights, size_t weights_bytes, void* d_workspace,
                               size_t workspace_bytes, sd_vae** out);
/* fp32 parameters concatenated in manifest order; synchronous. */
sd_status synerdiff_vae_load_weights(sd_vae* h, const float* h_params, size_t n_floats, void* hip_stream);

/* The decoder's stages (sub-blocks) in execution order: "in" (scaling,
 * post-quantisation conv, conv_in), every ResBlock ("mid.res0", "up0.res2",
 * ...), "mid.attn", every upsampling conv ("up1.up", ...), "out" (GroupNorm,
 * SiLU, conv_out).  stage_flops gives a stage's algorithmic FLOPs per image
 * (2 x MACs of its convolutions, linears and attention products). */
int32_t synerdiff_vae_stage_count(const sd_vae* h);
sd_status synerdiff_vae_stage_name(const sd_vae* h, int32_t i, char* name, size_t name_cap);
sd_status synerdiff_vae_stage_flops(const sd_vae* h, int32_t i, double* flop);

/* Run stages [begin, end) for n images (1 <= n <= max_images).
 *   d_latents [n, latent_c, H, W] fp32 (NCHW), read when begin = 0;
 *   d_image   [n, out_c, 8 H, 8 W] fp32 (NCHW) for the default SD depth
 *             (2^(n_levels-1) H in general), written when end = stage count.
 * A decode split into chunks calls this with consecutive ranges
 * [0, b1), [b1, b2), ... on one handle with the same n; the activation
 * between chunks stays in the workspace.  begin must be 0 or the end of the
 * previous call (else SD_ERR_INVALID_ARG).  Asynchronous on hip_stream; a
 * handle decodes one batch at a time. */
sd_status synerdiff_vae_run(sd_vae* h, int32_t n, const float* d_latents, int32_t begin, int32_t end, float* d_image,
                            void* hip_stream);
/* Where the activation after stage i lives once a run has ended at stage
 * i + 1 (i < stage count - 1): its byte offset within the caller's
 * workspace buffer and its shape [n, H, W, C] (channels-last, the handle's
 * dtype).  For inspection between chunks; host only. */
sd_status synerdiff_vae_activation(const sd_vae* h, int32_t i, int64_t* offset_bytes, int32_t* H, int32_t* W,
                                   int32_t* C);
void synerdiff_vae_destroy(sd_vae* h);

/* VAE Chunking's partition (Sec. III-B: "temporally equivalent" sub-blocks
 * at ResNet-block boundaries): split stages 0..n_stages-1 with per-stage
 * costs stage_cost[] (e.g. measured solo milliseconds) into c contiguous
 * chunks minimising the largest chunk cost (ties: the earliest boundaries).
 * bounds[0..c] receives 0 = b_0 < b_1 < ... < b_c = n_stages.  Host only.
 * 1 <= c <= n_stages. */
sd_status synerdiff_vae_chunk_plan(const double* stage_cost, int32_t n_stages, int32_t c, int32_t* bounds);

/* Eq. (2) (Sec. III-C): the cumulative latencies over c rounds from the
 * per-round UNet and VAE latencies t_u[i], t_v[i] (i < c):
 *   T_u(c) = sum_{i<c} max(t_u[i], t_v[i]),
 *   T_v(c) = sum_{i<c-1} max(t_u[i], t_v[i]) + t_v[c-1];
 * and Eq. (1): L(c) = lambda (T_u(c) - T_u0) / T_u0 + (1 - lambda) (T_v(c) - T_v0) / T_v0
 * with the solo latencies T_u0, T_v0.  Host only. */
sd_status synerdiff_chunk_cost(const double* t_u, const double* t_v, int32_t c, double T_u0, double T_v0,
                               double lambda, double* T_u, double* T_v, double* L);

#ifdef __cplusplus
}
#endif
#endif /* SYNERDIFF_VAE_H */
