/*
 * synerdiff.h - C ABI of the MI355X (gfx950) step-level continuous-batching
 * UNet denoising step with Adaptive Skip-CFG.
 *
 * The operation (SynerDiff, Sec. III-B and the problem statement of Sec. III-D):
 * one UNet denoising iteration over a ragged batch of requests.  Request r is
 * at its own timestep t_r (its own denoising progress), has its own guidance
 * scale w_r, and either keeps classifier-free guidance (cfg_on = 1: a
 * conditional and an unconditional UNet evaluation, combined as
 * eps = eps_u + w (eps_c - eps_u)) or runs Skip-CFG (cfg_on = 0: the
 * unconditional branch is bypassed and eps = eps_c).  The step ends with the
 * deterministic DDIM update x' = A_r x + B_r eps (Song et al. 2021, eta = 0).
 * The UNet is the latent-diffusion UNet (Rombach et al. 2022) in its SD-1.5
 * and SDXL shapes (Sec. IV-A serves SD-v1.5).
 *
 * Conventions shared by every entry point:
 *  - Device pointers ("d_") point to memory the caller allocated on the
 *    current HIP device; host pointers ("h_") to ordinary host memory.  The
 *    library never frees caller memory and allocates no device memory; it
 *    owns only a small pinned host staging ring per handle.
 *  - All work is enqueued on the caller's stream (`hip_stream`, a
 *    hipStream_t; NULL = the default stream) and the call returns after
 *    enqueue unless stated otherwise.
 *  - Arguments are validated before anything is enqueued; on error nothing
 *    is enqueued, outputs are untouched, and synerdiff_last_error() holds a
 *    message.  A HIP launch or copy failure returns SD_ERR_HIP.
 *  - A handle serves one host thread at a time.
 */
#ifndef SYNERDIFF_H
#define SYNERDIFF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SYNERDIFF_ABI_VERSION 1

typedef enum {
  SD_OK = 0,
  SD_ERR_INVALID_ARG = -1, /* NULL pointer, value out of range, bad aliasing   */
  SD_ERR_UNSUPPORTED = -2, /* shape the kernels do not support                 */
  SD_ERR_CAPACITY = -3,    /* more requests than the handle was created for    */
  SD_ERR_WORKSPACE = -4,   /* weight or workspace buffer too small             */
  SD_ERR_HIP = -5          /* a HIP runtime call or kernel launch failed       */
} sd_status;

typedef enum { SD_F32 = 0, SD_BF16 = 1 } sd_dtype;
typedef enum { SD_SCHED_LINEAR = 0, SD_SCHED_SCALED_LINEAR = 1 } sd_schedule;

/* UNet shape.  One struct describes the tiny fp32 UNet, SD-1.5 and SDXL.
 * Supported: latent_c <= 8; ch[l] multiples of 8 and of gn_groups; at most
 * 4 levels; head width (ch/heads or head_dim) a multiple of 8 and <= 256;
 * ctx_dim a multiple of 8; latent_h, latent_w divisible by 2^(n_levels-1). */
typedef struct {
  int32_t latent_c, latent_h, latent_w; /* latent per request (C, H, W)           */
  int32_t n_levels;                     /* resolution levels (<= 4)               */
  int32_t ch[4];                        /* channel width per level                */
  int32_t n_res;                        /* ResBlocks per down level (+1 per up)   */
  int32_t tx_depth[4];                  /* transformer blocks per Transformer2D   */
  int32_t mid_tx_depth;                 /* ... in the mid block (0 = none)        */
  int32_t heads, head_dim;              /* exactly one non-zero                   */
  int32_t gn_groups;                    /* GroupNorm groups                       */
  int32_t ctx_len, ctx_dim;             /* text context tokens x width            */
  int32_t temb_in, temb_dim;            /* sinusoid width, time-embedding width   */
  int32_t add_in;                       /* added-embedding input width, 0 = none  */
  int32_t pooled_dim, time_id_dim, n_time_ids; /* add_in = pooled + ids*id_dim */
  int32_t max_requests;                 /* batch capacity; rows <= 2*max_requests */
  int32_t dtype;                        /* sd_dtype: storage/compute type         */
} sd_unet_config;

typedef struct sd_unet sd_unet; /* opaque, host-side handle */

int32_t synerdiff_abi_version(void);

/* Thread-local message describing the last error; valid until the next call. */
const char* synerdiff_last_error(void);

/* SD_OK if the shape is supported, else SD_ERR_UNSUPPORTED / INVALID_ARG. */
sd_status synerdiff_config_check(const sd_unet_config* cfg);

/* Parameter manifest: the tensors synerdiff_load_weights expects, in order.
 * synerdiff_param_count returns the number of tensors (< 0 on bad config).
 * synerdiff_param_info writes the name (NUL-terminated, truncated to
 * name_cap) and the shape (out, in[, kh, kw]; ndim <= 4) of tensor i. */
int64_t synerdiff_param_count(const sd_unet_config* cfg);
sd_status synerdiff_param_info(const sd_unet_config* cfg, int64_t i, char* name, size_t name_cap,
                               int64_t shape[4], int32_t* ndim);

/* Device bytes the caller must provide for packed weights and for the
 * per-step workspace (sized for cfg->max_requests).  0 on bad config. */
size_t synerdiff_weights_bytes(const sd_unet_config* cfg);
size_t synerdiff_workspace_bytes(const sd_unet_config* cfg);

/* Create a handle over caller-owned device buffers (256-byte aligned, on the
 * current device).  The buffers must outlive the handle. */
sd_status synerdiff_unet_create(const sd_unet_config* cfg, void* d_weights, size_t weights_bytes,
                                void* d_workspace, size_t workspace_bytes, sd_unet** out);

/* A handle for another latent size that uses the packed weights of `src`
 * (no second copy, no load): for serving requests of several resolutions
 * (the paper's requests are 512, 768 or 1024 px, Sec. IV-A) with one set of
 * weights, one handle per resolution, each step over one resolution's
 * ragged batch.  cfg must equal src's config in every field except
 * latent_h, latent_w and max_requests.  The weights buffer stays owned by
 * src's caller and must outlive this handle; loading weights through either
 * handle updates both. */
sd_status synerdiff_unet_create_shared(const sd_unet_config* cfg, const sd_unet* src, void* d_workspace,
                                       size_t workspace_bytes, sd_unet** out);

/* Load all parameters: h_params holds every manifest tensor, fp32, row-major,
 * concatenated in manifest order (n_floats = sum of their sizes).  The
 * library repacks them (bf16 for SD_BF16) into d_weights.  Synchronous: the
 * stream is synchronised before return. */
sd_status synerdiff_load_weights(sd_unet* h, const float* h_params, size_t n_floats, void* hip_stream);

/* One denoising step over n_req requests (0 <= n_req <= max_requests;
 * n_req == 0 does nothing).  Rows: the conditional row of request r is row
 * r; requests with cfg_on get an unconditional row n_req + (number of
 * cfg_on requests before r).
 *   d_latents_in    [n_req, C, H, W] fp32 (NCHW)
 *   h_timesteps     [n_req] in [0, 999]
 *   h_cfg_on        [n_req] 0 (Skip-CFG: conditional row only) or 1
 *   h_guidance      [n_req] finite; read only where cfg_on = 1
 *   d_ctx_cond      [n_req, ctx_len, ctx_dim] in cfg dtype (fp32 or bf16)
 *   d_ctx_uncond    [ctx_len, ctx_dim] in cfg dtype, the shared null context
 *   d_pooled_cond   [n_req, pooled_dim] fp32 (add_in > 0 only, else NULL)
 *   d_pooled_uncond [pooled_dim] fp32 (add_in > 0 only, else NULL)
 *   h_time_ids      [n_time_ids] (add_in > 0 only, else NULL)
 *   h_sampler_coef  [n_req, 2] = (A_r, B_r), finite: x' = A x + B eps
 *   d_latents_out   [n_req, C, H, W] fp32; may equal d_latents_in exactly
 *                   (in place); any other overlap is SD_ERR_INVALID_ARG
 *   d_eps_out       optional [n_req, C, H, W] fp32 guided eps; NULL = off
 * Two calls on one handle must not overlap in time on different streams
 * (they share the workspace). */
sd_status synerdiff_unet_step(sd_unet* h, int32_t n_req, const float* d_latents_in,
                              const int32_t* h_timesteps, const uint8_t* h_cfg_on,
                              const float* h_guidance, const void* d_ctx_cond,
                              const void* d_ctx_uncond, const float* d_pooled_cond,
                              const float* d_pooled_uncond, const float* h_time_ids,
                              const float* h_sampler_coef, float* d_latents_out,
                              float* d_eps_out, void* hip_stream);

/* Row plan of the ragged CFG packing (host only, no GPU work): writes
 * row_req[rows], row_branch[rows] (0 cond, 1 uncond), req_row_u[n_req]
 * (-1 under Skip-CFG) and *n_rows.  Arrays must hold 2*n_req entries. */
sd_status synerdiff_row_plan(int32_t n_req, const uint8_t* h_cfg_on, int32_t* row_req,
                             int32_t* row_branch, int32_t* req_row_u, int32_t* n_rows);

/* Cumulative alpha products abar_t = prod_{s<=t}(1 - beta_s), t < 1000, of
 * the DDPM linear (1e-4..0.02) or latent-diffusion scaled-linear
 * (sqrt: sqrt(0.00085)..sqrt(0.012)) beta schedule.  Host only. */
sd_status synerdiff_alphas_cumprod(int32_t schedule, double out[1000]);

/* DDIM (eta = 0) coefficients of x' = A x + B eps for t -> t_prev, with
 * abar_prev = 1 when t_prev < 0.  Host only. */
sd_status synerdiff_ddim_coef(const double* alphas_cumprod, int32_t t, int32_t t_prev, float out_AB[2]);

/* The same update for a v-prediction UNet (SD-2.x; Salimans & Ho 2022):
 * the network predicts v = sqrt(abar) eps - sqrt(1 - abar) x0, the guidance
 * combine acts on v, and x' = A x + B v with
 *   A = sqrt(abar_prev abar_t) + sqrt((1 - abar_prev)(1 - abar_t)),
 *   B = sqrt((1 - abar_prev) abar_t) - sqrt(abar_prev (1 - abar_t)),
 * which is the DDIM step through x0 = sqrt(abar_t) x - sqrt(1 - abar_t) v and
 * eps = sqrt(1 - abar_t) x + sqrt(abar_t) v.  Pass these (A, B) to
 * synerdiff_unet_step; d_eps_out then holds the guided v.  Host only. */
sd_status synerdiff_ddim_coef_v(const double* alphas_cumprod, int32_t t, int32_t t_prev, float out_AB[2]);

/* Per-kernel timing of the step (the offline-profiling measurements of
 * Sec. III-C: latency of the UNet step's components).  While enabled, the
 * step records a HIP event on its stream after every launch; the time
 * between consecutive events is that launch's device time.
 * synerdiff_profile_read waits for the recorded events and returns totals
 * per kernel class since the last reset: launches, device milliseconds and
 * the algorithmic work of those launches (flop: 2*MACs of the real, unpadded
 * products; bytes: one read of every input and one write of every output).
 * Returns the number of classes in *n_out (entries beyond cap are counted
 * but not written). */
typedef struct {
  char name[24];
  int64_t launches;
  double ms;
  double flop;
  double bytes;
} sd_kernel_stat;
sd_status synerdiff_profile(sd_unet* h, int32_t enable);
sd_status synerdiff_profile_read(sd_unet* h, sd_kernel_stat* out, int32_t cap, int32_t* n_out, int32_t reset);
/* The same totals per layer instead of per class: one entry per distinct
 * launch name ("conv1 196608x320x2880" = a GEMM named conv1 with M x N x K,
 * "self-attention 4096x4096 d40" = query x key tokens and head width, other
 * kernels by their step name), in first-launch order.  Same arguments and
 * reset semantics as synerdiff_profile_read. */
typedef struct {
  char name[64];
  int64_t launches;
  double ms;
  double flop;
  double bytes;
} sd_layer_stat;
sd_status synerdiff_profile_read_layers(sd_unet* h, sd_layer_stat* out, int32_t cap, int32_t* n_out,
                                        int32_t reset);

void synerdiff_unet_destroy(sd_unet* h);

#ifdef __cplusplus
}
#endif
#endif /* SYNERDIFF_H */
