/*
 * synerdiff_ops.h - kernel-level entry points of the UNet step.
 *
 * Each call runs one of the step's kernels on caller-owned device buffers so
 * that a kernel can be checked on its own against the layer it implements.
 * Conventions as in synerdiff.h: device pointers, the caller's stream,
 * validation before enqueue, SD_ERR_HIP on a launch failure.  `dtype` is
 * SD_F32 or SD_BF16 and types every activation and weight argument; norm
 * statistics, biases and affine parameters are always fp32.
 * Activations are channels-last: [n, H, W, C].
 */
#ifndef SYNERDIFF_OPS_H
#define SYNERDIFF_OPS_H

#include "synerdiff.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Convolution as an implicit GEMM (3x3 or 1x1 layers of the UNet):
 *   out[i, y, x, o] = bias[o] + resid[i, y, x, o]
 *       + sum_{ky, kx, c} A(i, s*y + ky - p, s*x + kx - p, c) * w[o, (ky*ks + kx)*cin + c]
 * with p = (ks - 1) / 2, cin = c0 + c1, A the channel concat [x0 | x1]
 * (x1 may be NULL with c1 = 0), optionally nearest-2x upsampled first
 * (up = 1), optionally transformed per (image, channel) as
 * v * scale + shift (GroupNorm affine; scale/shift [n, cin] fp32 or NULL)
 * and then SiLU (silu = 1), and zero outside the image (zero padding after
 * the transform).  Output size: H/stride (stride 2 needs even H, W) or 2H
 * when upsampling.  w is the packed weight [cout, ks*ks*cin] (tap-major,
 * channel-minor).  bias may be NULL; resid ([n, Ho, Wo, cout], activation
 * dtype) may be NULL or equal to out.  out_f32 = 1 writes fp32 output.
 * d_scratch (fp32, scratch_floats long, may be NULL) lets the call split K
 * the way the step does for long-K 3x3 layers on small images (ks = 1 never
 * splits);
 * synerdiff_op_conv_scratch_floats returns the floats that needs (0 = no
 * split for this shape).
 * Constraints: ks in {1, 3}; stride in {1, 2}; c0, c1 multiples of 8;
 * bf16: cout a multiple of 4. */
sd_status synerdiff_op_conv(int32_t dtype, const void* d_x0, int32_t c0, const void* d_x1, int32_t c1,
                            int32_t n, int32_t H, int32_t W, int32_t ks, int32_t stride, int32_t up,
                            const float* d_scale, const float* d_shift, int32_t silu, const void* d_w,
                            int32_t cout, const float* d_bias, const void* d_resid, void* d_out,
                            int32_t out_f32, float* d_scratch, int64_t scratch_floats, void* hip_stream);
int64_t synerdiff_op_conv_scratch_floats(int32_t dtype, int32_t c0, int32_t c1, int32_t n, int32_t H, int32_t W,
                                         int32_t ks, int32_t stride, int32_t up, int32_t cout);

/* The 3x3 convolution (zero padding 1) of a nearest-2x upsampled input, as
 * the bf16 step runs the UNet's upsampling layers: four 2x2 convolutions on
 * the input grid, one per output phase.  Output pixel (2y + py, 2x + px)
 * = bias + sum over taps (ty, tx) in {0,1}^2 and channels c of
 * x[y + py - 1 + ty, x + px - 1 + tx, c] (zero outside) * w[2 py + px, o, 2 ty + tx, c],
 * where phase weight (ty, tx) is the sum of the 3x3 taps (ky, kx) with
 * floor((py + ky - 1) / 2) = py - 1 + ty and floor((px + kx - 1) / 2) =
 * px - 1 + tx.  x [n, H, W, cin] and out [n, 2H, 2W, cout] bf16, w bf16
 * [4][cout][4 cin], bias fp32 [cout] or NULL.  dtype must be SD_BF16;
 * cin a multiple of 32, cout of 160 (else SD_ERR_INVALID_ARG). */
sd_status synerdiff_op_upconv(int32_t dtype, const void* d_x, int32_t n, int32_t H, int32_t W, int32_t cin,
                              const void* d_w, int32_t cout, const float* d_bias, void* d_out, void* hip_stream);

/* Multi-head attention O = softmax(Q K^T * scale) V per image and head
 * (head h uses channels [h*d, (h+1)*d)).  Q: image i, token t, channel c at
 * q + i*q_img + t*q_ld + c; K likewise with k_img, k_ld and image
 * kv_index[i] (d_kv_index NULL = image i); V likewise with v_img, v_ld
 * (fp32), or, with v_transposed = 1 (required for bf16), at
 * v + j*v_img + c*v_ld + t (channel-major, the layout the step's
 * projections write); O like Q with o_img, o_ld.  Strides in elements.
 * q_log2 = 1: Q already holds q * scale * log2(e), as the step's bf16
 * projections write it (scale is then unused).  Constraints: d a multiple
 * of 8; bf16: d rounded up to 16 is 16..96, 128, 160, 192 or 256; fp32:
 * d <= 256 (V row-major). */
sd_status synerdiff_op_attention(int32_t dtype, const void* d_q, int64_t q_ld, int64_t q_img,
                                 const void* d_k, int64_t k_ld, int64_t k_img, const void* d_v,
                                 int64_t v_ld, int64_t v_img, int32_t v_transposed,
                                 const int32_t* d_kv_index, void* d_o, int64_t o_ld, int64_t o_img,
                                 int32_t n, int32_t heads, int32_t d, int32_t n_q, int32_t n_k,
                                 float scale, int32_t q_log2, void* hip_stream);

/* GroupNorm statistics of the concat [x0 | x1] ([n, hw, c0 + c1]) with
 * `groups` groups of consecutive channels, biased variance, eps: writes the
 * per-(image, channel) affine scale = gamma * rstd, shift = beta - mean *
 * scale (fp32 [n, cin]) that synerdiff_op_conv applies.  d_partial is
 * scratch of synerdiff_op_groupnorm_scratch_floats(n, hw, cin) floats. */
size_t synerdiff_op_groupnorm_scratch_floats(int32_t n, int32_t hw, int32_t cin);
sd_status synerdiff_op_groupnorm_stats(int32_t dtype, const void* d_x0, int32_t c0, const void* d_x1,
                                       int32_t c1, int32_t n, int32_t hw, int32_t groups, float eps,
                                       const float* d_gamma, const float* d_beta, float* d_partial,
                                       float* d_scale, float* d_shift, void* hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * synerdiff_op_groupnorm_stats without d_partial.  The partial sums go to a
 * device array the library owns, SYNERDIFF_GN_NOALLOC_SCRATCH_FLOATS floats
 * (16 MiB) per device, held until the process ends; the call itself
 * allocates nothing.  A call whose partial sums,
 * synerdiff_op_groupnorm_scratch_floats(n, hw, c0 + c1), exceed that size
 * returns SD_ERR_CAPACITY before enqueueing anything.  Every call on a device
 * shares its array: calls that overlap in time on one device (different
 * streams or host threads) race.  Each call writes every partial it reads,
 * so no clearing is needed between calls.  Arguments and outputs as for
 * synerdiff_op_groupnorm_stats. */
#define SYNERDIFF_GN_NOALLOC_SCRATCH_FLOATS (1u << 22)
sd_status synerdiff_op_groupnorm_stats_noalloc(int32_t dtype, const void* d_x0, int32_t c0, const void* d_x1,
                                               int32_t c1, int32_t n, int32_t hw, int32_t groups, float eps,
                                               const float* d_gamma, const float* d_beta, float* d_scale,
                                               float* d_shift, void* hip_stream);

/* GroupNorm of the concat [x0 | x1] ([n, hw, c0 + c1], `groups` groups of
 * consecutive channels, biased variance, eps) followed by SiLU when silu =
 * 1, written to out [n, hw, c0 + c1]: the normalisation in front of every
 * ResBlock conv of the latent-diffusion UNet the paper serves (Sec. IV-A),
 * as the step runs it on its small images, statistics and apply in one
 * kernel (one block per (group, image)).  bf16 only; the channels per group
 * a multiple of 4, c0 and c1 multiples of 4, and hw * (channels per group)
 * / 4 <= 5120 (SD_ERR_UNSUPPORTED otherwise).  gamma, beta fp32 [c0 + c1].
 * n = 0 does nothing. */
sd_status synerdiff_op_groupnorm_fused(int32_t dtype, const void* d_x0, int32_t c0, const void* d_x1, int32_t c1,
                                       int32_t n, int32_t hw, int32_t groups, float eps, const float* d_gamma,
                                       const float* d_beta, int32_t silu, void* d_out, void* hip_stream);

/* LayerNorm over the last axis of x [tokens, C] (biased variance):
 * y = (x - mean) * rstd * gamma + beta.  C a multiple of 8, <= 2048. */
sd_status synerdiff_op_layernorm(int32_t dtype, const void* d_x, void* d_y, int64_t tokens, int32_t C,
                                 const float* d_gamma, const float* d_beta, float eps, void* hip_stream);

/* The LayerNorm scale alone, rstd[t] = 1 / sqrt(var_t + eps) with the
 * biased variance of token t of x [tokens, C] (C a multiple of 8, <= 2048):
 * the per-token factor of the SD transformer blocks' LayerNorms when their
 * mean, gain and shift are folded into the projection weights (the
 * latent-diffusion UNet the paper serves, Sec. IV-A).  rstd is fp32
 * [tokens], device memory owned by the caller; nothing else is written.
 * tokens = 0 does nothing. */
sd_status synerdiff_op_layernorm_rstd(int32_t dtype, const void* d_x, float* d_rstd, int64_t tokens, int32_t C,
                                      float eps, void* hip_stream);

/* Linear layer over a few fp32 rows, the per-request timestep-embedding
 * MLP and time projections of the latent-diffusion UNet the paper serves
 * (Sec. IV-A):
 *   out[m, n] = act_out(bias[n] + add[m, n] + sum_k act_in(in[m, k]) * w[n, k])
 * with act_* = SiLU where silu_* = 1, else the identity.  in [M, K] and out
 * [M, N] fp32 (out must not overlap in; add may equal out), w [N, K] in
 * `dtype`, bias [N] fp32; bias and add may be NULL.  K a multiple of 4;
 * buffers 16-byte aligned.  M = 0 or N = 0 does nothing. */
sd_status synerdiff_op_linear_rows(int32_t dtype, const float* d_in, int32_t M, int32_t K, const void* d_w,
                                   const float* d_bias, const float* d_add, float* d_out, int32_t N,
                                   int32_t silu_in, int32_t silu_out, void* hip_stream);

/* GEGLU: y[t, j] = x[t, j] * GELU(x[t, half + j]) with exact GELU; x is
 * [tokens, 2*half], y [tokens, half]; half a multiple of 8. */
sd_status synerdiff_op_geglu(int32_t dtype, const void* d_x, void* d_y, int64_t tokens, int32_t half,
                             void* hip_stream);

/* The step's last stage as one kernel: the UNet's output convolution, the
 * classifier-free guidance combine and the DDIM update (CFG as in Ho &
 * Salimans 2022; Skip-CFG bypasses the unconditional branch, Sec. II-B and
 * Sec. III-B; DDIM eta = 0, Song et al. 2021).  For request r < n_req and
 * each pixel p, channel o < 4:
 *   eps_c = b[o] + sum_{ky, kx, c} x[r, y + ky - 1, x + kx - 1, c] w[o, (3 ky + kx) C + c]
 *   (zero outside the image); eps_u likewise from row req_row_u[r] when it
 *   is >= 0; eps = eps_u + w_r (eps_c - eps_u) if so, else eps_c;
 *   lat_out[r, o, p] = A_r lat_in[r, o, p] + B_r eps;  eps_out (if not NULL) = eps.
 * x: device bf16 [rows, H, W, C] (rows covering every index used), the
 * normalised (GroupNorm + SiLU) input of the output conv.  w: device bf16
 * [4][9 C] (the layout synerdiff_op_conv takes), bias fp32 [4].
 * d_req_row_u: device int32 [n_req]; d_req_coef: device fp32 [n_req, 3] =
 * (A_r, B_r, w_r).  lat_in, lat_out, eps_out: device fp32 [n_req, 4, H, W]
 * (NCHW); lat_out may equal lat_in, eps_out must not overlap either.
 * dtype must be SD_BF16; C a multiple of 32 and <= 320, W <= 128
 * (SD_ERR_UNSUPPORTED otherwise).  n_req = 0 does nothing. */
sd_status synerdiff_op_conv_out_cfg_ddim(int32_t dtype, const void* d_x, int32_t H, int32_t W, int32_t C,
                                         const void* d_w, const float* d_bias, int32_t n_req,
                                         const int32_t* d_req_row_u, const float* d_req_coef,
                                         const float* d_lat_in, float* d_lat_out, float* d_eps_out,
                                         void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* SYNERDIFF_OPS_H */
