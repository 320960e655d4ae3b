// Internal interface between the host runtime and the HIP kernels.
// Activations are NHWC ("rows" = packed CFG rows = images), stored in the
// handle's dtype (fp32 or bf16); statistics, biases and accumulators are fp32.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace sd {

enum DType { F32 = 0, BF16 = 1 };
// bf16 storage as seen from host code (the kernels read it as __bf16).
typedef uint16_t bf16_t;

// One K-segment of an implicit-GEMM A operand.  Row m of A is output pixel
// (img, oy, ox) of an Ho x Wo image; column k is (tap, c) with
// tap = k / cin (ky = tap / ks, kx = tap % ks) and input channel c.  The
// element is the input pixel under that tap, after the optional nearest-2x
// upsample, the optional per-(img, channel) affine (GroupNorm) and SiLU, and
// zero outside the image (conv zero padding).  Channels c < c0 come from
// src0, the rest from src1 (the skip concat [h | skip] of the up path).
struct ASeg {
  const void* src0;
  const void* src1;
  const float* scale;  // [imgs, cin] or null
  const float* shift;  // [imgs, cin]
  int c0, c1, cin;     // cin = c0 + c1; c0, c1 multiples of 8
  int ks;              // 1 or 3; 2: one phase of a nearest-2x upsample + 3x3 conv (below)
  int stride;          // 1 or 2
  int up;              // 1: nearest-2x upsample before the conv
  int Hi, Wi, Ho, Wo;  // input (before upsampling) and output sizes
  int K;               // ks * ks * cin
  int silu;
  int py, px;          // ks == 2: output phase (2 y + py, 2 x + px); tap (ty, tx) reads the
                       //   input at (y + py - 1 + ty, x + px - 1 + tx), zero outside
};

// Epilogue: out[m, n] = acc + bias[n] + tbias[row_req... ] + resid[m, n].
struct Epi {
  const float* bias;      // [N] or null
  const float* tbias;     // time bias: tbias[img * tb_ld + tb_off + n], or null
  int tb_ld, tb_off, hw;  // img = m / hw
  const void* resid;      // [M, ldr] in the activation dtype, or null (may equal out)
  int ldr;
  void* out;              // [M, ldo]
  int ldo;
  int out_f32;            // 1: fp32 output regardless of the activation dtype
  int geglu;              // bf16 only: columns packed as 32-blocks [a(16) | gate(16)];
                          // out[m, 16t + u] = (a + b) * GELU(gate + b), ldo = N / 2
  void* vt_out;           // bf16 only: columns n >= vt_col0 are written transposed (no bias),
  int vt_col0, vt_hw;     //   vt_out[(m / vt_hw) * vt_img + (n - vt_col0) * vt_ld + m % vt_hw]
  int vt_ld;
  long vt_img;
  int qcols;              // columns n < qcols are multiplied by qscale before rounding
  float qscale;           //   (attention queries stored in base-2 logit units)
  int phase, ph_h, ph_w;  // phase = 1 + 2 py + px: GEMM row m = (image i, y, x) of an ph_h x ph_w
                          //   grid is output row i (4 ph_h ph_w) + (2 y + py) (2 ph_w) + 2 x + px;
                          //   0: row m is output row m
  const float* rowscale;  // bf16 only: acc -> rowscale[m] * acc before the bias, or null (the
                          //   LayerNorm rstd of input row m when the LN is folded into the weights)
};

struct GemmArgs {
  int M, N, K;       // K = seg[0].K + seg[1].K (seg[1].K = 0 if unused)
  ASeg seg[2];
  const void* B;     // packed weights [N, ldb], K contiguous, activation dtype
  int ldb;
  Epi epi;
  int ksplit;        // >= 1; > 1: K split into ksplit ranges, fp32 partials in
  float* partial;    //   partial[ksplit][M][N], summed in order by a second kernel
};

// bf16 requires N % 4 == 0, 8-byte aligned outputs and ldo, ldr % 4 == 0.
hipError_t launch_gemm(DType dt, const GemmArgs& a, hipStream_t s);
// Split-K factor launch_gemm supports for this bf16 GEMM (1 = no split).
int gemm_ksplit(const GemmArgs& a);

// Attention: O = softmax(Q K^T * scale) V per (img, head).
struct AttnArgs {
  const void* q; long q_ld, q_img;   // Q[img][token][c]: token stride, image stride (elements)
  const void* k; long k_ld, k_img;   // K likewise
  const void* v; long v_ld, v_img;   // V: vt = 0 like K; vt = 1 transposed, V[img][c][token] at
  int vt;                            //    v + img*v_img + c*v_ld + token (bf16 only)
  const int* kv_index;               // kv image of each q image, or null (= same)
  void* o; long o_ld, o_img;
  int imgs, heads, d, Nq, Nk;
  float scale;
  int q_log2;                        // 1: Q already holds q * scale * log2(e) (bf16 only)
};
hipError_t launch_attention(DType dt, const AttnArgs& a, hipStream_t s);
// bf16 head widths the attention kernel is built for: d a multiple of 8
// whose rounding up to 16 is 16..96, 128, 160, 192 or 256.
bool attention_width_ok(int d);

// GroupNorm statistics over up to two channel-concatenated NHWC sources;
// writes per-(img, channel) scale = gamma*rstd and shift = beta - mean*scale.
hipError_t launch_groupnorm_stats(DType dt, const void* src0, int c0, const void* src1, int c1,
                                  int imgs, int hw, int groups, float eps, const float* gamma,
                                  const float* beta, float* partial, float* scale, float* shift,
                                  hipStream_t s);
size_t groupnorm_partial_floats(int imgs, int hw, int cin);
// The library's own partial-sum array on the current device (a static
// __device__ array of groupnorm_scratch_floats_max() floats; its address is
// looked up once per device) for the entry point that allocates nothing.
size_t groupnorm_scratch_floats_max();
hipError_t groupnorm_scratch(float** out);
// out = act(x * scale + shift) over the concat [src0 | src1] (act = SiLU or identity).
// Statistics and apply in one launch for small images (bf16; see
// groupnorm_fused_ok for the shapes it takes).
bool groupnorm_fused_ok(DType dt, int c0, int c1, int hw, int groups);
hipError_t launch_groupnorm_fused(DType dt, const void* src0, int c0, const void* src1, int c1, int imgs, int hw,
                                  int groups, float eps, const float* gamma, const float* beta, int silu, void* out,
                                  hipStream_t s);
hipError_t launch_groupnorm_apply(DType dt, const void* src0, int c0, const void* src1, int c1, int imgs,
                                  int hw, const float* scale, const float* shift, int silu, void* out,
                                  hipStream_t s);

hipError_t launch_layernorm(DType dt, const void* x, void* y, long tokens, int C, const float* gamma,
                            const float* beta, float eps, hipStream_t s);
// Per-token LayerNorm scale: rstd[t] = 1 / sqrt(var_t + eps) (biased variance).
hipError_t launch_layernorm_rstd(DType dt, const void* x, float* rstd, long tokens, int C, float eps,
                                 hipStream_t s);

// y[t, j] = x[t, j] * gelu(x[t, half + j]), j < half; x is [tokens, 2*half].
hipError_t launch_geglu(DType dt, const void* x, void* y, long tokens, int half, hipStream_t s);

// Per-row scalars of a step (device arrays in the workspace).
struct RowMaps {
  const int* row_req;     // [rows]
  const int* row_branch;  // [rows]
  const int* row_ctx;     // [rows]
  const float* row_t;     // [rows]
  const int* req_row_u;   // [n_req]
  const float* req_coef;  // [n_req, 3] = (A, B, w)
};

hipError_t launch_pack_latents(DType dt, const float* lat, void* x0, int rows, int lc, int hw,
                               int cpad, const int* row_req, hipStream_t s);
// e[row, :] = [cos(t f_i) | sin(t f_i)] (+ [pooled | sinusoids of time ids] for add_in)
hipError_t launch_time_inputs(const float* row_t, int rows, int temb_in, float* e,
                              const float* pooled_cond, const float* pooled_uncond,
                              const int* row_req, const int* row_branch, int pooled_dim,
                              const float* time_ids_dev, int n_ids, int id_dim, float* a,
                              hipStream_t s);
// out[m, n] = act_out(sum_k act_in(in[m, k]) W[n, k] + bias[n] + add[m, n]) for a few rows; K % 4 == 0.
hipError_t launch_linear_smallm(DType wdt, const float* in, int M, int K, const void* W,
                                const float* bias, const float* add, float* out, int N,
                                int silu_in, int silu_out, hipStream_t s);
// Rows dst0 .. dst0 + n - 1 of a row-major tensor (row_bytes each, a
// multiple of 16) become copies of rows src_rows[0 .. n - 1].
hipError_t launch_copy_rows(void* base, long row_bytes, int dst0, int n, const int* src_rows, hipStream_t s);
// Output conv (3x3, C -> 4) of each request's rows + CFG combine + DDIM in
// one kernel (bf16): x holds the normalised (GroupNorm + SiLU) rows
// [rows, H, W, C]; w the conv weight packed [4][9 C] (tap-major, channel-
// minor), bias [4].  Request r reads row r and, if req_row_u[r] >= 0, that
// unconditional row; lat_* are [n_req, 4, H, W] fp32.  order (or null)
// lists the requests in launch order.
struct OutArgs {
  const bf16_t* x;
  const bf16_t* w;
  const float* bias;
  const float* lat_in;
  float* lat_out;
  float* eps_out;  // or null
  const int* req_row_u;
  const float* req_coef;  // [n_req, 3] = (A, B, w)
  const int* order;
  int n_req, H, W, C;
  int tiles;  // set by the launcher
};
bool out_cfg_ddim_ok(DType dt, int latent_c, int H, int W, int C);
size_t out_cfg_ddim_lds_bytes(int W);
hipError_t launch_out_cfg_ddim(const OutArgs& a, hipStream_t s);
hipError_t launch_cfg_ddim(const float* eps_rows, const float* lat_in, float* lat_out,
                           float* eps_out, int n_req, int lc, int hw, const int* req_row_u,
                           const float* req_coef, hipStream_t s);

}  // namespace sd
