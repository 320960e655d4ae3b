// Kernel-level C entry points (synerdiff_ops.h): validation + one launch.
#include <hip/hip_runtime_api.h>
#include <string.h>

#include <string>

#include "kernels.h"
#include "synerdiff_ops.h"

namespace sd {
extern thread_local std::string g_err;
}
using namespace sd;

static sd_status op_fail(sd_status s, const char* m) {
  g_err = m;
  return s;
}
static sd_status op_hip(hipError_t e, const char* w) {
  if (e == hipSuccess) return SD_OK;
  g_err = std::string(w) + ": " + hipGetErrorString(e);
  return SD_ERR_HIP;
}
static bool bad_dtype(int32_t d) { return d != SD_F32 && d != SD_BF16; }

extern "C" {

static bool conv_args(int32_t dtype, const void* x0, int32_t c0, const void* x1, int32_t c1, int32_t n, int32_t H,
                      int32_t W, int32_t ks, int32_t stride, int32_t up, const float* scale, const float* shift,
                      int32_t silu, const void* w, int32_t cout, const float* bias, const void* resid, void* out,
                      int32_t out_f32, GemmArgs& a) {
  memset(&a, 0, sizeof(a));
  ASeg& s = a.seg[0];
  s.src0 = x0; s.src1 = x1; s.c0 = c0; s.c1 = c1; s.cin = c0 + c1;
  s.scale = scale; s.shift = shift; s.silu = silu ? 1 : 0;
  s.ks = ks; s.stride = stride; s.up = up ? 1 : 0;
  s.Hi = H; s.Wi = W;
  s.Ho = up ? 2 * H : H / stride;
  s.Wo = up ? 2 * W : W / stride;
  s.K = ks * ks * s.cin;
  const long M = (long)n * s.Ho * s.Wo;
  if (M > 0x7FFFFFFFL) return false;
  a.M = (int)M; a.N = cout; a.K = s.K; a.B = w; a.ldb = s.K;
  a.epi.bias = bias; a.epi.resid = resid; a.epi.ldr = cout; a.epi.out = out; a.epi.ldo = cout;
  a.epi.out_f32 = out_f32 ? 1 : 0; a.epi.hw = 1;
  a.ksplit = 1;
  (void)dtype;
  return true;
}

int64_t synerdiff_op_conv_scratch_floats(int32_t dtype, int32_t c0, int32_t c1, int32_t n, int32_t H, int32_t W,
                                         int32_t ks, int32_t stride, int32_t up, int32_t cout) {
  if (dtype != SD_BF16 || n <= 0 || H < 1 || W < 1 || c0 < 8 || cout < 1) return 0;
  GemmArgs a;
  static int dummy;
  if (!conv_args(dtype, &dummy, c0, c1 ? &dummy : nullptr, c1, n, H, W, ks, stride, up, nullptr, nullptr, 0,
                 &dummy, cout, nullptr, nullptr, &dummy, 0, a))
    return 0;
  const int ksplit = gemm_ksplit(a);
  return ksplit > 1 ? (int64_t)ksplit * a.M * a.N : 0;
}

sd_status synerdiff_op_conv(int32_t dtype, const void* x0, int32_t c0, const void* x1, int32_t c1, int32_t n,
                            int32_t H, int32_t W, int32_t ks, int32_t stride, int32_t up, const float* scale,
                            const float* shift, int32_t silu, const void* w, int32_t cout, const float* bias,
                            const void* resid, void* out, int32_t out_f32, float* scratch, int64_t scratch_floats,
                            void* stream) {
  if (bad_dtype(dtype)) return op_fail(SD_ERR_INVALID_ARG, "bad dtype");
  if (!x0 || !w || !out || (c1 && !x1) || (!scale) != (!shift)) return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  if (n < 0 || H < 1 || W < 1 || c0 < 8 || c0 % 8 || c1 < 0 || c1 % 8 || cout < 1)
    return op_fail(SD_ERR_INVALID_ARG, "bad shape");
  if ((ks != 1 && ks != 3) || (stride != 1 && stride != 2) || (up && stride != 1) || (ks == 1 && (stride != 1 || up)))
    return op_fail(SD_ERR_UNSUPPORTED, "unsupported ks/stride/up");
  if (stride == 2 && (H % 2 || W % 2)) return op_fail(SD_ERR_UNSUPPORTED, "stride 2 needs even H, W");
  if (dtype == SD_BF16 && cout % 4) return op_fail(SD_ERR_UNSUPPORTED, "bf16 needs cout % 4 == 0");
  if (n == 0) return SD_OK;
  GemmArgs a;
  if (!conv_args(dtype, x0, c0, x1, c1, n, H, W, ks, stride, up, scale, shift, silu, w, cout, bias, resid, out,
                 out_f32, a))
    return op_fail(SD_ERR_UNSUPPORTED, "too many output pixels");
  if (dtype == SD_BF16 && scratch) {
    const int ksplit = gemm_ksplit(a);
    if (ksplit > 1 && scratch_floats >= (int64_t)ksplit * a.M * a.N) {
      a.ksplit = ksplit;
      a.partial = scratch;
    }
  }
  return op_hip(launch_gemm((DType)dtype, a, (hipStream_t)stream), "conv");
}

sd_status synerdiff_op_upconv(int32_t dtype, const void* x, int32_t n, int32_t H, int32_t W, int32_t cin,
                              const void* w, int32_t cout, const float* bias, void* out, void* stream) {
  if (dtype != SD_BF16) return op_fail(SD_ERR_UNSUPPORTED, "upconv is bf16 only");
  if (!x || !w || !out) return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  if (n < 0 || H < 1 || W < 1 || cin < 32 || cin % 32 || cout < 160 || cout % 160)
    return op_fail(SD_ERR_INVALID_ARG, "bad shape (cin % 32, cout % 160)");
  if ((long)n * H * W > 0x7FFFFFFFL / 4) return op_fail(SD_ERR_UNSUPPORTED, "too many output pixels");
  if (n == 0) return SD_OK;
  for (int ph = 0; ph < 4; ++ph) {
    GemmArgs a;
    memset(&a, 0, sizeof(a));
    ASeg& s = a.seg[0];
    s.src0 = x; s.c0 = cin; s.cin = cin; s.ks = 2; s.stride = 1;
    s.Hi = H; s.Wi = W; s.Ho = H; s.Wo = W; s.K = 4 * cin;
    s.py = ph >> 1; s.px = ph & 1;
    a.M = n * H * W; a.N = cout; a.K = s.K; a.ldb = s.K;
    a.B = (const uint8_t*)w + (size_t)ph * cout * s.K * 2;
    a.ksplit = 1;
    a.epi.bias = bias; a.epi.out = out; a.epi.ldo = cout; a.epi.hw = 1;
    a.epi.phase = 1 + ph; a.epi.ph_h = H; a.epi.ph_w = W;
    const sd_status st = op_hip(launch_gemm(BF16, a, (hipStream_t)stream), "upconv");
    if (st != SD_OK) return st;
  }
  return SD_OK;
}

sd_status synerdiff_op_attention(int32_t dtype, const void* q, int64_t q_ld, int64_t q_img, const void* k,
                                 int64_t k_ld, int64_t k_img, const void* v, int64_t v_ld, int64_t v_img,
                                 int32_t v_transposed, const int32_t* kv_index, void* o, int64_t o_ld,
                                 int64_t o_img, int32_t n, int32_t heads, int32_t d, int32_t nq, int32_t nk,
                                 float scale, int32_t q_log2, void* stream) {
  if (bad_dtype(dtype)) return op_fail(SD_ERR_INVALID_ARG, "bad dtype");
  if (!q || !k || !v || !o) return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  if (n < 0 || heads < 1 || d < 8 || d % 8 || nq < 0 || nk < 1) return op_fail(SD_ERR_INVALID_ARG, "bad shape");
  if (dtype == SD_BF16 ? !attention_width_ok(d) : d > 256) return op_fail(SD_ERR_UNSUPPORTED, "unsupported head width");
  if ((v_transposed != 0) != (dtype == SD_BF16)) return op_fail(SD_ERR_UNSUPPORTED, "V is transposed for bf16 and only for bf16");
  if (n == 0 || nq == 0) return SD_OK;
  AttnArgs a;
  memset(&a, 0, sizeof(a));
  a.q = q; a.q_ld = q_ld; a.q_img = q_img;
  a.k = k; a.k_ld = k_ld; a.k_img = k_img;
  a.v = v; a.v_ld = v_ld; a.v_img = v_img; a.vt = v_transposed ? 1 : 0;
  a.kv_index = kv_index;
  a.o = o; a.o_ld = o_ld; a.o_img = o_img;
  a.imgs = n; a.heads = heads; a.d = d; a.Nq = nq; a.Nk = nk; a.scale = scale; a.q_log2 = q_log2 ? 1 : 0;
  return op_hip(launch_attention((DType)dtype, a, (hipStream_t)stream), "attention");
}

size_t synerdiff_op_groupnorm_scratch_floats(int32_t n, int32_t hw, int32_t cin) {
  if (n < 0 || hw < 1 || cin < 1) return 0;
  return groupnorm_partial_floats(n, hw, cin);
}

sd_status synerdiff_op_groupnorm_stats(int32_t dtype, const void* x0, int32_t c0, const void* x1, int32_t c1,
                                       int32_t n, int32_t hw, int32_t groups, float eps, const float* gamma,
                                       const float* beta, float* partial, float* scale, float* shift,
                                       void* stream) {
  if (bad_dtype(dtype)) return op_fail(SD_ERR_INVALID_ARG, "bad dtype");
  if (!x0 || (c1 && !x1) || !gamma || !beta || !partial || !scale || !shift)
    return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  const int cin = c0 + c1;
  if (n < 0 || hw < 1 || c0 < 8 || c0 % 8 || c1 < 0 || c1 % 8 || groups < 1 || cin % groups)
    return op_fail(SD_ERR_INVALID_ARG, "bad shape");
  if (cin > 4096) return op_fail(SD_ERR_UNSUPPORTED, "too many channels");
  if (n == 0) return SD_OK;
  return op_hip(launch_groupnorm_stats((DType)dtype, x0, c0, x1, c1, n, hw, groups, eps, gamma, beta, partial,
                                       scale, shift, (hipStream_t)stream),
                "groupnorm");
}

sd_status synerdiff_op_groupnorm_stats_noalloc(int32_t dtype, const void* x0, int32_t c0, const void* x1, int32_t c1,
                                               int32_t n, int32_t hw, int32_t groups, float eps, const float* gamma,
                                               const float* beta, float* scale, float* shift, void* stream) {
  if (bad_dtype(dtype)) return op_fail(SD_ERR_INVALID_ARG, "bad dtype");
  if (!x0 || (c1 && !x1) || !gamma || !beta || !scale || !shift) return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  const int cin = c0 + c1;
  if (n < 0 || hw < 1 || c0 < 8 || c0 % 8 || c1 < 0 || c1 % 8 || groups < 1 || cin % groups)
    return op_fail(SD_ERR_INVALID_ARG, "bad shape");
  if (cin > 4096) return op_fail(SD_ERR_UNSUPPORTED, "too many channels");
  if (n == 0) return SD_OK;
  const size_t need = groupnorm_partial_floats(n, hw, cin);
  if (need > groupnorm_scratch_floats_max()) {
    g_err = "groupnorm_stats_noalloc: " + std::to_string(need) + " partial floats exceed the library scratch of " +
            std::to_string(groupnorm_scratch_floats_max()) + " (use synerdiff_op_groupnorm_stats with a buffer)";
    return SD_ERR_CAPACITY;
  }
  float* part = nullptr;
  const sd_status st = op_hip(groupnorm_scratch(&part), "groupnorm scratch address");
  if (st != SD_OK) return st;
  return op_hip(launch_groupnorm_stats((DType)dtype, x0, c0, x1, c1, n, hw, groups, eps, gamma, beta, part, scale,
                                       shift, (hipStream_t)stream),
                "groupnorm_noalloc");
}

sd_status synerdiff_op_groupnorm_fused(int32_t dtype, const void* x0, int32_t c0, const void* x1, int32_t c1,
                                       int32_t n, int32_t hw, int32_t groups, float eps, const float* gamma,
                                       const float* beta, int32_t silu, void* out, void* stream) {
  if (dtype != SD_BF16) return op_fail(SD_ERR_UNSUPPORTED, "the one-kernel GroupNorm is bf16 only");
  const int cin = c0 + c1;
  if (n < 0 || hw < 1 || c0 < 4 || c1 < 0 || groups < 1 || cin % groups) return op_fail(SD_ERR_INVALID_ARG, "bad shape");
  if (!groupnorm_fused_ok(BF16, c0, c1, hw, groups) || n > 65535)
    return op_fail(SD_ERR_UNSUPPORTED, "shape outside the one-kernel GroupNorm's range");
  if (n == 0) return SD_OK;
  if (!x0 || (c1 && !x1) || !gamma || !beta || !out) return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  return op_hip(launch_groupnorm_fused(BF16, x0, c0, x1, c1, n, hw, groups, eps, gamma, beta, silu ? 1 : 0, out,
                                       (hipStream_t)stream),
                "groupnorm_fused");
}

sd_status synerdiff_op_layernorm(int32_t dtype, const void* x, void* y, int64_t tokens, int32_t C,
                                 const float* gamma, const float* beta, float eps, void* stream) {
  if (bad_dtype(dtype)) return op_fail(SD_ERR_INVALID_ARG, "bad dtype");
  if (!x || !y || !gamma || !beta) return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  if (tokens < 0 || C < 8 || C % 8 || C > 2048) return op_fail(SD_ERR_INVALID_ARG, "bad shape");
  return op_hip(launch_layernorm((DType)dtype, x, y, tokens, C, gamma, beta, eps, (hipStream_t)stream), "layernorm");
}

sd_status synerdiff_op_layernorm_rstd(int32_t dtype, const void* x, float* rstd, int64_t tokens, int32_t C,
                                      float eps, void* stream) {
  if (bad_dtype(dtype)) return op_fail(SD_ERR_INVALID_ARG, "bad dtype");
  if (tokens < 0 || C < 8 || C % 8 || C > 2048) return op_fail(SD_ERR_INVALID_ARG, "bad shape");
  if (tokens == 0) return SD_OK;
  if (!x || !rstd) return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  return op_hip(launch_layernorm_rstd((DType)dtype, x, rstd, tokens, C, eps, (hipStream_t)stream),
                "layernorm_rstd");
}

sd_status synerdiff_op_linear_rows(int32_t dtype, const float* in, int32_t M, int32_t K, const void* w,
                                   const float* bias, const float* add, float* out, int32_t N, int32_t silu_in,
                                   int32_t silu_out, void* stream) {
  if (bad_dtype(dtype)) return op_fail(SD_ERR_INVALID_ARG, "bad dtype");
  if (M < 0 || N < 0 || K <= 0 || K % 4) return op_fail(SD_ERR_INVALID_ARG, "bad shape");
  if (M == 0 || N == 0) return SD_OK;
  if (!in || !w || !out) return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  const auto al = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  if (!al(in) || !al(w) || !al(out) || (bias && !al(bias)) || (add && !al(add)))
    return op_fail(SD_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
  return op_hip(launch_linear_smallm((DType)dtype, in, M, K, w, bias, add, out, N, silu_in, silu_out,
                                     (hipStream_t)stream),
                "linear_rows");
}

sd_status synerdiff_op_geglu(int32_t dtype, const void* x, void* y, int64_t tokens, int32_t half, void* stream) {
  if (bad_dtype(dtype)) return op_fail(SD_ERR_INVALID_ARG, "bad dtype");
  if (!x || !y) return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  if (tokens < 0 || half < 8 || half % 8) return op_fail(SD_ERR_INVALID_ARG, "bad shape");
  return op_hip(launch_geglu((DType)dtype, x, y, tokens, half, (hipStream_t)stream), "geglu");
}

sd_status synerdiff_op_conv_out_cfg_ddim(int32_t dtype, const void* x, int32_t H, int32_t W, int32_t C,
                                         const void* w, const float* bias, int32_t n_req, const int32_t* req_row_u,
                                         const float* req_coef, const float* lat_in, float* lat_out, float* eps_out,
                                         void* stream) {
  if (dtype != SD_BF16) return op_fail(SD_ERR_UNSUPPORTED, "the fused output kernel is bf16 only");
  if (n_req < 0 || H < 1 || W < 1) return op_fail(SD_ERR_INVALID_ARG, "bad shape");
  if (!out_cfg_ddim_ok(BF16, 4, H, W, C)) return op_fail(SD_ERR_UNSUPPORTED, "unsupported shape (C % 32, C <= 320, W <= 128)");
  if (n_req == 0) return SD_OK;
  if (!x || !w || !bias || !req_row_u || !req_coef || !lat_in || !lat_out)
    return op_fail(SD_ERR_INVALID_ARG, "NULL argument");
  const size_t lat = (size_t)n_req * 4 * H * W * 4;
  const auto overlap = [](const void* a, const void* b, size_t n) {
    const uint8_t *pa = (const uint8_t*)a, *pb = (const uint8_t*)b;
    return pa < pb + n && pb < pa + n;
  };
  if (lat_out != lat_in && overlap(lat_out, lat_in, lat)) return op_fail(SD_ERR_INVALID_ARG, "latents overlap");
  if (eps_out && (overlap(eps_out, lat_in, lat) || overlap(eps_out, lat_out, lat)))
    return op_fail(SD_ERR_INVALID_ARG, "eps_out overlaps the latents");
  OutArgs a;
  memset(&a, 0, sizeof(a));
  a.x = (const bf16_t*)x;
  a.w = (const bf16_t*)w;
  a.bias = bias;
  a.lat_in = lat_in;
  a.lat_out = lat_out;
  a.eps_out = eps_out;
  a.req_row_u = req_row_u;
  a.req_coef = req_coef;
  a.order = nullptr;
  a.n_req = n_req;
  a.H = H;
  a.W = W;
  a.C = C;
  return op_hip(launch_out_cfg_ddim(a, (hipStream_t)stream), "conv_out_cfg_ddim");
}

}  // extern "C"
