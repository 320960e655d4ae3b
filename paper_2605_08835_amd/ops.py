"""Python wrappers of the kernel-level entry points (include/synerdiff_ops.h).
Tensors are torch device tensors; activations channels-last."""
import torch

from .binding import SD_BF16, SD_F32, _check, _ptr, lib


def _dt(t):
    if t.dtype == torch.bfloat16:
        return SD_BF16
    if t.dtype == torch.float32:
        return SD_F32
    raise TypeError(t.dtype)


def _s():
    return torch.cuda.current_stream().cuda_stream


def conv(x0, w_packed, cout, ks=3, stride=1, up=0, x1=None, scale=None, shift=None, silu=0, bias=None,
         resid=None, out=None, out_f32=False, split=True):
    n, H, W, c0 = x0.shape
    c1 = 0 if x1 is None else x1.shape[3]
    Ho, Wo = (2 * H, 2 * W) if up else (H // stride, W // stride)
    if out is None:
        out = torch.empty(n, Ho, Wo, cout, device=x0.device, dtype=torch.float32 if out_f32 else x0.dtype)
    nsc = lib().synerdiff_op_conv_scratch_floats(_dt(x0), c0, c1, n, H, W, ks, stride, up, cout) if split else 0
    scratch = torch.empty(nsc, device=x0.device) if nsc > 0 else None
    _check(lib().synerdiff_op_conv(_dt(x0), _ptr(x0), c0, _ptr(x1), c1, n, H, W, ks, stride, up, _ptr(scale),
                                   _ptr(shift), silu, _ptr(w_packed), cout, _ptr(bias), _ptr(resid), _ptr(out),
                                   int(out_f32), _ptr(scratch), nsc, _s()))
    return out


def attention(q, k, v, o, n, heads, d, n_q, n_k, q_ld, q_img, k_ld, k_img, v_ld, v_img, o_ld, o_img, scale,
              kv_index=None, v_transposed=False, q_log2=False):
    _check(lib().synerdiff_op_attention(_dt(q), _ptr(q), q_ld, q_img, _ptr(k), k_ld, k_img, _ptr(v), v_ld, v_img,
                                        int(v_transposed), _ptr(kv_index), _ptr(o), o_ld, o_img, n, heads, d, n_q,
                                        n_k, float(scale), int(q_log2), _s()))
    return o


def groupnorm_stats(x0, groups, eps, gamma, beta, x1=None):
    n, H, W, c0 = x0.shape
    c1 = 0 if x1 is None else x1.shape[3]
    cin = c0 + c1
    part = torch.empty(lib().synerdiff_op_groupnorm_scratch_floats(n, H * W, cin), device=x0.device)
    scale = torch.empty(n, cin, device=x0.device)
    shift = torch.empty(n, cin, device=x0.device)
    _check(lib().synerdiff_op_groupnorm_stats(_dt(x0), _ptr(x0), c0, _ptr(x1), c1, n, H * W, groups, float(eps),
                                              _ptr(gamma), _ptr(beta), _ptr(part), _ptr(scale), _ptr(shift), _s()))
    return scale, shift


def layernorm(x, gamma, beta, eps=1e-5):
    y = torch.empty_like(x)
    C = x.shape[-1]
    _check(lib().synerdiff_op_layernorm(_dt(x), _ptr(x), _ptr(y), x.numel() // C, C, _ptr(gamma), _ptr(beta),
                                        float(eps), _s()))
    return y


def layernorm_rstd(x, eps=1e-5):
    """fp32 [tokens] = 1 / sqrt(var + eps) of each row of x [tokens, C]."""
    C = x.shape[-1]
    rstd = torch.empty(x.numel() // C, device=x.device)
    _check(lib().synerdiff_op_layernorm_rstd(_dt(x), _ptr(x), _ptr(rstd), x.numel() // C, C, float(eps), _s()))
    return rstd


def upconv(x, w_phases, cout, bias=None):
    """Nearest-2x upsample + 3x3 conv of bf16 x [n, H, W, cin] as four phase
    convolutions; w_phases bf16 [4, cout, 4 * cin]."""
    n, H, W, cin = x.shape
    out = torch.empty(n, 2 * H, 2 * W, cout, device=x.device, dtype=x.dtype)
    _check(lib().synerdiff_op_upconv(_dt(x), _ptr(x), n, H, W, cin, _ptr(w_phases), cout, _ptr(bias), _ptr(out),
                                     _s()))
    return out


def linear_rows(x, w, bias=None, add=None, silu_in=0, silu_out=0):
    """x fp32 [M, K], w [N, K] (fp32 or bf16) -> fp32 [M, N]."""
    M, K = x.shape
    N = w.shape[0]
    y = torch.empty(M, N, device=x.device, dtype=torch.float32)
    _check(lib().synerdiff_op_linear_rows(_dt(w), _ptr(x), M, K, _ptr(w), _ptr(bias), _ptr(add), _ptr(y), N,
                                          int(silu_in), int(silu_out), _s()))
    return y


def geglu(x):
    half = x.shape[-1] // 2
    y = torch.empty(x.shape[:-1] + (half,), device=x.device, dtype=x.dtype)
    _check(lib().synerdiff_op_geglu(_dt(x), _ptr(x), _ptr(y), x.numel() // x.shape[-1], half, _s()))
    return y


def conv_out_cfg_ddim(x, w_packed, bias, req_row_u, req_coef, lat_in, lat_out=None, eps_out=None):
    """Output conv (3x3, C -> 4) + CFG combine + DDIM; x [rows, H, W, C] bf16,
    req_row_u int32 [n_req] and req_coef fp32 [n_req, 3] on the device."""
    n, H, W, C = x.shape
    n_req = int(req_row_u.shape[0])
    if lat_out is None:
        lat_out = torch.empty_like(lat_in)
    _check(lib().synerdiff_op_conv_out_cfg_ddim(_dt(x), _ptr(x), H, W, C, _ptr(w_packed), _ptr(bias), n_req,
                                                _ptr(req_row_u), _ptr(req_coef), _ptr(lat_in), _ptr(lat_out),
                                                _ptr(eps_out), _s()))
    return lat_out


def groupnorm_fused(x0, groups, eps, gamma, beta, x1=None, silu=True):
    """GroupNorm (+ SiLU) of [x0 | x1] in one kernel (bf16, small images)."""
    n, H, W, c0 = x0.shape
    c1 = 0 if x1 is None else x1.shape[3]
    out = torch.empty(n, H, W, c0 + c1, device=x0.device, dtype=x0.dtype)
    _check(lib().synerdiff_op_groupnorm_fused(_dt(x0), _ptr(x0), c0, _ptr(x1), c1, n, H * W, groups, float(eps),
                                              _ptr(gamma), _ptr(beta), int(silu), _ptr(out), _s()))
    return out


def groupnorm_stats_noalloc(x0, groups, eps, gamma, beta, x1=None, scale=None, shift=None):
    """GroupNorm statistics through the entry point that allocates nothing
    (the partial sums live in the library's own device array)."""
    n, H, W, c0 = x0.shape
    c1 = 0 if x1 is None else x1.shape[3]
    cin = c0 + c1
    scale = torch.empty(n, cin, device=x0.device) if scale is None else scale
    shift = torch.empty(n, cin, device=x0.device) if shift is None else shift
    _check(lib().synerdiff_op_groupnorm_stats_noalloc(_dt(x0), _ptr(x0), c0, _ptr(x1), c1, n, H * W, groups,
                                                      float(eps), _ptr(gamma), _ptr(beta), _ptr(scale),
                                                      _ptr(shift), _s()))
    return scale, shift
