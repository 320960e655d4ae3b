"""Pins of the oracle's layer operations against brute force, closed forms
and independent library routines (torch CPU).  CPU only."""
import itertools
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as TF

from oracle import ops

rng = np.random.default_rng(7)


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x))


# ---- timestep embedding: closed forms ------------------------------------

@pytest.mark.parametrize("dim", [32, 256, 320])
def test_temb_t0_is_cos_then_sin(dim):
    e = ops.timestep_embedding(0, dim)
    h = dim // 2
    assert np.array_equal(e[:h], np.ones(h)) and np.array_equal(e[h:], np.zeros(h))


@pytest.mark.parametrize("dim", [32, 320])
def test_temb_pythagoras_pairs_cos_with_sin(dim):
    e = ops.timestep_embedding(777.25, dim)
    h = dim // 2
    assert np.allclose(e[:h] ** 2 + e[h:] ** 2, 1.0, atol=1e-14)


@pytest.mark.parametrize("dim", [32, 320])
def test_temb_frequencies_are_ten_thousand_to_minus_i_over_half(dim):
    # f_i = 10^(-4 i / h): at t = pi / f_i the cos entry is exactly -1 and the
    # sin entry 0.  Index h/2 (f = 1e-2) and h-1 separate i/h from i/(h-1).
    h = dim // 2
    for i in (0, h // 4, h // 2, h - 1):
        f = 10.0 ** (-4.0 * i / h)
        e = ops.timestep_embedding(math.pi / f, dim)
        assert abs(e[i] + 1.0) < 1e-9 and abs(e[h + i]) < 1e-8, i


# ---- element-wise functions ------------------------------------------------

def test_silu_gelu_against_torch_and_limits():
    x = np.linspace(-9, 9, 1001)
    assert np.allclose(ops.silu(x), TF.silu(_t(x)).numpy(), rtol=1e-13, atol=1e-15)
    assert np.allclose(ops.gelu(x), TF.gelu(_t(x)).numpy(), rtol=1e-13, atol=1e-15)
    assert ops.gelu(np.array(0.0)) == 0.0 and ops.silu(np.array(0.0)) == 0.0
    assert abs(ops.gelu(np.array(12.0)) - 12.0) < 1e-12
    assert abs(ops.gelu(np.array(1.0)) - 0.5 * (1 + math.erf(1 / math.sqrt(2)))) < 1e-15


# ---- convolution ----------------------------------------------------------

def _conv_brute(x, w, b, stride):
    H, W, cin = x.shape
    cout, _, k, _ = w.shape
    p = (k - 1) // 2
    Ho, Wo = (H + 2 * p - k) // stride + 1, (W + 2 * p - k) // stride + 1
    out = np.zeros((Ho, Wo, cout))
    for y, xx, o in itertools.product(range(Ho), range(Wo), range(cout)):
        s = b[o]
        for c, ky, kx in itertools.product(range(cin), range(k), range(k)):
            iy, ix = stride * y + ky - p, stride * xx + kx - p
            if 0 <= iy < H and 0 <= ix < W:
                s += x[iy, ix, c] * w[o, c, ky, kx]
        out[y, xx, o] = s
    return out


@pytest.mark.parametrize("H,W,cin,cout,k,stride", [(5, 4, 3, 2, 3, 1), (6, 7, 2, 3, 3, 2),
                                                   (3, 5, 4, 3, 1, 1), (5, 5, 1, 1, 3, 2)])
def test_conv_brute_force(H, W, cin, cout, k, stride):
    x = rng.standard_normal((H, W, cin))
    w = rng.standard_normal((cout, cin, k, k))
    b = rng.standard_normal(cout)
    assert np.allclose(ops.conv2d(x, w, b, stride), _conv_brute(x, w, b, stride), atol=1e-12)


@pytest.mark.parametrize("stride", [1, 2])
def test_conv_against_torch(stride):
    x = rng.standard_normal((13, 10, 16))
    w = rng.standard_normal((24, 16, 3, 3))
    b = rng.standard_normal(24)
    ref = TF.conv2d(_t(x.transpose(2, 0, 1))[None], _t(w), _t(b), stride=stride, padding=1)
    assert np.allclose(ops.conv2d(x, w, b, stride), ref[0].numpy().transpose(1, 2, 0), atol=1e-11)


def test_upsample_nearest():
    x = rng.standard_normal((3, 4, 2))
    up = ops.upsample_nearest2x(x)
    ref = TF.interpolate(_t(x.transpose(2, 0, 1))[None], scale_factor=2, mode="nearest")
    assert np.array_equal(up, ref[0].numpy().transpose(1, 2, 0))


# ---- normalisation -----------------------------------------------------------

@pytest.mark.parametrize("C,G,eps", [(32, 8, 1e-5), (64, 32, 1e-6), (60, 32 // 16, 1e-5)])
def test_group_norm_against_torch(C, G, eps):
    x = rng.standard_normal((7, 5, C)) * 3 + 1.5
    g, b = rng.standard_normal(C), rng.standard_normal(C)
    ref = TF.group_norm(_t(x.transpose(2, 0, 1))[None], G, _t(g), _t(b), eps)
    assert np.allclose(ops.group_norm(x, G, g, b, eps), ref[0].numpy().transpose(1, 2, 0), atol=1e-12)


def test_group_norm_special_cases():
    x = rng.standard_normal((4, 6, 12))
    g, b = rng.standard_normal(12), rng.standard_normal(12)
    inst = TF.instance_norm(_t(x.transpose(2, 0, 1))[None], weight=_t(g), bias=_t(b), eps=1e-5)
    assert np.allclose(ops.group_norm(x, 12, g, b, 1e-5), inst[0].numpy().transpose(1, 2, 0), atol=1e-12)
    const = np.full((4, 6, 12), 3.7)
    assert np.allclose(ops.group_norm(const, 4, g, b, 1e-5), np.broadcast_to(b, const.shape), atol=1e-12)
    # a group that straddles two concatenated sources equals GN of the concat
    a1, a2 = rng.standard_normal((4, 6, 6)), rng.standard_normal((4, 6, 6))
    cat = np.concatenate([a1, a2], axis=2)
    ref = TF.group_norm(_t(cat.transpose(2, 0, 1))[None], 4, _t(g), _t(b), 1e-5)
    assert np.allclose(ops.group_norm(cat, 4, g, b, 1e-5), ref[0].numpy().transpose(1, 2, 0), atol=1e-12)


def test_layer_norm_against_torch():
    x = rng.standard_normal((9, 40)) * 2 - 1
    g, b = rng.standard_normal(40), rng.standard_normal(40)
    ref = TF.layer_norm(_t(x), (40,), _t(g), _t(b), 1e-5)
    assert np.allclose(ops.layer_norm(x, g, b), ref.numpy(), atol=1e-12)


# ---- attention --------------------------------------------------------------

def _attn_brute(q, k, v, heads):
    Nq, C = q.shape
    d = C // heads
    out = np.zeros((Nq, C))
    for h in range(heads):
        for i in range(Nq):
            s = [sum(q[i, h * d + c] * k[j, h * d + c] for c in range(d)) / math.sqrt(d)
                 for j in range(k.shape[0])]
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = math.fsum(e)
            for c in range(d):
                out[i, h * d + c] = math.fsum(e[j] * v[j, h * d + c] for j in range(k.shape[0])) / z
    return out


@pytest.mark.parametrize("scale", [1.0, 30.0])
def test_attention_brute_force(scale):
    q = rng.standard_normal((5, 8)) * scale
    k = rng.standard_normal((7, 8)) * scale
    v = rng.standard_normal((7, 8))
    assert np.allclose(ops.attention(q, k, v, 2), _attn_brute(q, k, v, 2), atol=1e-12)


def test_attention_against_torch_sdpa():
    q, k, v = rng.standard_normal((33, 40)), rng.standard_normal((21, 40)), rng.standard_normal((21, 40))
    heads, d = 4, 10
    th = lambda a: _t(a.reshape(a.shape[0], heads, d).transpose(1, 0, 2))
    ref = TF.scaled_dot_product_attention(th(q), th(k), th(v))
    ref = ref.numpy().transpose(1, 0, 2).reshape(33, 40)
    assert np.allclose(ops.attention(q, k, v, heads), ref, atol=1e-12)


def test_attention_special_cases():
    q = rng.standard_normal((6, 12))
    v1 = rng.standard_normal((1, 12))
    assert np.allclose(ops.attention(q, rng.standard_normal((1, 12)), v1, 3), np.broadcast_to(v1, (6, 12)))
    kk = np.broadcast_to(rng.standard_normal((1, 12)), (5, 12))
    vv = rng.standard_normal((5, 12))
    assert np.allclose(ops.attention(q, kk, vv, 3), np.broadcast_to(vv.mean(0), (6, 12)), atol=1e-14)


def test_attention_sublayer_against_torch_mha():
    """Projection + head split + output projection as in the transformer's
    cross-attention equals torch's MultiheadAttention with the same weights
    (zero input-projection bias)."""
    C, D, heads = 24, 10, 4
    x, ctx = rng.standard_normal((9, C)), rng.standard_normal((6, D))
    wq, wk, wv = rng.standard_normal((C, C)), rng.standard_normal((C, D)), rng.standard_normal((C, D))
    wo, bo = rng.standard_normal((C, C)), rng.standard_normal(C)
    ours = ops.linear(ops.attention(ops.linear(x, wq), ops.linear(ctx, wk), ops.linear(ctx, wv), heads), wo, bo)
    mha = torch.nn.MultiheadAttention(C, heads, kdim=D, vdim=D, batch_first=True, dtype=torch.float64)
    with torch.no_grad():
        mha.q_proj_weight.copy_(_t(wq)); mha.k_proj_weight.copy_(_t(wk)); mha.v_proj_weight.copy_(_t(wv))
        mha.in_proj_bias.zero_()
        mha.out_proj.weight.copy_(_t(wo)); mha.out_proj.bias.copy_(_t(bo))
        ref, _ = mha(_t(x)[None], _t(ctx)[None], _t(ctx)[None], need_weights=False)
    assert np.allclose(ours, ref[0].numpy(), atol=1e-11)


def test_linear_against_torch():
    x, w, b = rng.standard_normal((3, 4, 7)), rng.standard_normal((5, 7)), rng.standard_normal(5)
    assert np.allclose(ops.linear(x, w, b), TF.linear(_t(x), _t(w), _t(b)).numpy(), atol=1e-13)
