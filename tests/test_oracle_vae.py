"""Pins of the VAE-decoder oracle (oracle/vae.py) and the decoder's host
logic in the C ABI (manifest, VAE Chunking's partition, Eq. (1)-(2)).

The paper prints no decoder value, so the oracle is pinned by: the public
parameter count of the autoencoder it belongs to (the decoder manifest plus
a shape walk of the published encoder gives SD's AutoencoderKL total of
83,653,863), by library routines (torch conv2d / interpolate /
scaled_dot_product_attention on the same weights), by special cases
(a zeroed conv2 makes a ResBlock the identity; a zeroed conv_out gives its
bias everywhere), and by chunked decoding equalling the plain one."""
import ctypes
import itertools
import math

import numpy as np
import pytest

from fixtures.vae import VAE_CONFIGS, make_vae_latents, make_vae_weights, vae_manifest, vae_param_count
from oracle import vae as OV
from oracle.unet import Weights

torch = pytest.importorskip("torch")
F = torch.nn.functional


def _encoder_param_count(ch=(128, 256, 512, 512), n_res=2, in_c=3, z=4):
    """Shape walk of the published KL-f8 encoder (conv_in; per level n_res
    ResBlocks and a stride-2 conv except at the last; mid ResBlock +
    attention + ResBlock; GroupNorm; conv_out to 2z moments; 1x1
    quant_conv): parameters only, nothing is built."""
    def res(ci, co):
        return 2 * ci + 9 * ci * co + co + 2 * co + 9 * co * co + co + ((ci * co + co) if ci != co else 0)
    n = 9 * in_c * ch[0] + ch[0]
    cur = ch[0]
    for i, c in enumerate(ch):
        for _ in range(n_res):
            n += res(cur, c)
            cur = c
        if i != len(ch) - 1:
            n += 9 * cur * cur + cur
    n += 2 * res(cur, cur) + 2 * cur + 4 * (cur * cur + cur)
    n += 2 * cur + 9 * cur * 2 * z + 2 * z
    n += (2 * z) * (2 * z) + 2 * z
    return n


def test_decoder_and_encoder_reproduce_the_public_autoencoder_count():
    vae = VAE_CONFIGS["vae_sd15"]["vae"]
    dec = vae_param_count(vae)
    assert dec == 49_490_199
    assert dec + _encoder_param_count() == 83_653_863


@pytest.fixture(scope="module")
def tiny():
    vae = VAE_CONFIGS["vae_tiny_f32"]["vae"]
    w = make_vae_weights("vae_tiny_f32")
    z = make_vae_latents("vae_tiny_f32")
    return vae, w, z


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float64))


def _torch_conv(x_hwc, w, b, up=False):
    x = _t(x_hwc).permute(2, 0, 1)[None]
    if up:
        x = F.interpolate(x, scale_factor=2, mode="nearest")
    return F.conv2d(x, _t(w), _t(b), padding=1)[0].permute(1, 2, 0).numpy()


def _torch_res(W, p, h, g):
    x = _t(h).permute(2, 0, 1)[None]
    u = F.silu(F.group_norm(x, g, _t(W(f"{p}.norm1.g")), _t(W(f"{p}.norm1.b")), 1e-6))
    u = F.conv2d(u, _t(W(f"{p}.conv1.w")), _t(W(f"{p}.conv1.b")), padding=1)
    u = F.silu(F.group_norm(u, g, _t(W(f"{p}.norm2.g")), _t(W(f"{p}.norm2.b")), 1e-6))
    u = F.conv2d(u, _t(W(f"{p}.conv2.w")), _t(W(f"{p}.conv2.b")), padding=1)
    if u.shape[1] != x.shape[1]:
        x = F.conv2d(x, _t(W(f"{p}.skip.w"))[:, :, None, None], _t(W(f"{p}.skip.b")))
    return (u + x)[0].permute(1, 2, 0).numpy()


def _torch_attn(W, h, g):
    H, Wd, C = h.shape
    x = _t(h).permute(2, 0, 1)[None]
    n = F.group_norm(x, g, _t(W("mid.attn.norm.g")), _t(W("mid.attn.norm.b")), 1e-6)[0].reshape(C, H * Wd).T
    q = F.linear(n, _t(W("mid.attn.q.w")), _t(W("mid.attn.q.b")))
    k = F.linear(n, _t(W("mid.attn.k.w")), _t(W("mid.attn.k.b")))
    v = F.linear(n, _t(W("mid.attn.v.w")), _t(W("mid.attn.v.b")))
    o = F.scaled_dot_product_attention(q[None], k[None], v[None])[0]
    o = F.linear(o, _t(W("mid.attn.o.w")), _t(W("mid.attn.o.b")))
    return h + o.numpy().reshape(H, Wd, C)


def test_every_stage_matches_torch_layers(tiny):
    vae, w, z = tiny
    W = Weights(w)
    g = vae["gn_groups"]
    h = None
    for name in OV.stages(vae):
        if name == "in":
            x = z[0].astype(np.float64).transpose(1, 2, 0) / vae["scaling"]
            pq = F.conv2d(_t(x).permute(2, 0, 1)[None], _t(W("post_quant.w"))[:, :, None, None], _t(W("post_quant.b")))
            ref = _torch_conv(pq[0].permute(1, 2, 0).numpy(), W("conv_in.w"), W("conv_in.b"))
            got = OV.run_stage(vae, W, name, z[0])
        elif name == "mid.attn":
            ref, got = _torch_attn(W, h, g), OV.run_stage(vae, W, name, h)
        elif name.endswith(".up"):
            ref, got = _torch_conv(h, W(f"{name}.w"), W(f"{name}.b"), up=True), OV.run_stage(vae, W, name, h)
        elif name == "out":
            x = F.silu(F.group_norm(_t(h).permute(2, 0, 1)[None], g, _t(W("out.norm.g")), _t(W("out.norm.b")), 1e-6))
            ref = F.conv2d(x, _t(W("out.conv.w")), _t(W("out.conv.b")), padding=1)[0].numpy()
            got = OV.run_stage(vae, W, name, h)
        else:
            ref, got = _torch_res(W, name, h, g), OV.run_stage(vae, W, name, h)
        assert got.shape == ref.shape, name
        assert np.allclose(got, ref, rtol=1e-10, atol=1e-10), name
        h = got
    assert W.used == set(w)
    assert h.shape == (vae["out_c"], 16, 16)


def test_zeroed_conv2_makes_a_resblock_the_identity(tiny):
    vae, w, z = tiny
    w2 = dict(w)
    w2["up0.res1.conv2.w"] = np.zeros_like(w["up0.res1.conv2.w"])
    w2["up0.res1.conv2.b"] = np.zeros_like(w["up0.res1.conv2.b"])
    W = Weights(w2)
    names = OV.stages(vae)
    i = names.index("up0.res1")
    h = OV.decode(vae, W, z[0], 0, i)
    assert np.array_equal(OV.run_stage(vae, W, "up0.res1", h), h)


def test_zeroed_conv_out_weights_give_the_bias(tiny):
    vae, w, z = tiny
    w2 = dict(w, **{"out.conv.w": np.zeros_like(w["out.conv.w"])})
    img = OV.decode(vae, Weights(w2), z[0])
    for c in range(vae["out_c"]):
        assert np.all(img[c] == np.float64(w["out.conv.b"][c]))


def test_chunked_decode_equals_the_plain_decode(tiny):
    vae, w, z = tiny
    W = Weights(w)
    full = OV.decode(vae, W, z[1])
    n = len(OV.stages(vae))
    for bounds in ([0, 5, n], [0, 1, 2, 9, n], [0, n - 1, n]):
        h = None
        for b, e in zip(bounds[:-1], bounds[1:]):
            h = OV.decode(vae, W, z[1], b, e, h)
        assert np.array_equal(h, full), bounds


def test_stage_list_is_resnet_block_level():
    vae = VAE_CONFIGS["vae_sd15"]["vae"]
    s = OV.stages(vae)
    assert s[:4] == ["in", "mid.res0", "mid.attn", "mid.res1"] and s[-1] == "out"
    assert sum(1 for x in s if ".res" in x) == 2 + 4 * 3 and sum(1 for x in s if x.endswith(".up")) == 3
    assert len(s) == 20


# ------------------------------------------------------------- host logic
P = pytest.importorskip("paper_2605_08835_amd")


@pytest.fixture(scope="module")
def lib():
    import os
    if not os.path.exists(P.binding.LIB_PATH):
        pytest.skip("libsynerdiff.so not built")
    return P.lib()


@pytest.mark.parametrize("name", sorted(VAE_CONFIGS))
def test_library_manifest_matches_the_generator(lib, name):
    vae = VAE_CONFIGS[name]["vae"]
    cfg = P.vae_config_from_dict(vae, 2)
    assert P.vae_manifest(cfg) == [(n, tuple(s)) for n, s, _ in vae_manifest(vae)]
    assert lib.synerdiff_vae_weights_bytes(ctypes.byref(cfg)) > 0
    assert lib.synerdiff_vae_workspace_bytes(ctypes.byref(cfg)) > 0


def test_vae_config_validation(lib):
    vae = VAE_CONFIGS["vae_sd15"]["vae"]
    assert lib.synerdiff_vae_config_check(ctypes.byref(P.vae_config_from_dict(vae, 1))) == 0
    for bad in [dict(vae, ch=(128, 256, 512, 500)), dict(vae, gn_groups=0), dict(vae, out_c=5),
                dict(vae, latent_h=128, latent_w=128), dict(vae, scaling=0.0)]:
        assert lib.synerdiff_vae_config_check(ctypes.byref(P.vae_config_from_dict(bad, 1))) != 0


def _brute_plan(cost, c):
    n = len(cost)
    best = None
    for cut in itertools.combinations(range(1, n), c - 1):
        b = [0, *cut, n]
        worst = max(sum(cost[b[i]:b[i + 1]]) for i in range(c))
        if best is None or worst < best[0] - 1e-12:
            best = (worst, b)
    return best


@pytest.mark.parametrize("seed", range(6))
def test_chunk_plan_is_the_minmax_partition(lib, seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(3, 9))
    cost = rng.uniform(0.1, 3.0, n).round(3)
    for c in range(1, n + 1):
        b = P.vae_chunk_plan(cost, c)
        assert b[0] == 0 and b[-1] == n and all(x < y for x, y in zip(b, b[1:]))
        worst = max(cost[b[i]:b[i + 1]].sum() for i in range(c))
        assert math.isclose(worst, _brute_plan(list(cost), c)[0], rel_tol=1e-12)


def test_chunk_cost_worked_example():
    # rounds (t_u, t_v) = (10, 8), (12, 11): T_u = 10 + 12 = 22; T_v = 10 + 11 = 21 (the VAE does not
    # wait for the UNet in the last round); L = 0.5 (22 - 20) / 20 + 0.5 (21 - 15) / 15 = 0.25
    Tu, Tv, L = P.chunk_cost([10, 12], [8, 11], 20.0, 15.0, 0.5)
    assert (Tu, Tv) == (22.0, 21.0) and math.isclose(L, 0.25)
    # one round: T_u = max(t_u, t_v), T_v = t_v
    Tu, Tv, L = P.chunk_cost([5.0], [9.0], 5.0, 9.0, 0.3)
    assert (Tu, Tv) == (9.0, 9.0) and math.isclose(L, 0.3 * 4 / 5)
