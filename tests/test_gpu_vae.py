"""VAE decoder on the GPU against the oracle (oracle/vae.py): whole decodes
on small latents, stage-by-stage parity of the SD decoder at its full size
(64x64 latents -> 512x512 images), chunked decoding (VAE Chunking) equal
to the one-call decode bit for bit, and batch independence."""
import numpy as np
import pytest

from fixtures.vae import VAE_CONFIGS, make_vae_latents, make_vae_weights
from oracle import vae as OV
from oracle.unet import Weights
from tests.gpu_util import log, rel_l2

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TOL = {"f32": 1e-4, "bf16": 3e-2}   # whole decode, relative L2 per image
TOL_STAGE = 2e-2                    # one bf16 stage on the GPU's own input

_CACHE = {}


def vae_for(name, max_images=None):
    from paper_2605_08835_amd import VAE
    key = (name, max_images)
    if key not in _CACHE:
        spec = VAE_CONFIGS[name]
        m = VAE(spec["vae"], max_images=max_images or spec["images"])
        m.load_weights(make_vae_weights(name))
        _CACHE[key] = m
    return _CACHE[key]


def _decode(m, z, bounds=None):
    lat = torch.from_numpy(np.ascontiguousarray(z)).cuda()
    n = len(m.stages)
    bounds = bounds or [0, n]
    img = torch.empty(m.image_shape(lat.shape[0]), device="cuda")
    for b, e in zip(bounds[:-1], bounds[1:]):
        m.run(lat, b, e, image=img)
    torch.cuda.synchronize()
    return img.cpu().double().numpy()


@pytest.mark.parametrize("name", ["vae_tiny_f32", "vae_t12x8"])
def test_decode_matches_the_oracle(name):
    spec = VAE_CONFIGS[name]
    vae = spec["vae"]
    m = vae_for(name)
    z = make_vae_latents(name)
    got = _decode(m, z)
    W = Weights(make_vae_weights(name))
    for i in range(len(z)):
        ref = OV.decode(vae, W, z[i])
        err = rel_l2(got[i], ref)
        log(f"  vae {name} image {i}: rel L2 {err:.3e}")
        assert np.isfinite(got[i]).all() and err <= TOL[vae["dtype"]], (i, err)


def test_chunked_decode_is_bitwise_the_plain_decode():
    m = vae_for("vae_t16")
    z = make_vae_latents("vae_t16")
    n = len(m.stages)
    full = _decode(m, z)
    from paper_2605_08835_amd import vae_chunk_plan
    for c in (2, 3, 7):
        bounds = vae_chunk_plan(m.stage_flops, c)
        assert np.array_equal(_decode(m, z, bounds), full), bounds
    assert np.array_equal(_decode(m, z, [0, 1, n - 1, n]), full)


def test_an_image_alone_equals_it_inside_the_batch():
    m = vae_for("vae_t16")
    z = make_vae_latents("vae_t16")
    both = _decode(m, z)
    one = _decode(m, z[1:2])
    assert np.array_equal(both[1], one[0])


def test_chunk_order_is_enforced():
    from paper_2605_08835_amd import SynerDiffError
    m = vae_for("vae_t16")
    lat = torch.from_numpy(make_vae_latents("vae_t16")).cuda()
    m.run(lat, 0, 3)
    with pytest.raises(SynerDiffError):
        m.run(lat, 5, 7)       # does not continue at stage 3
    with pytest.raises(SynerDiffError):
        m.run(lat[:1], 3, 5)   # a different batch size mid-decode
    m.run(lat, 0, len(m.stages))
    torch.cuda.synchronize()


@pytest.mark.timeout(1200)
def test_sd_decoder_full_size_stage_by_stage():
    """The SD decoder at 64x64 -> 512x512 (bf16): every stage run on the GPU
    alone, its output compared with the oracle's stage applied to the GPU's
    own input of that stage."""
    name = "vae_sd15"
    vae = VAE_CONFIGS[name]["vae"]
    m = vae_for(name)
    z = make_vae_latents(name)
    W = Weights(make_vae_weights(name))
    lat = torch.from_numpy(z).cuda()
    n = len(m.stages)
    img = torch.empty(m.image_shape(1), device="cuda")
    prev = None
    for i, st in enumerate(m.stages):
        m.run(lat, i, i + 1, image=img)
        torch.cuda.synchronize()
        got = img.cpu().double().numpy()[0] if i == n - 1 else m.activation(i, 1).float().cpu().double().numpy()[0]
        ref = OV.run_stage(vae, W, st, z[0] if i == 0 else prev)
        err = rel_l2(got, ref)
        log(f"  vae_sd15 stage {i} {st}: output {tuple(got.shape)}, rel L2 {err:.3e}")
        assert np.isfinite(got).all() and err <= TOL_STAGE, (st, err)
        prev = got
