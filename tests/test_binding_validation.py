"""UNet.step() rejects, before any C-ABI call, device tensors and host
arrays that do not match the handle's configuration: the library receives
raw pointers and cannot check buffer sizes itself.  Runs on the CPU: the
binding object is built without a device handle, on the CPU device, so
every case fails in the Python checks."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
from fixtures import get_config  # noqa: E402
from paper_2605_08835_amd.binding import UNet  # noqa: E402


class _NoLib(UNet):
    def __init__(self, unet):  # no handle, no library call
        self.torch = torch
        self.unet = unet
        self.device = torch.device("cpu")
        self.act_dtype = torch.bfloat16 if unet["dtype"] == "bf16" else torch.float32
        self.h = None

    def close(self):
        pass


def _good(unet, n=3):
    L, D = unet["ctx_len"], unet["ctx_dim"]
    act = torch.bfloat16 if unet["dtype"] == "bf16" else torch.float32
    return dict(latents=torch.zeros(n, unet["latent_c"], unet["latent_h"], unet["latent_w"]),
                timesteps=np.full(n, 500, np.int32), cfg_on=np.ones(n, np.uint8),
                guidance=np.full(n, 7.5, np.float32), ctx_cond=torch.zeros(n, L, D, dtype=act),
                ctx_uncond=torch.zeros(L, D, dtype=act), coef=np.ones((n, 2), np.float32))


def _call(m, a, **over):
    a = dict(a, **over)
    return m.step(a.pop("latents"), a.pop("timesteps"), a.pop("cfg_on"), a.pop("guidance"), a.pop("ctx_cond"),
                  a.pop("ctx_uncond"), a.pop("coef"), **a)


def _bad_cases(unet):
    L, D = unet["ctx_len"], unet["ctx_dim"]
    H, W = unet["latent_h"], unet["latent_w"]
    act = torch.bfloat16 if unet["dtype"] == "bf16" else torch.float32
    other = torch.float32 if act == torch.bfloat16 else torch.bfloat16
    big = torch.zeros(3, 4, H, 2 * W)
    return {
        "latent dtype": dict(latents=torch.zeros(3, 4, H, W, dtype=torch.float64)),
        "latent size": dict(latents=torch.zeros(3, 4, H + 8, W)),
        "latent strided": dict(latents=big[..., ::2]),
        "latent not a tensor": dict(latents=np.zeros((3, 4, H, W), np.float32)),
        "short timesteps": dict(timesteps=np.zeros(2, np.int32)),
        "short cfg_on": dict(cfg_on=np.ones(2, np.uint8)),
        "short guidance": dict(guidance=np.ones(1, np.float32)),
        "short coef": dict(coef=np.ones((2, 2), np.float32)),
        "flat coef": dict(coef=np.ones(6, np.float32)),
        "ctx dtype": dict(ctx_cond=torch.zeros(3, L, D, dtype=other)),
        "ctx tokens": dict(ctx_cond=torch.zeros(3, L - 1, D, dtype=act)),
        "ctx count": dict(ctx_cond=torch.zeros(2, L, D, dtype=act)),
        "null ctx shape": dict(ctx_uncond=torch.zeros(L, D + 8, dtype=act)),
        "null ctx dtype": dict(ctx_uncond=torch.zeros(L, D, dtype=other)),
        "out shape": dict(out=torch.zeros(2, 4, H, W)),
        "eps_out dtype": dict(eps_out=torch.zeros(3, 4, H, W, dtype=torch.bfloat16)),
        "pooled without added embedding": dict(pooled_cond=torch.zeros(3, 1280)),
    }


@pytest.mark.parametrize("workload", ["c3_sd15_mixed32", "c1_tiny_f32"])
def test_step_rejects_mismatched_buffers(workload):
    unet = get_config(workload)["unet"]
    m = _NoLib(unet)
    good = _good(unet)
    for name, over in _bad_cases(unet).items():
        with pytest.raises(ValueError):
            _call(m, good, **over)
    with pytest.raises(ValueError, match="ctx_cond"):
        _call(m, good, ctx_cond=good["ctx_cond"][:2])


def test_step_checks_the_added_embedding():
    unet = get_config("c4_sdxl_cfg8")["unet"]
    m = _NoLib(unet)
    good = _good(unet, n=2)
    P = unet["pooled_dim"]
    ok = dict(pooled_cond=torch.zeros(2, P), pooled_uncond=torch.zeros(P), time_ids=np.zeros(6, np.float32))
    for over in [dict(ok, pooled_cond=torch.zeros(2, P - 1)), dict(ok, pooled_cond=None),
                 dict(ok, pooled_uncond=torch.zeros(P + 1)), dict(ok, time_ids=np.zeros(5, np.float32)),
                 dict(ok, time_ids=None)]:
        with pytest.raises(ValueError):
            _call(m, good, **over)


def test_rejections_happen_before_the_library_is_called(monkeypatch):
    import paper_2605_08835_amd.binding as b

    def boom():
        raise AssertionError("the C ABI was reached")

    monkeypatch.setattr(b, "lib", boom)
    unet = get_config("c3_sd15_mixed32")["unet"]
    m = _NoLib(unet)
    with pytest.raises(ValueError):
        _call(m, _good(unet), coef=np.ones((1, 2), np.float32))
