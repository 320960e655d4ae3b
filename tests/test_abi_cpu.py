"""The C-ABI library on the CPU (no GPU work): it loads, exports every
declared entry point, and its host logic (manifest, row plan, schedules,
DDIM coefficients, argument validation) agrees with independent
definitions."""
import ctypes
import glob
import math
import os
import re

import numpy as np
import pytest

import oracle
from fixtures import CONFIGS, get_config, manifest as fixture_manifest

P = pytest.importorskip("paper_2605_08835_amd")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(P.binding.LIB_PATH):
        pytest.skip("libsynerdiff.so not built (run __graft_entry__.build())")
    return P.lib()


def declared_functions():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(synerdiff_\w+)\s*\(", src))
    return names


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 20
    for n in sorted(names):
        assert hasattr(lib, n), n
    assert lib.synerdiff_abi_version() == 1


@pytest.mark.parametrize("workload", sorted(CONFIGS))
def test_manifest_matches_the_generator(lib, workload):
    unet = get_config(workload)["unet"]
    cfg = P.config_from_dict(unet, 4)
    assert P.manifest(cfg) == [(n, tuple(s)) for n, s, _ in fixture_manifest(unet)]
    assert lib.synerdiff_weights_bytes(ctypes.byref(cfg)) > 0
    assert lib.synerdiff_workspace_bytes(ctypes.byref(cfg)) > 0


def test_row_plan_layout():
    rp = P.row_plan([1, 0, 1, 1, 0, 0, 1])
    n = 7
    assert rp["n_rows"] == n + 4
    assert list(rp["row_req"][:n]) == list(range(n)) and not rp["row_branch"][:n].any()
    assert list(rp["row_req"][n:]) == [0, 2, 3, 6] and rp["row_branch"][n:].all()
    assert list(rp["req_row_u"]) == [7, -1, 8, 9, -1, -1, 10]
    assert P.row_plan([])["n_rows"] == 0
    assert P.row_plan([0, 0])["n_rows"] == 2


@pytest.mark.parametrize("schedule", ["linear", "scaled_linear"])
def test_schedules_and_ddim_coefficients_match_the_oracle(schedule):
    ab = P.alphas_cumprod(schedule)
    ref = oracle.alphas_cumprod(oracle.betas(schedule))
    assert np.allclose(ab, ref, rtol=1e-13, atol=0)
    for t, tp in [(999, 979), (500, 480), (20, 0), (10, -10), (0, -20), (731, 711)]:
        A, B = P.ddim_coef(ab, t, tp)
        rA, rB = oracle.ddim_coefficients(oracle.sampler.abar_at(ref, t), oracle.sampler.abar_at(ref, tp))
        assert math.isclose(A, rA, rel_tol=1e-6) and math.isclose(B, rB, rel_tol=1e-6, abs_tol=1e-9)


def test_config_validation(lib):
    unet = dict(get_config("c3_sd15_mixed32")["unet"])
    assert lib.synerdiff_config_check(ctypes.byref(P.config_from_dict(unet, 32))) == 0
    bad = [dict(unet, heads=0, head_dim=0), dict(unet, ch=(320, 640, 1280, 1283)), dict(unet, latent_h=63),
           dict(unet, gn_groups=7), dict(unet, ctx_dim=77)]
    for b in bad:
        assert lib.synerdiff_config_check(ctypes.byref(P.config_from_dict(b, 32))) != 0
    assert lib.synerdiff_config_check(ctypes.byref(P.config_from_dict(unet, 0))) != 0
    assert lib.synerdiff_config_check(ctypes.byref(P.config_from_dict(dict(unet, dtype="f32"), 4))) != 0  # d=160


def _handle(lib, workload, R):
    unet = get_config(workload)["unet"]
    cfg = P.config_from_dict(unet, R)
    wb = lib.synerdiff_weights_bytes(ctypes.byref(cfg))
    sb = lib.synerdiff_workspace_bytes(ctypes.byref(cfg))
    h = ctypes.c_void_p()
    fake_w, fake_s = 1 << 40, 1 << 41  # never dereferenced by the validation paths
    assert lib.synerdiff_unet_create(ctypes.byref(cfg), fake_w, wb - 256, fake_s, sb, ctypes.byref(h)) == -4
    assert lib.synerdiff_unet_create(ctypes.byref(cfg), fake_w + 8, wb, fake_s, sb, ctypes.byref(h)) == -1
    assert lib.synerdiff_unet_create(ctypes.byref(cfg), fake_w, wb, fake_s, sb, ctypes.byref(h)) == 0
    return h


def test_step_argument_validation_happens_before_any_gpu_work(lib):
    """Every rejected call returns before enqueueing anything (no GPU here)."""
    h = _handle(lib, "c1_tiny_f32", 2)
    lat, out = 1 << 42, 1 << 43
    ctx, unc = 1 << 44, 1 << 45
    ts = np.array([999, 500], np.int32)
    cfg_on = np.array([1, 0], np.uint8)
    w = np.array([7.5, 7.5], np.float32)
    coef = np.ones((2, 2), np.float32)
    p = lambda a: a.ctypes.data

    def step(n=2, lat_=lat, ts_=ts, cfg_=cfg_on, w_=w, coef_=coef, out_=out, unc_=unc, eps=None, pooled=None):
        return lib.synerdiff_unet_step(h, n, lat_, p(ts_), p(cfg_), p(w_), ctx, unc_, pooled, None, None,
                                       p(coef_), out_, eps, None)

    assert step(n=0) == 0                                # empty batch: nothing to do
    assert step(n=3) == -3                               # over capacity
    assert step(n=-1) == -1
    assert step(ts_=np.array([1000, 5], np.int32)) == -1
    assert step(cfg_=np.array([2, 0], np.uint8)) == -1
    assert step(w_=np.array([np.nan, 1], np.float32)) == -1
    assert step(coef_=np.array([[np.inf, 1], [1, 1]], np.float32)) == -1
    assert step(out_=lat + 4) == -1                      # partial overlap with the input
    assert step(eps=lat) == -1                           # eps_out over the latents
    assert step(unc_=None) == -1                         # CFG row without a null context
    assert step(pooled=1 << 46) == -1                    # pooled input on a config without it
    assert step(lat_=None) == -1
    assert "overlap" in lib.synerdiff_last_error().decode() or lib.synerdiff_last_error()
    lib.synerdiff_unet_destroy(h)


def test_split_k_factor_depends_on_layer_shape_only(lib):
    """The K split of a convolution is a function of the layer (K, per-image
    size, width), never of the number of images, and linear (1x1) layers are
    not split; this is what keeps a request's bits independent of its
    batch-mates."""
    f = lib.synerdiff_op_conv_scratch_floats
    BF16 = 1
    for (c0, c1, H, W, ks, stride, up, cout) in [(640, 0, 4, 4, 3, 1, 0, 320), (1280, 0, 8, 8, 3, 1, 0, 1280),
                                                (1280, 1280, 8, 8, 3, 1, 0, 1280), (1280, 0, 16, 16, 3, 2, 0, 1280),
                                                (1280, 0, 8, 8, 3, 1, 1, 1280), (320, 0, 32, 32, 3, 1, 0, 320)]:
        Ho, Wo = (2 * H, 2 * W) if up else (H // stride, W // stride)
        ks_per_n = {f(BF16, c0, c1, n, H, W, ks, stride, up, cout) // (n * Ho * Wo * cout) for n in (1, 2, 3, 7, 48)}
        assert len(ks_per_n) == 1, (c0, H, ks_per_n)
    assert f(BF16, 640, 0, 1, 8, 8, 3, 1, 0, 640) // (64 * 640) == 4      # K = 5760 on 8x8: split in 4
    assert f(BF16, 640, 0, 1, 16, 16, 3, 1, 0, 640) // (256 * 640) == 2  # 16x16: split in 2
    assert f(BF16, 320, 0, 1, 32, 32, 3, 1, 0, 320) == 0                 # short K: no split
    for n in (1, 8, 64, 300):                                            # linear layers: rows as width
        assert f(BF16, 5120, 0, 1, 1, n, 1, 1, 0, 1280) == 0
    assert f(0, 640, 0, 1, 8, 8, 3, 1, 0, 640) == 0                      # fp32: no split
