"""The seeded input generator: published SplitMix64 outputs, distribution
moments, determinism and workload recipes.  CPU only."""
import numpy as np

from fixtures import Stream, bf16_round, get_config, make_requests
from fixtures.rng import normal_many


def test_splitmix64_reference_sequence():
    # First outputs of SplitMix64 seeded with 1234567 (Vigna's reference
    # implementation); our counter form mix(key + (i + 1) * golden) equals it.
    s = Stream("any", 0)
    s.key = np.uint64(1234567)
    assert list(map(int, s.bits(0, 5))) == [6457827717110365317, 3203168211198807973,
                                            9817491932198370423, 4593380528125082431,
                                            16408922859458223821]


def test_normals_moments_and_chunk_independence():
    a = Stream("w", 0, "x").normal(2_000_001, dtype=np.float64)
    assert abs(a.mean()) < 3e-3 and abs(a.std() - 1) < 3e-3
    assert abs(((a ** 4).mean()) - 3.0) < 0.03  # Gaussian kurtosis
    b = normal_many([(Stream("w", 0, "x"), 2_000_001, None)], dtype=np.float64)[0]
    assert np.array_equal(a, b)


def test_bf16_round_ties_to_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -9], np.float32)
    y = bf16_round(x)
    assert list(y) == [1.0, 1.0, 1.0 + 2 ** -6, -2.5, 1.0]


def test_request_recipes():
    r = make_requests("c3_sd15_mixed32")
    assert r["cfg_on"].sum() == 16 and len(r["cfg_on"]) == 32
    assert r["latents"].shape == (32, 4, 64, 64) and r["ctx_cond"].shape == (32, 77, 768)
    assert ((r["guidance"] >= 5) & (r["guidance"] <= 9)).all()
    assert ((r["timesteps"] >= 0) & (r["timesteps"] <= 999)).all()
    assert np.array_equal(r["t_prev"], r["timesteps"] - 20)
    r1 = make_requests("c1_tiny_f32")
    assert list(r1["timesteps"]) == [999, 500] and list(r1["cfg_on"]) == [1, 0]
    assert get_config("c1_tiny_f32")["unet"]["schedule"] == "linear"
    r2 = make_requests("c3_sd15_mixed32")
    assert np.array_equal(r["latents"], r2["latents"])
