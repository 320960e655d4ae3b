"""The offline profiler (Sec. III-C) on the GPU with a small UNet and a
small VAE decoder: the chunking sweep's bookkeeping (chunk bounds, Eq. (1)
and (2) recomputed from its own per-round latencies, C_max and the chosen
c), the lookup grid, the planner on the interpolated table, and that running
the UNet step and the decoder chunks concurrently on two streams leaves both
results bit-identical to running them alone."""
import numpy as np
import pytest

from fixtures import get_config, make_requests, make_weights
from fixtures.vae import VAE_CONFIGS, make_vae_latents, make_vae_weights
from tests.gpu_util import log

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

WL, VN = "t_tiny_bf16", "vae_t16"


@pytest.fixture(scope="module")
def prof():
    from paper_2605_08835_amd import VAE, UNet
    from paper_2605_08835_amd.profiler import Profiler
    spec = get_config(WL)
    req = make_requests(WL)
    R = len(req["timesteps"])
    m = UNet(spec["unet"], max_requests=R)
    m.load_weights(make_weights(WL))
    act = m.act_dtype
    inputs = dict(latents=torch.from_numpy(req["latents"]).cuda(), timesteps=req["timesteps"],
                  cfg_on=req["cfg_on"], guidance=req["guidance"],
                  ctx_cond=torch.from_numpy(req["ctx_cond"]).cuda().to(act),
                  ctx_uncond=torch.from_numpy(req["ctx_uncond"]).cuda().to(act),
                  coef=m.coefficients(req["schedule"], req["timesteps"], req["t_prev"]))
    v = VAE(VAE_CONFIGS[VN]["vae"], max_images=2)
    v.load_weights(make_vae_weights(VN))
    z = torch.from_numpy(make_vae_latents(VN, 2)).cuda()
    yield Profiler(m, inputs, v, z), m, v, z, inputs
    m.close()
    v.close()


def test_chunking_sweep_bookkeeping(prof):
    from paper_2605_08835_amd import chunk_cost
    P, m, v, z, inputs = prof
    log(f"profiler chunking sweep: {WL} beside {VN}")
    ch = P.choose_chunking(c_limit=4, reps=1, overhead=-1.0)  # no early stop: every c up to 4
    ns = len(v.stages)
    assert ch["C_max"] == 4 and len(ch["rounds"]) == 4
    assert len(ch["stage_ms"]) == ns and all(t > 0 for t in ch["stage_ms"])
    for r in ch["rounds"]:
        c, b = r["c"], r["bounds"]
        assert len(b) == c + 1 and b[0] == 0 and b[-1] == ns and all(x < y for x, y in zip(b, b[1:]))
        assert len(r["t_u"]) == c and len(r["t_v"]) == c
        Tu, Tv, L = chunk_cost(r["t_u"], r["t_v"], r["T_u0"], r["T_v0"], ch["lam"])
        assert (Tu, Tv, L) == (r["T_u"], r["T_v"], r["L"])
        assert r["T_u0"] == pytest.approx(c * ch["t_u_solo"])
    assert ch["chosen_c"] == min(ch["rounds"], key=lambda r: r["L"])["c"]


def test_concurrent_rounds_leave_results_bit_identical(prof):
    P, m, v, z, inputs = prof
    ns = len(v.stages)
    # alone: one step and one plain decode on the current stream
    ref_out = m.step(inputs["latents"], inputs["timesteps"], inputs["cfg_on"], inputs["guidance"],
                     inputs["ctx_cond"], inputs["ctx_uncond"], inputs["coef"])
    ref_img = v.decode(z)
    torch.cuda.synchronize()
    ref_out, ref_img = ref_out.cpu().numpy(), ref_img.cpu().numpy()
    # concurrent: the decode in three chunks, each beside a full step
    P.out.zero_()
    P.img.zero_()
    torch.cuda.synchronize()
    P.rounds([0, ns // 3, 2 * ns // 3, ns])
    torch.cuda.synchronize()
    assert np.array_equal(P.out.cpu().numpy(), ref_out)
    assert np.array_equal(P.img.cpu().numpy(), ref_img)


def test_lookup_grid_and_planner(prof):
    from paper_2605_08835_amd import plan_sequence
    from paper_2605_08835_amd.profiler import dense_table
    P, m, v, z, inputs = prof
    R = len(inputs["timesteps"])
    g1 = P.lookup_grid(1, [1, R], [0, 2], reps=1)  # c = 1: the whole decode in one round
    assert np.all(np.array(g1["tau"]) > 0)
    g = P.lookup_grid(2, list(range(1, R + 1)), [0, 1, 2], reps=1)
    tau, delta = np.array(g["tau"]), np.array(g["delta"])
    assert tau.shape == (R, 3, 3) and np.all(tau > 0)
    assert np.all(delta[:, 0, :] == 0) and np.all(delta[:, 1:, :] > 0) and np.all(tau >= delta)
    T, D = dense_table(g, R)
    # grid points come back unchanged (k = f m lands on the grid for f = 0, 1)
    for a, mm in enumerate(g["m_grid"]):
        for b, n in enumerate(g["n_grid"]):
            if n <= mm:
                assert T[mm, n, 0] == pytest.approx(tau[a, b, 0]) and T[mm, n, mm] == pytest.approx(tau[a, b, 2])
    seq, cost, tm = plan_sequence(R, 2, 1, T, D, 1e9, exact=True)
    assert sum(s[0] for s in seq) == R and sum(s[1] for s in seq) == 2 and sum(s[2] for s in seq) <= 1
    assert cost > 0 and tm > 0


def test_saturation_batch(prof):
    P, m, v, z, inputs = prof
    R = len(inputs["timesteps"])
    bmax, thr = P.saturation_batch(list(range(1, R + 1)), reps=1)
    assert 1 <= bmax <= R and set(thr) == set(range(1, R + 1)) and all(t > 0 for t in thr.values())
