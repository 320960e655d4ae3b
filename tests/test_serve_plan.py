"""Host bookkeeping of the continuous-batching loop (CPU only): per-request
timestep schedule, Skip-CFG window and retirement."""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")


class _FakeModel:
    unet = dict(latent_c=4, latent_h=2, latent_w=2, ctx_len=3, ctx_dim=8)
    act_dtype = torch.float32

    def __init__(self):
        self.calls = []

    def step(self, lat, t, cfg, w, ctx, null, coef, out=None, eps_out=None, stream=None):
        self.calls.append((np.array(t), np.array(cfg), np.array(coef)))
        return out


def test_schedule_skip_window_and_retirement():
    from paper_2605_08835_amd.serve import ContinuousBatcher
    m = _FakeModel()
    b = ContinuousBatcher(m, 4, "scaled_linear", 0.6, device="cpu")
    for rid, S in enumerate([20, 23, 50]):
        b.admit(rid, torch.zeros(4, 2, 2), torch.zeros(3, 8), S, 7.0)
    rows = {0: 0, 1: 0, 2: 0}
    ts = {0: [], 1: [], 2: []}
    done = []
    while b.n:
        ids = list(b.ids[:b.n])
        inp = b.step()
        for j, rid in enumerate(ids):
            rows[rid] += 1 + int(inp["cfg_on"][j])
            ts[rid].append(int(inp["t"][j]))
            assert 0 <= inp["t"][j] <= 999 and inp["t_prev"][j] == inp["t"][j] - 1000 // [20, 23, 50][rid]
        done += [r for r, _ in b.retire()]
    assert sorted(done) == [0, 1, 2]
    for rid, S in enumerate([20, 23, 50]):
        assert rows[rid] == S + math.ceil(0.6 * S)          # Skip-CFG for the last 40% of steps
        assert ts[rid][-1] == 0 and ts[rid] == sorted(ts[rid], reverse=True) and len(ts[rid]) == S
    # the final step of a request ends at x0 (abar_prev = 1)
    assert all(np.isfinite(c[2]).all() for c in m.calls)


def test_stage_assignment_covers_the_window():
    """Slots of a planned window (Problem P stages): stage t takes k_t
    requests past their threshold (run without CFG) and m_t - k_t others,
    under-threshold ones first."""
    from paper_2605_08835_amd.serve import assign_stages
    cfg = [1, 0, 1, 0, 1, 0]
    order, flags, bounds = assign_stages([(2, 1, 1), (4, 0, 1)], cfg)
    assert sorted(order) == list(range(6)) and bounds == [0, 2, 6]
    assert order[:2] == [1, 0] and flags[:2] == [0, 1]          # stage 1: one skip, one with CFG
    assert flags[2:].count(0) == 1 and cfg[order[2]] == 0        # stage 2: exactly one skip
    # a skip budget below the eligible count: the others run with CFG
    order, flags, bounds = assign_stages([(6, 0, 0)], cfg)
    assert flags == [1] * 6 and order[:3] == [0, 2, 4]
    import pytest
    with pytest.raises(ValueError):
        assign_stages([(3, 0, 0)], cfg)  # does not cover the window
