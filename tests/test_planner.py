"""The inter-concurrency scheduler's sequence planner (Sec. III-D, Problem P,
Alg. 1).  The oracle's exact dynamic program is pinned by brute-force
enumeration of every stage sequence on tiny workloads; the oracle's Alg. 1
by feasibility, its own cost recomputed from its sequence, and never beating
the optimum; the C-ABI planner (C++) must return exactly the oracle's
sequences and costs in both modes."""
import math

import numpy as np
import pytest

from oracle import planner as OP

P = pytest.importorskip("paper_2605_08835_amd")


def _lut(rng, bmax):
    """A random lookup table with the shape profiling gives: round latency
    growing sub-linearly in m (batching), plus VAE and Skip-CFG effects."""
    B = bmax + 1
    tau = np.zeros((B, B, B))
    delta = np.zeros((B, B, B))
    base_u, base_v = rng.uniform(20, 40), rng.uniform(50, 120)
    for m in range(1, B):
        for n in range(m + 1):
            for k in range(m + 1):
                u = base_u * (1 + 0.6 * (m - 1)) * (1 - 0.25 * k / m)  # Skip-CFG trims UNet work
                v = base_v * (1 + 0.8 * max(n - 1, 0)) if n else 0.0
                tau[m, n, k] = max(u, 0.7 * v) + 0.3 * min(u, v) + rng.uniform(0, 3)
                delta[m, n, k] = (v * (1 + 0.15 * m) + rng.uniform(0, 3)) if n else rng.uniform(0, 1)
    return tau, delta


def _instances(n, seed, small=True):
    rng = np.random.default_rng(seed)
    for _ in range(n):
        bmax = int(rng.integers(1, 4)) if small else int(rng.integers(2, 6))
        M = int(rng.integers(1, 5)) if small else int(rng.integers(3, 11))
        N = int(rng.integers(0, M + 1))
        K = int(rng.integers(0, M + 1))
        tau, delta = _lut(rng, bmax)
        tf, df = OP.lut_functions(tau, delta)
        # the throughput cap: (1 + alpha) x a max-batch schedule's latency, alpha = 10 % (Sec. IV-A),
        # sometimes tightened so that pruning matters
        full = 0.0
        left = M
        while left > 0:
            m = min(bmax, left)
            full += tau[m, min(m, N), min(m, K)]
            left -= m
        T_lim = (1.1 if rng.uniform() < 0.6 else rng.uniform(0.9, 1.5)) * full
        yield M, N, K, bmax, tau, delta, tf, df, T_lim


def test_exact_dp_equals_brute_force():
    checked = 0
    for M, N, K, bmax, tau, delta, tf, df, T_lim in _instances(60, 1):
        bf = OP.brute_force(M, N, K, tf, df, T_lim, bmax)
        ex = OP.exact(M, N, K, tf, df, T_lim, bmax)
        assert ex == bf, (M, N, K, bmax)
        checked += bf[0] < math.inf
    assert checked >= 30


def test_alg1_is_feasible_and_never_beats_the_optimum():
    worse = 0
    for M, N, K, bmax, tau, delta, tf, df, T_lim in _instances(80, 2):
        seq, c, t = OP.alg1(M, N, K, tf, df, T_lim, bmax)
        ex = OP.exact(M, N, K, tf, df, T_lim, bmax)
        if seq is None:  # every path Alg. 1 kept ran past T_lim (its one label per state may be the slower one)
            continue
        assert sum(s[0] for s in seq) == M and sum(s[1] for s in seq) == N and sum(s[2] for s in seq) <= K
        assert all(1 <= m <= bmax and 0 <= n <= m and 0 <= k <= m for m, n, k in seq)
        assert OP.objective(seq, tf, df) == (c, t) and t <= T_lim
        assert c >= ex[0]
        worse += c > ex[0]
    print(f"Alg. 1 above the optimum on {worse} of 80 instances")


def test_alg1_example_where_one_label_per_state_loses():
    """M = 3 UNet and N = 2 VAE tasks, no Skip-CFG, b_max = 2, with
    tau(1,0) = 3, tau(1,1) = 7, delta(1,1) = 3, tau(2,0) = 1, tau(2,1) = 2,
    delta(2,1) = 6, tau(2,2) = 4, delta(2,2) = 7.  State (2, 1, 0) is reached
    by (2,1) alone (cost 6 at time 2) or by (1,1),(1,0) (cost 3 at time 10);
    Alg. 1 keeps the cheaper label, which is late, and ends at cost 13
    ((1,1),(1,1),(1,0)), while (2,1),(1,1) costs 6 + (2 + 3) = 11 at time 9."""
    B = 3
    tau = np.full((B, B, B), 50.0)
    delta = np.full((B, B, B), 50.0)
    for (m, n), (t, d) in {(1, 0): (3, 4), (1, 1): (7, 3), (2, 0): (1, 6), (2, 1): (2, 6), (2, 2): (4, 7)}.items():
        tau[m, n, 0], delta[m, n, 0] = t, d
    tf, df = OP.lut_functions(tau, delta)
    seq, c, t = OP.alg1(3, 2, 0, tf, df, 1e9, 2)
    assert (seq, c, t) == ([(1, 1, 0), (1, 1, 0), (1, 0, 0)], 13.0, 17.0)
    assert OP.exact(3, 2, 0, tf, df, 1e9, 2) == OP.brute_force(3, 2, 0, tf, df, 1e9, 2) == (11.0, 9.0)
    assert P.plan_sequence(3, 2, 0, tau, delta, 1e9)[1:] == (13.0, 17.0)
    assert P.plan_sequence(3, 2, 0, tau, delta, 1e9, exact=True) == ([(2, 1, 0), (1, 1, 0)], 11.0, 9.0)


@pytest.mark.parametrize("exact", [False, True])
def test_library_planner_matches_the_oracle(exact):
    for M, N, K, bmax, tau, delta, tf, df, T_lim in _instances(40, 3 + exact, small=False):
        if exact:
            ref = OP.exact(M, N, K, tf, df, T_lim, bmax)
        else:
            rseq, rc, rt = OP.alg1(M, N, K, tf, df, T_lim, bmax)
            ref = (rc, rt)
        if ref[0] == math.inf:
            with pytest.raises(P.SynerDiffError):
                P.plan_sequence(M, N, K, tau, delta, T_lim, exact=exact)
            continue
        seq, c, t = P.plan_sequence(M, N, K, tau, delta, T_lim, exact=exact)
        assert (c, t) == ref, (M, N, K, bmax)
        assert OP.objective(seq, tf, df) == (c, t)
        if not exact:
            assert seq == rseq


def test_planner_argument_checks():
    tau = np.ones((3, 3, 3))
    with pytest.raises(P.SynerDiffError):
        P.plan_sequence(4, 2, 1, tau, tau, 0.5)      # nothing fits under the cap
    assert P.plan_sequence(0, 0, 0, tau, tau, 1.0)[0] == []
    bad = tau.copy()
    bad[1, 0, 0] = np.nan
    with pytest.raises(P.SynerDiffError):
        P.plan_sequence(2, 1, 0, bad, tau, 10.0)
