"""Sequence planning of the inter-concurrency scheduler (Sec. III-D), plain
Python.

TEST INFRASTRUCTURE ONLY (see the package docstring).

A workload of M UNet tasks, N VAE tasks and at most K Skip-CFG-eligible
UNet tasks runs as a sequence of stages S = [(m_t, n_t, k_t)]: stage t runs
m_t UNet tasks, n_t VAE tasks and k_t Skip-CFG tasks concurrently, with
profiled round latency tau(m, n, k) and VAE latency delta(m, n, k) from the
offline lookup table (Sec. III-C).  Problem P (Eq. (3a)-(3f)) asks for the
sequence minimising the VAE tasks' completion times, V(t) = (sum of tau over
the stages before t) + delta(stage t), under: all tasks done (3c),
0 <= n_t, k_t <= m_t (3d), sum k_t <= K (3e) and total latency within the
throughput cap T_lim = (1 + alpha) tau(M, N, K) (3f).

Readings taken (the printed problem indexes stages from 0 in (3b) and (3f)
although they start at 1, and does not fix these points):
  * the objective is sum_t n_t V(t): the U_i and A_i terms of (3a) do not
    depend on how VAE tasks are placed, and this is the cost Alg. 1 adds up;
  * a stage runs at least one UNet task (m_t >= 1; (3d) then allows n_t and
    k_t up to m_t) and at most b_max (the lookup table's bound);
  * a path may end at any u <= K Skip-CFG tasks (Alg. 1 returns the best
    DP[M, N, u] over u).

`alg1` follows Alg. 1: one <cost, time> label per state (i, j, u), states
visited in lexicographic order (every action raises i, so this is a
topological order), actions (m, n, k) in lexicographic order, a label
replaced only by a strictly smaller cost, transitions whose time exceeds
T_lim pruned.  Because a state keeps one label, a cheaper label reached at a
later time can hide a path that ends cheaper; `exact` keeps every
non-dominated <cost, time> label per state instead and is the optimum of
Problem P, which `brute_force` checks by enumeration on tiny instances.
"""
INF = float("inf")


def actions(bmax):
    """Stage configurations (m, n, k): 1 <= m <= bmax, 0 <= n, k <= m."""
    return [(m, n, k) for m in range(1, bmax + 1) for n in range(m + 1) for k in range(m + 1)]


def objective(seq, tau, delta):
    """(sum_t n_t V(t), total latency) of a stage sequence."""
    t = 0.0
    cost = 0.0
    for (m, n, k) in seq:
        if n > 0:
            cost += n * (t + delta(m, n, k))
        t += tau(m, n, k)
    return cost, t


def alg1(M, N, K, tau, delta, T_lim, bmax):
    """Alg. 1: returns (sequence, cost, time) or (None, inf, inf)."""
    dp = {(0, 0, 0): (0.0, 0.0)}
    parent = {}
    acts = actions(bmax)
    for i in range(M + 1):
        for j in range(N + 1):
            for u in range(K + 1):
                if (i, j, u) not in dp:
                    continue
                c, t = dp[(i, j, u)]
                for (m, n, k) in acts:
                    if i + m > M or j + n > N or u + k > K:
                        continue
                    t_new = t + tau(m, n, k)
                    if t_new > T_lim:
                        continue
                    cv = (t + delta(m, n, k)) if n > 0 else 0.0
                    c_new = c + cv * n
                    nxt = (i + m, j + n, u + k)
                    if c_new < dp.get(nxt, (INF, 0.0))[0]:
                        dp[nxt] = (c_new, t_new)
                        parent[nxt] = ((i, j, u), (m, n, k))
    best = None
    for u in range(K + 1):
        if (M, N, u) in dp and (best is None or dp[(M, N, u)][0] < dp[best][0]):
            best = (M, N, u)
    if best is None:
        return None, INF, INF
    seq = []
    s = best
    while s != (0, 0, 0):
        s, a = parent[s]
        seq.append(a)
    seq.reverse()
    return seq, dp[best][0], dp[best][1]


def exact(M, N, K, tau, delta, T_lim, bmax):
    """Optimum of Problem P: per state the set of non-dominated (cost, time)
    labels (a label survives unless another has cost and time both <= and
    one strictly smaller).  Returns (cost, time) or (inf, inf)."""
    labels = {(0, 0, 0): [(0.0, 0.0)]}
    acts = actions(bmax)
    for i in range(M + 1):
        for j in range(N + 1):
            for u in range(K + 1):
                for (c, t) in labels.get((i, j, u), []):
                    for (m, n, k) in acts:
                        if i + m > M or j + n > N or u + k > K:
                            continue
                        t_new = t + tau(m, n, k)
                        if t_new > T_lim:
                            continue
                        c_new = c + ((t + delta(m, n, k)) * n if n > 0 else 0.0)
                        lst = labels.setdefault((i + m, j + n, u + k), [])
                        if any(c2 <= c_new and t2 <= t_new for (c2, t2) in lst):
                            continue
                        lst[:] = [(c2, t2) for (c2, t2) in lst if not (c_new <= c2 and t_new <= t2)]
                        lst.append((c_new, t_new))
    best = (INF, INF)
    for u in range(K + 1):
        for lab in labels.get((M, N, u), []):
            best = min(best, lab)
    return best


def brute_force(M, N, K, tau, delta, T_lim, bmax):
    """Enumerate every stage sequence that completes the workload (tiny
    instances only); returns the minimum (cost, time)."""
    acts = actions(bmax)
    best = (INF, INF)

    def rec(i, j, u, seq):
        nonlocal best
        if i == M and j == N:
            c, t = objective(seq, tau, delta)
            if t <= T_lim:
                best = min(best, (c, t))
            return
        for (m, n, k) in acts:
            if i + m <= M and j + n <= N and u + k <= K:
                seq.append((m, n, k))
                rec(i + m, j + n, u + k, seq)
                seq.pop()

    rec(0, 0, 0, [])
    return best


def lut_functions(tau_tab, delta_tab):
    """tau(m, n, k) and delta(m, n, k) from nested lists / arrays indexed [m][n][k]."""
    return (lambda m, n, k: float(tau_tab[m][n][k])), (lambda m, n, k: float(delta_tab[m][n][k]))
