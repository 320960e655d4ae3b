"""Host logic of the offline profiler: the lookup table filled in from a
measured grid (multilinear in m, n and k / m) reproduces grid values exactly
and any function affine in each of those coordinates everywhere inside the
grid; n beyond the grid takes the largest measured n."""
import numpy as np
import pytest

from paper_2605_08835_amd.profiler import dense_table


def _grid(f, m_grid, n_grid, k_fracs):
    tau = [[[f(m, n, kf) for kf in k_fracs] for n in n_grid] for m in m_grid]
    return dict(m_grid=m_grid, n_grid=n_grid, k_fracs=k_fracs, tau=tau, delta=tau)


def test_affine_function_is_reproduced():
    f = lambda m, n, kf: 3.0 + 0.5 * m + 2.0 * n - 1.5 * kf  # noqa: E731
    g = _grid(f, [1, 4, 8], [0, 1, 3], [0.0, 0.5, 1.0])
    tau, delta = dense_table(g, 8)
    for m in range(1, 9):
        for n in range(0, min(m, 3) + 1):
            for k in range(m + 1):
                assert tau[m, n, k] == pytest.approx(f(m, n, k / m), abs=1e-12)
    assert np.array_equal(tau, delta)


def test_products_of_coordinates_are_reproduced():
    # multilinear interpolation is exact for m * n * (k / m) = n k as well
    f = lambda m, n, kf: m * n * kf  # noqa: E731
    g = _grid(f, [1, 2, 4, 8], [0, 2, 4], [0.0, 1.0])
    tau, _ = dense_table(g, 8)
    assert tau[3, 1, 2] == pytest.approx(2.0) and tau[6, 3, 3] == pytest.approx(9.0)


def test_clamping_outside_the_grid():
    f = lambda m, n, kf: 10.0 * m + n  # noqa: E731
    g = _grid(f, [2, 4], [0, 1], [0.0, 1.0])
    tau, _ = dense_table(g, 6)
    assert tau[1, 0, 0] == pytest.approx(20.0)      # m below the grid: the first m
    assert tau[6, 5, 2] == pytest.approx(41.0)      # m, n above: the last m, the last n
    assert tau[3, 1, 1] == pytest.approx(31.0)
