"""The load-adaptive feedback controller (Sec. III-D) on synthetic queue
traces: build-up first lowers the Skip-CFG point (raises the quality
threshold) down to its floor, then raises the VAE Chunking granularity up
to C_max; relief gives chunks back first, then restores the threshold; a
flat queue changes nothing."""
import pytest

from paper_2605_08835_amd.control import FeedbackController


def _drive(ctl, trace):
    out = []
    for q in trace:
        out.append(ctl.update(q))
    return out


def test_buildup_raises_skip_cfg_then_chunking():
    ctl = FeedbackController(skip_after=0.6, skip_floor=0.4, step=0.1, c0=1, c_max=3, window=4)
    _drive(ctl, [10 + 3 * i for i in range(200)])   # a queue that keeps growing
    assert ctl.skip_after == pytest.approx(0.4) and ctl.c == 3
    skips = [s for _, s, _ in ctl.log]
    cs = [c for _, _, c in ctl.log]
    # the threshold moves first (0.5, 0.4), the chunking only once it sits at the floor
    assert skips[:2] == [pytest.approx(0.5), pytest.approx(0.4)] and cs[:2] == [1, 1]
    assert cs[2:] == [2, 3] and all(s == pytest.approx(0.4) for s in skips[2:])


def test_relief_returns_chunks_first_then_fidelity():
    ctl = FeedbackController(skip_after=0.6, skip_floor=0.4, step=0.1, c0=1, c_max=3, window=4)
    _drive(ctl, [10 + 3 * i for i in range(200)])
    top = 10 + 3 * 199
    _drive(ctl, [max(top - 4 * i, 0) for i in range(400)])  # the queue drains, then stays empty
    assert ctl.c == 1 and ctl.skip_after == pytest.approx(0.6)
    after = ctl.log[4:]
    first_skip_change = next(i for i, (_, s, _) in enumerate(after) if s != pytest.approx(0.4))
    assert all(c == 1 for _, _, c in after[first_skip_change:])  # fidelity only after every chunk is back


def test_steady_queue_changes_nothing():
    ctl = FeedbackController()
    _drive(ctl, [7] * 300)
    assert ctl.log == [] and ctl.skip_after == 0.6 and ctl.c == 1


def test_bad_parameters_are_rejected():
    with pytest.raises(ValueError):
        FeedbackController(skip_after=0.3, skip_floor=0.5)
    with pytest.raises(ValueError):
        FeedbackController(c0=3, c_max=2)
