"""Host logic of the block-trace checker (paper_2304_13724_amd/trace.py) on
traces simulated here from the stratum schedule of Section 1.1: every block
starts when both its predecessors (its row-block's previous block, the
previous holder of its column-block) have ended, plus a latency.  The
checker must accept those, flag planted early starts by kind, skip
untraced blocks, and recover the critical path and the latency."""
import numpy as np
import pytest

from paper_2304_13724_amd import trace as T


def _simulate(p, seed, lat=3, per_stratum=False, heavy_col=None):
    rng = np.random.default_rng(seed)
    dur = rng.integers(5, 40, (p, p)).astype(np.int64)
    if heavy_col is not None:
        for s in range(p):
            dur[s, (heavy_col - s) % p] = 400  # block (b, s) with (b + s) mod p == heavy_col
    begin = np.zeros((p, p), np.int64)
    end = np.zeros((p, p), np.int64)
    for s in range(p):
        for b in range(p):
            if s == 0:
                begin[s, b] = 100 + rng.integers(0, 5)
            elif per_stratum:
                begin[s, b] = end[s - 1].max() + lat
            else:
                begin[s, b] = max(end[s - 1, b], end[s - 1, (b + 1) % p]) + lat
            end[s, b] = begin[s, b] + dur[s, b]
    return begin, end


@pytest.mark.parametrize("seed", range(3))
def test_simulated_schedules_pass(seed):
    b, e = _simulate(16, seed)
    assert T.violations(b, e) == []
    b, e = _simulate(16, seed, per_stratum=True)
    assert T.violations(b, e, per_stratum=True) == []


def test_planted_early_starts_are_flagged():
    p = 12
    b, e = _simulate(p, 7)
    # a block whose column-block's previous holder ended well after its own
    # row-block's previous block: start it just before that holder ended
    col_prev = np.roll(e[:-1], -1, axis=1)
    s, r = [(int(x) + 1, int(y)) for x, y in zip(*np.nonzero(col_prev - e[:-1] >= 2))][0]
    b[s, r] = col_prev[s - 1, r] - 1
    assert T.violations(b, e) == [(s, r, "column")]
    b2, e2 = _simulate(p, 8)
    b2[4, 2] = e2[3, 2] - 1  # before its own row-block's previous block ended
    assert (4, 2, "row") in T.violations(b2, e2)
    b3, e3 = _simulate(p, 9)
    e3[6, 0] = b3[6, 0] - 1  # ends before it begins
    assert (6, 0, "order") in T.violations(b3, e3)


def test_stratum_order_only_with_one_launch_per_stratum():
    p = 10
    b, e = _simulate(p, 3)  # neighbour-synchronised: strata overlap
    assert T.violations(b, e) == []
    kinds = {k for _, _, k in T.violations(b, e, per_stratum=True)}
    assert kinds == {"stratum"}


def test_untraced_blocks_are_skipped():
    p = 9
    b, e = _simulate(p, 4)
    b[5], e[5] = 0, 0  # a stratum the epoch did not visit
    b[2, 3], e[2, 3] = 0, 0
    assert T.violations(b, e) == []
    with pytest.raises(ValueError):
        T.critical_path(b, e)
    out = T.summary(b, e, 100_000_000)
    assert out["blocks"] == p * p - p - 1 and "critical_blocks" not in out


def test_critical_path_follows_the_heavy_column():
    p, heavy, lat = 16, 5, 3
    b, e = _simulate(p, 11, lat=lat, heavy_col=heavy)
    path, busy, wait = T.critical_path(b, e)
    assert len(path) == p and [s for s, _ in path] == list(range(p))
    s0, b0 = path[0]
    sl, bl = path[-1]
    assert busy + wait == e[sl, bl] - b[s0, b0]
    on_heavy = sum((bb + s) % p == heavy for s, bb in path)
    assert on_heavy == p
    assert busy == 400 * p and wait == lat * (p - 1)


def test_handover_gaps_are_the_latency():
    b, e = _simulate(16, 12, lat=7)
    g = T.handover_gaps(b, e)
    assert g.size > 0 and np.all(g == 7)
    out = T.summary(b, e, 100_000_000)
    assert out["handover_us_median"] == pytest.approx(0.07)
    assert out["critical_busy_us"] + out["critical_wait_us"] <= out["span_us"] + 1e-9


def test_degenerate_traces():
    z = np.zeros((3, 3), np.int64)
    assert T.violations(z, z) == [] and T.summary(z, z, 100_000_000) == {"span_us": 0.0, "blocks": 0}
    b, e = _simulate(1, 0)  # p = 1: one block, no hand-overs
    assert T.violations(b, e) == [] and T.handover_gaps(b, e).size == 0
    path, busy, wait = T.critical_path(b, e)
    assert path == [(0, 0)] and busy == e[0, 0] - b[0, 0] and wait == 0
