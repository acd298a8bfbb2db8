"""Checks and summaries of a block trace of one epoch (``bgmf_get_trace``).

The stratum schedule (Section 1.1, Algorithm 1's inner loop) orders the
blocks of an epoch in two ways.  A row-block's blocks run in stratum order,
so block (b, s) follows block (b, s - 1).  The column-block of block
(b, s), C = (b + s) mod p, was last updated in stratum s - 1 by row-block
b + 1 (mod p), so block (b, s) also follows block (b + 1, s - 1).  With one
launch per stratum every block of stratum s follows every block of stratum
s - 1.  A trace in which a block began before a predecessor handed its
results on shows a broken hand-over (a race on U or V rows).

Arrays are [p, p], indexed [s, b]; values are device clock ticks, and a
block no launch visited holds begin = end = 0.  Host logic only (numpy).
"""
from __future__ import annotations

import numpy as np


def _traced(begin: np.ndarray, end: np.ndarray) -> np.ndarray:
    return (begin != 0) | (end != 0)


def violations(begin: np.ndarray, end: np.ndarray, per_stratum: bool = False):
    """Blocks whose start precedes the hand-on of a predecessor.

    Returns a list of (s, b, kind) with kind one of "order" (begin after
    end), "row" (before block (b, s - 1) ended), "column" (before block
    (b + 1 mod p, s - 1) ended) or "stratum" (with one launch per stratum:
    before the last block of the previous traced stratum ended).  Only
    traced blocks are checked, each against its latest traced predecessor
    stratum.
    """
    begin = np.asarray(begin, dtype=np.int64)
    end = np.asarray(end, dtype=np.int64)
    p = begin.shape[0]
    seen = _traced(begin, end)
    out = [(int(s), int(b), "order") for s, b in zip(*np.nonzero(seen & (begin > end)))]
    row_end = np.zeros(p, dtype=np.int64)  # by row-block: end of its latest traced block
    have_row = np.zeros(p, dtype=bool)
    col_end = np.zeros(p, dtype=np.int64)  # by column-block: the same
    have_col = np.zeros(p, dtype=bool)
    stratum_end = None  # end of the latest traced stratum
    rows = np.arange(p)
    for s in range(p):
        cols = (rows + s) % p
        t = seen[s]
        checks = [("row", have_row & (begin[s] < row_end)),
                  ("column", have_col[cols] & (begin[s] < col_end[cols]))]
        if per_stratum and stratum_end is not None:
            checks.append(("stratum", begin[s] < stratum_end))
        for kind, bad in checks:
            out += [(s, int(b), kind) for b in np.nonzero(t & bad)[0]]
        if t.any():
            row_end[t] = end[s][t]
            have_row |= t
            col_end[cols[t]] = end[s][t]
            have_col[cols[t]] = True
            stratum_end = int(end[s][t].max())
    return out


def critical_path(begin: np.ndarray, end: np.ndarray):
    """The chain of blocks that set the epoch's length.

    Starts at the block that ended last and steps back, stratum by stratum,
    to whichever predecessor (same row-block, or the previous holder of the
    column-block) ended later.  Returns (path, busy, wait): path as a list
    of (s, b) from stratum 0 on, busy = the sum of end - begin over the
    path, wait = the sum of the gaps between a predecessor's end and the
    next block's begin (hand-over latency and, at the first block, nothing).
    Every block of the epoch must be traced.
    """
    begin = np.asarray(begin, dtype=np.int64)
    end = np.asarray(end, dtype=np.int64)
    p = begin.shape[0]
    if not _traced(begin, end).all():
        raise ValueError("critical_path needs a trace of every block")
    s, b = np.unravel_index(int(np.argmax(end)), end.shape)
    s, b = int(s), int(b)
    path = [(s, b)]
    busy = int(end[s, b] - begin[s, b])
    wait = 0
    while s > 0:
        cands = [(s - 1, b), (s - 1, (b + 1) % p)]
        ps, pb = max(cands, key=lambda x: end[x])
        wait += max(0, int(begin[s, b] - end[ps, pb]))
        s, b = ps, pb
        busy += int(end[s, b] - begin[s, b])
        path.append((s, b))
    path.reverse()
    return path, busy, wait


def handover_gaps(begin: np.ndarray, end: np.ndarray) -> np.ndarray:
    """For blocks of strata 1.. whose start was set by their column-block's
    previous holder (it ended after the row-block's own previous block):
    begin - that holder's end, in ticks.  A 1-D array."""
    begin = np.asarray(begin, dtype=np.int64)
    end = np.asarray(end, dtype=np.int64)
    col_prev = np.roll(end[:-1], -1, axis=1)  # end of block (b + 1, s - 1)
    row_prev = end[:-1]
    sel = col_prev > row_prev
    return (begin[1:] - col_prev)[sel]


def summary(begin: np.ndarray, end: np.ndarray, ticks_per_s: int) -> dict:
    """Epoch span, critical path (blocks, busy and waiting time) and the
    column hand-over latencies, in microseconds."""
    us = 1e6 / ticks_per_s
    seen = _traced(begin, end)
    if not seen.any():
        return {"span_us": 0.0, "blocks": 0}
    span = (end[seen].max() - begin[seen].min()) * us
    out = {"span_us": float(span), "blocks": int(seen.sum())}
    if seen.all():
        path, busy, wait = critical_path(begin, end)
        out.update(critical_blocks=len(path), critical_busy_us=busy * us,
                   critical_wait_us=wait * us)
    gaps = handover_gaps(begin, end) * us
    if gaps.size:
        out.update(handover_us_median=float(np.median(gaps)),
                   handover_us_p90=float(np.percentile(gaps, 90)),
                   handover_count=int(gaps.size))
    return out
