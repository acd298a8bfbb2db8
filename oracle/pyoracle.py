"""Pure-Python twin of the C oracle — TEST INFRASTRUCTURE, tiny inputs only.

Written independently of ``bgmf_oracle.c`` (Python loops, numpy float32
scalars, one rounding per operation) so that the two can be checked against
each other bit for bit.  Follows the paper's Section 1: the block grid of
Eq. 4, the strata of Section 1.1, the per-rating update of Eq. 2-3 and the
whole-matrix RMSE of Algorithm 1's termination test.
"""
from __future__ import annotations

import math

import numpy as np

f32 = np.float32


def block_key(i: int, j: int, n: int, m: int, p: int):
    """(slot, row) sort key of a rating at (i, j) on the p x p grid."""
    R = (i * p) // n
    C = (j * p) // m
    s = (C - R) % p
    return s * p + R, i


def bucket(n, m, p, rows, cols):
    """Brute force: sort indices by (slot, row, index)."""
    nnz = len(rows)
    keys = [block_key(int(rows[e]), int(cols[e]), n, m, p) for e in range(nnz)]
    perm = sorted(range(nnz), key=lambda e: (keys[e][0], keys[e][1], e))
    block_ptr = [0] * (p * p + 1)
    for e in range(nnz):
        block_ptr[keys[e][0] + 1] += 1
    for q in range(p * p):
        block_ptr[q + 1] += block_ptr[q]
    return np.array(block_ptr, dtype=np.int64), np.array(perm, dtype=np.int32)


def sgd_update(u, v, x, alpha, beta):
    """One rating step, float32 scalars, returns new lists (old u in v's update)."""
    a, b, xx = f32(alpha), f32(beta), f32(x)
    acc = f32(0.0)
    for g in range(len(u)):
        acc = f32(acc + f32(f32(u[g]) * f32(v[g])))
    err = f32(xx - acc)
    nu, nv = list(u), list(v)
    for g in range(len(u)):
        uo, vo = f32(u[g]), f32(v[g])
        nu[g] = f32(uo + f32(a * f32(f32(err * vo) - f32(b * uo))))
        nv[g] = f32(vo + f32(a * f32(f32(err * uo) - f32(b * vo))))
    return nu, nv


def epoch(p, rows, cols, vals, block_ptr, perm, U, V, alpha, beta):
    """Blocked epoch on numpy float32 arrays, in place."""
    for s in range(p):
        for b in range(p):
            q = s * p + b
            for t in range(int(block_ptr[q]), int(block_ptr[q + 1])):
                e = int(perm[t])
                i, j = int(rows[e]), int(cols[e])
                nu, nv = sgd_update(list(U[i]), list(V[j]), vals[e], alpha, beta)
                U[i, :] = np.array(nu, dtype=np.float32)
                V[j, :] = np.array(nv, dtype=np.float32)


def rmse(rows, cols, vals, U, V):
    sq = 0.0
    for e in range(len(rows)):
        u, v = U[int(rows[e])], V[int(cols[e])]
        acc = f32(0.0)
        for g in range(len(u)):
            acc = f32(acc + f32(u[g] * v[g]))
        d = f32(f32(vals[e]) - acc)
        sq += float(d) * float(d)
    return math.sqrt(sq / len(rows)) if len(rows) else 0.0
