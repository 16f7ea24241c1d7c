"""Brute-force references and small hand-built inputs for the test suite.

Everything here is plain Python over sets and lists, written from the
definitions of the method, independent of both the oracle and the HIP path.
"""
from __future__ import annotations

import itertools
import os
import subprocess
import tempfile

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def csr_from_edges(n, edges, bits=64):
    """CSR with rows ascending and each row's targets sorted (like synth)."""
    rows = [[] for _ in range(n)]
    for s, d in edges:
        rows[s].append(d)
    row_ptr = [0]
    col = []
    for r in rows:
        col.extend(sorted(r))
        row_ptr.append(len(col))
    dt = np.int64 if bits == 64 else np.int32
    return np.array(row_ptr, dtype=dt), np.array(col, dtype=np.int32)


def random_graph(n, m, rng, self_loops=True):
    edges = []
    for _ in range(m):
        s = int(rng.integers(0, n))
        d = int(rng.integers(0, n))
        if not self_loops and s == d:
            continue
        edges.append((s, d))
    return csr_from_edges(n, edges)


def neighbours(row_ptr, col_idx, u):
    return [int(x) for x in col_idx[row_ptr[u]:row_ptr[u + 1]]]


def bfs_ball(row_ptr, col_idx, seeds, hops):
    """Nodes within `hops` out-hops of the seeds."""
    ball = set(int(s) for s in seeds)
    front = set(ball)
    for _ in range(hops):
        nxt = set()
        for u in front:
            nxt.update(neighbours(row_ptr, col_idx, u))
        front = nxt - ball
        ball |= nxt
    return sorted(ball)


def is_subsequence_at_distinct_positions(sub, row):
    """True iff `sub` equals row[p0], row[p1], ... for some p0 < p1 < ..."""
    it = iter(row)
    return all(any(x == y for y in it) for x in sub)


def owner_of(kind, P, range_start, u):
    if kind == 0:
        return u % P
    for m in range(P):
        if range_start[m] <= u < range_start[m + 1]:
            return m
    raise ValueError(u)


def row_of(kind, P, range_start, u):
    if kind == 0:
        return u // P
    return u - range_start[owner_of(kind, P, range_start, u)]


def segments(ids, off, L, W):
    """ids of segment (l, b) as lists, level-major layout."""
    return [[list(map(int, ids[off[l * W + b]:off[l * W + b + 1]])) for b in range(W)]
            for l in range(L + 1)]


def floyd_sequences(d, k):
    """Every sequence of Floyd draws (t_0..t_{k-1}), t_i in [0, d-k+i]."""
    ranges = [range(0, d - k + i + 1) for i in range(k)]
    return itertools.product(*ranges)


_built = {}


def build_helper(src_name, extra=(), compiler="gcc", subdir="pins"):
    """Compiles a helper under tests/<subdir> into a temp dir (cached per
    session)."""
    if src_name in _built:
        return _built[src_name]
    out = os.path.join(tempfile.mkdtemp(prefix="ggpin_"), os.path.splitext(src_name)[0])
    cmd = [compiler, "-O2", os.path.join(ROOT, "tests", subdir, src_name), "-o", out, *extra]
    subprocess.run(cmd, check=True)
    _built[src_name] = out
    return out
