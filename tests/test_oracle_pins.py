"""Pins of the oracle's building blocks against things other than itself.

* Philox4x32-10 against PyTorch's independent header-only engine.
* The bounded map against its exact preimage counts (every value of [0, B)
  is hit floor(2^32/B) or ceil(2^32/B) times), by exhaustive enumeration.
* Floyd's k-of-d algorithm against brute-force enumeration of every draw
  sequence: each k-subset must come out exactly k! times.
"""
import collections
import itertools
import math
import os
import subprocess

import numpy as np
import pytest

from oracle import ggref
from tests import helpers


def _torch_include():
    import torch
    return os.path.join(os.path.dirname(torch.__file__), "include")


def test_philox_matches_independent_engine():
    exe = helpers.build_helper("philox_torch.cpp", extra=["-std=c++17", "-I" + _torch_include()],
                               compiler="g++")
    rng = np.random.default_rng(1234)
    cases = [(0, 0, 0, 0, 0, 0), (2**32 - 1,) * 6, (1, 2, 3, 4, 5, 6)]
    cases += [tuple(int(x) for x in rng.integers(0, 2**32, size=6, dtype=np.uint64))
              for _ in range(3000)]
    # The counter layout the sampler uses: (u, batch, epoch, (l << 16) | q).
    cases += [(u, b, e, (l << 16) | q, 0, 0) for u in (0, 7, 10**6) for b in (0, 3)
              for e in (0, 1) for l in (0, 2) for q in (0, 5)]
    inp = "\n".join(" ".join(str(v) for v in c) for c in cases) + "\n"
    res = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True)
    lines = res.stdout.strip().split("\n")
    assert len(lines) == len(cases)
    for c, line in zip(cases, lines):
        want = [int(x) for x in line.split()]
        got = ggref.philox(c[:4], c[4:]).tolist()
        assert got == want, (c, got, want)


@pytest.mark.parametrize("bound", [3, 7])
def test_bounded_map_preimage_counts_exhaustive(bound):
    exe = helpers.build_helper("bounded_count.c",
                               extra=["-fopenmp", "-L" + os.path.dirname(ggref.LIB_PATH),
                                      "-lggref",
                                      "-Wl,-rpath," + os.path.dirname(ggref.LIB_PATH)])
    out = subprocess.run([exe, str(bound)], capture_output=True, text=True, check=True)
    mn, mx, nv, mono, first, last, oor = (int(x) for x in out.stdout.split())
    assert oor == 0
    assert nv == bound
    assert mono == 1
    assert first == 0 and last == bound - 1
    assert mn in (2**32 // bound, -(-2**32 // bound))
    assert mx in (2**32 // bound, -(-2**32 // bound))
    assert mx - mn <= 1


def test_bounded_map_extremes():
    # r = 0 maps to 0 and r = 2^32 - 1 maps to bound - 1 for every bound.
    for bound in (1, 2, 10, 489, 10**6 + 3, 2**31, 2**32 - 1, 2**32):
        assert ggref.bounded(0, bound) == 0
        assert ggref.bounded(2**32 - 1, bound) == bound - 1
        # the midpoint word lands in the middle of the range
        assert ggref.bounded(2**31, bound) == bound // 2


@pytest.mark.parametrize("d,k", [(d, k) for d in range(2, 9) for k in range(1, min(d, 5))])
def test_floyd_uniform_over_all_draw_sequences(d, k):
    seen = collections.Counter()
    n_seq = 0
    for t in helpers.floyd_sequences(d, k):
        pos = ggref.floyd(d, k, list(t)).tolist()
        assert pos == sorted(pos)
        assert len(set(pos)) == k
        assert all(0 <= p < d for p in pos)
        seen[tuple(pos)] += 1
        n_seq += 1
    assert n_seq == math.perm(d, k)
    subsets = list(itertools.combinations(range(d), k))
    assert set(seen) == set(subsets)
    assert all(seen[s] == math.factorial(k) for s in subsets)


def test_floyd_rejects_bad_arguments():
    with pytest.raises(ggref.OracleError):
        ggref.floyd(3, 3, [0, 0, 0])       # needs d > k
    with pytest.raises(ggref.OracleError):
        ggref.floyd(5, 2, [4, 0])          # t_0 must lie in [0, d-k]


def test_owner_and_row_maps():
    p = ggref.make_part(4, ggref.PART_MOD, 0, 103)
    for u in range(103):
        assert ggref.owner(p, u) == u % 4 and ggref.row(p, u) == u // 4
    rs = [0, 10, 10, 60, 103]
    q = ggref.make_part(4, ggref.PART_RANGE, 0, 103, rs)
    for u in range(103):
        m = helpers.owner_of(1, 4, rs, u)
        assert ggref.owner(q, u) == m and ggref.row(q, u) == u - rs[m]
    assert m != 1  # the empty range owns nothing
