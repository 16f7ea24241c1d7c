"""Pins of the oracle's window pipeline against brute force and invariants.

Each check uses plain Python sets, BFS or direct indexing of the unsharded
feature matrix, never the oracle's own code paths.
"""
import collections
import json
import os

import numpy as np
import pytest

import synth
from oracle import ggref
from tests import helpers

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def make_world(row_ptr, col_idx, kind, P, local, row_bytes, stride, rng, range_start=None):
    """Partition book, random feature bytes and shards for a small graph."""
    N = row_ptr.shape[0] - 1
    if kind == ggref.PART_RANGE and range_start is None:
        range_start = [m * N // P for m in range(P)] + [N]
    part = ggref.make_part(P, kind, local, N, range_start)
    full = rng.integers(0, 256, size=(N, stride), dtype=np.uint8)
    rows = [[] for _ in range(P)]
    for u in range(N):
        rows[helpers.owner_of(kind, P, range_start, u)].append(u)
    shards = []
    for m in range(P):
        ids = sorted(rows[m], key=lambda u: helpers.row_of(kind, P, range_start, u))
        assert [helpers.row_of(kind, P, range_start, u) for u in ids] == list(range(len(ids)))
        shards.append(np.ascontiguousarray(full[ids]) if ids else np.zeros((0, stride), np.uint8))
    feat = ggref.make_feat(row_bytes, shards, [stride] * P)
    return part, feat, full, shards, range_start


def random_seeds(N, W, B, rng, ragged=True):
    sizes = [int(rng.integers(1, B + 1)) if ragged else B for _ in range(W)]
    seeds = np.concatenate([rng.integers(0, N, size=s) for s in sizes]).astype(np.int32)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    return seeds, off


GRAPHS = {
    "path": lambda rng: helpers.csr_from_edges(12, [(i, i + 1) for i in range(11)] +
                                               [(i + 1, i) for i in range(11)]),
    "star": lambda rng: helpers.csr_from_edges(101, [(0, i) for i in range(1, 101)] +
                                               [(i, 0) for i in range(1, 101)]),
    "complete8": lambda rng: helpers.csr_from_edges(8, [(i, j) for i in range(8) for j in range(8)
                                                        if i != j]),
    "loops_multi": lambda rng: helpers.csr_from_edges(
        20, [(i % 20, (i * 7) % 20) for i in range(300)] + [(i, i) for i in range(20)]),
    "isolated": lambda rng: helpers.csr_from_edges(30, [(0, 1), (1, 2), (2, 0)]),
    "random": lambda rng: helpers.random_graph(200, 3000, rng),
}


@pytest.mark.parametrize("gname", list(GRAPHS))
@pytest.mark.parametrize("fanout", [(3,), (4, 2), (5, 3, 2)])
def test_sampler_per_row_invariants_and_nested_frontiers(gname, fanout):
    rng = np.random.default_rng(7)
    row_ptr, col_idx = GRAPHS[gname](rng)
    N = row_ptr.shape[0] - 1
    W = 3
    seeds, soff = random_seeds(N, W, 6, rng)
    fids, foff, nids, noff = ggref.sample_window(row_ptr, col_idx, seeds, soff, fanout, 99, 2, 5)
    L = len(fanout)
    F = helpers.segments(fids, foff, L, W)
    for b in range(W):
        assert F[0][b] == sorted(set(seeds[soff[b]:soff[b + 1]].tolist()))
        for l in range(L):
            k = fanout[l]
            seg = nids[noff[l * W + b]:noff[l * W + b + 1]].tolist()
            assert len(seg) == k * len(F[l][b])
            sampled = set()
            for i, u in enumerate(F[l][b]):
                slot = seg[i * k:(i + 1) * k]
                row = helpers.neighbours(row_ptr, col_idx, u)
                cnt = min(len(row), k)
                assert all(v == -1 for v in slot[cnt:])
                got = slot[:cnt]
                assert all(v >= 0 for v in got)
                if len(row) <= k:
                    assert got == row                         # exact row copy
                else:
                    assert helpers.is_subsequence_at_distinct_positions(got, row)
                sampled.update(got)
            assert F[l + 1][b] == sorted(set(F[l][b]) | sampled)
    # strictly ascending segments
    for l in range(L + 1):
        for b in range(W):
            assert all(x < y for x, y in zip(F[l][b], F[l][b][1:]))


@pytest.mark.parametrize("gname", ["path", "random", "loops_multi", "star"])
def test_sampler_equals_bfs_ball_when_fanout_covers_every_degree(gname):
    rng = np.random.default_rng(3)
    row_ptr, col_idx = GRAPHS[gname](rng)
    N = row_ptr.shape[0] - 1
    maxdeg = int(np.diff(row_ptr).max())
    for L in (1, 2, 3):
        W = 2
        seeds, soff = random_seeds(N, W, 4, rng)
        fanout = [maxdeg + 1] * L
        fids, foff, _, _ = ggref.sample_window(row_ptr, col_idx, seeds, soff, fanout, 5, 0, 0)
        F = helpers.segments(fids, foff, L, W)
        for b in range(W):
            assert F[L][b] == helpers.bfs_ball(row_ptr, col_idx, seeds[soff[b]:soff[b + 1]], L)


@pytest.mark.parametrize("d,k", [(6, 3), (5, 4), (9, 2)])
def test_sampler_subsets_uniform_chi2(d, k):
    """The whole draw chain (Philox words, bounded map, Floyd) on one node of
    degree d > k: every k-subset of its neighbours is equally likely.
    20,000 batches, chi-square over the C(d, k) subsets."""
    import itertools
    row_ptr, col_idx = helpers.csr_from_edges(d + 1, [(0, i) for i in range(1, d + 1)])
    n_batches = 20000
    seeds = np.zeros(n_batches, dtype=np.int32)
    soff = np.arange(n_batches + 1, dtype=np.int64)
    _, _, nids, _ = ggref.sample_window(row_ptr, col_idx, seeds, soff, [k], 99, 0, 0)
    subsets = {c: i for i, c in enumerate(itertools.combinations(range(1, d + 1), k))}
    per = nids.reshape(n_batches, k)
    counts = np.zeros(len(subsets))
    for r in per.tolist():
        counts[subsets[tuple(r)]] += 1          # ascending and distinct, or KeyError
    expected = n_batches / len(subsets)
    chi2 = float(((counts - expected) ** 2 / expected).sum())
    # chi-square quantile 1 - 1e-6 for C(d, k) - 1 <= 35 degrees of freedom is below 90
    assert chi2 < 90.0, chi2
    # every position kept with probability k / d
    pos = np.bincount(per.ravel(), minlength=d + 1)[1:] / n_batches
    assert np.all(np.abs(pos - k / d) < 6 * np.sqrt(k / d * (1 - k / d) / n_batches)), pos


def test_sampler_star_leaves_uniform_chi2():
    # One hub with 100 leaves sampled at k = 10 across many batches: every
    # leaf must be kept with probability k / 100.
    row_ptr, col_idx = helpers.csr_from_edges(101, [(0, i) for i in range(1, 101)])
    n_batches, k = 2000, 10
    seeds = np.zeros(n_batches, dtype=np.int32)
    soff = np.arange(n_batches + 1, dtype=np.int64)
    _, _, nids, _ = ggref.sample_window(row_ptr, col_idx, seeds, soff, [k], 1234, 0, 0)
    counts = np.bincount(nids[nids >= 0], minlength=101)[1:]
    assert counts.sum() == n_batches * k
    expected = n_batches * k / 100.0
    chi2 = float(((counts - expected) ** 2 / expected).sum())
    # 99 degrees of freedom: the 0.999 quantile is about 148.2
    assert chi2 < 148.2, chi2
    # each batch keeps 10 distinct leaves
    per = nids.reshape(n_batches, k)
    assert all(len(set(r)) == k for r in per.tolist())


def test_sampler_batches_do_not_depend_on_window_size():
    # The counter is keyed by the global batch index, so N_b is identical
    # whichever window a batch falls in (the one-epoch trace fixes every
    # later access, Sec. IV-A).
    inst = synth.instance("tiny", with_features=False)
    wl = inst.wl
    seeds, boff = inst.seeds, inst.batch_off
    L = len(wl.fanout)
    ref = None
    for W in (1, 2, 4):
        got = []
        for k in range(synth.n_windows(boff, W)):
            b0, b1 = synth.window_batches(boff, W, k)
            so = boff[b0:b1 + 1] - boff[b0]
            fids, foff, _, _ = ggref.sample_window(inst.row_ptr, inst.col_idx,
                                                   seeds[boff[b0]:boff[b1]], so, wl.fanout, 0, 0,
                                                   b0)
            Wk = b1 - b0
            got += [fids[foff[L * Wk + b]:foff[L * Wk + b + 1]].tolist() for b in range(Wk)]
        if ref is None:
            ref = got
        assert got == ref


def test_sampler_epoch_and_seed_change_the_draws():
    inst = synth.instance("tiny", with_features=False)
    so = np.array([0, 256], dtype=np.int64)
    s = inst.seeds[:256]
    a = ggref.sample_window(inst.row_ptr, inst.col_idx, s, so, [10, 5], 0, 0, 0)[2]
    b = ggref.sample_window(inst.row_ptr, inst.col_idx, s, so, [10, 5], 0, 1, 0)[2]
    c = ggref.sample_window(inst.row_ptr, inst.col_idx, s, so, [10, 5], 1, 0, 0)[2]
    d = ggref.sample_window(inst.row_ptr, inst.col_idx, s, so, [10, 5], 0, 0, 0)[2]
    assert not np.array_equal(a[:1000], b[:1000])
    assert not np.array_equal(a[:1000], c[:1000])
    assert np.array_equal(a, d)


def _brute_hot(F, L, W, is_remote, n_hot):
    freq = collections.Counter()
    for b in range(W):
        for u in set(F[L][b]):
            if is_remote(u):
                freq[u] += 1
    items = sorted(freq.items())
    if 0 <= n_hot < len(items):
        items = sorted(items, key=lambda kv: (-kv[1], kv[0]))[:n_hot]
        items.sort()
    return [u for u, _ in items], [f for _, f in items]


@pytest.mark.parametrize("kind,local", [(0, 0), (1, 0), (1, 2), (0, -1)])
@pytest.mark.parametrize("n_hot", [-1, 0, 1, 7, 50, 10**6])
def test_hotset_matches_brute_force(kind, local, n_hot):
    rng = np.random.default_rng(11)
    row_ptr, col_idx = helpers.random_graph(300, 2500, rng)
    N = 300
    W, L = 5, 2
    seeds, soff = random_seeds(N, W, 8, rng)
    fids, foff, _, _ = ggref.sample_window(row_ptr, col_idx, seeds, soff, [4, 3], 3, 0, 0)
    rs = [0, 50, 120, 121, 300]
    part = ggref.make_part(4, kind, local, N, rs if kind == 1 else None)
    hot, freq = ggref.build_hotset(fids, foff, W, L, part, n_hot)
    F = helpers.segments(fids, foff, L, W)
    is_remote = lambda u: helpers.owner_of(kind, 4, rs, u) != local
    want_ids, want_freq = _brute_hot(F, L, W, is_remote, n_hot)
    assert hot.tolist() == want_ids
    assert freq.tolist() == want_freq
    if n_hot < 0:
        union = set()
        for b in range(W):
            union |= {u for u in F[L][b] if is_remote(u)}
        assert len(hot) == len(union)       # hot-set size equals the set union


@pytest.mark.parametrize("kind", [0, 1])
def test_bucket_is_a_stable_owner_partition(kind):
    rng = np.random.default_rng(5)
    N, P = 1000, 5
    rs = [0, 100, 100, 640, 700, 1000]
    part = ggref.make_part(P, kind, 0, N, rs if kind == 1 else None)
    hot = np.sort(rng.choice(N, size=400, replace=False)).astype(np.int32)
    bucket, off = ggref.bucket_by_owner(hot, part)
    assert off[0] == 0 and off[-1] == len(hot)
    assert sorted(bucket.tolist()) == hot.tolist()
    for m in range(P):
        seg = bucket[off[m]:off[m + 1]].tolist()
        want = [u for u in hot.tolist() if helpers.owner_of(kind, P, rs, u) == m]
        assert seg == want
    if kind == 1:
        assert bucket.tolist() == hot.tolist()   # ranges: already owner-major


def _window(row_ptr, col_idx, kind, local, W, fanout, rng, n_hot=-1, stride=48, row_bytes=44):
    N = row_ptr.shape[0] - 1
    part, feat, full, shards, rs = make_world(row_ptr, col_idx, kind, 4, local, row_bytes, stride,
                                              rng)
    seeds, soff = random_seeds(N, W, 10, rng)
    cache = np.zeros((N, stride), dtype=np.uint8)
    slot_of = np.full(N, -1, dtype=np.int32)
    res = ggref.run_window(row_ptr, col_idx, seeds, soff, fanout, 17, 0, 0, part, feat, cache,
                           stride, slot_of, None, n_hot)
    return res, part, feat, full, cache, slot_of, rs


@pytest.mark.parametrize("kind,local", [(0, 0), (1, 1), (0, -1)])
def test_stage_and_gather_against_the_unsharded_matrix(kind, local):
    rng = np.random.default_rng(21)
    row_ptr, col_idx = helpers.random_graph(400, 3000, rng)
    W, fanout = 4, (4, 3)
    res, part, feat, full, cache, slot_of, rs = _window(row_ptr, col_idx, kind, local, W, fanout,
                                                        rng)
    rb = feat.row_bytes
    hot = res["hot_ids"]
    bucket, off = res["bucket_ids"], res["owner_off"]
    # every cache row equals its source row; slot_of is a bijection H -> [0, |H|)
    for s, u in enumerate(bucket.tolist()):
        assert np.array_equal(cache[s, :rb], full[u, :rb])
        assert slot_of[u] == s
    assert sorted(np.nonzero(slot_of >= 0)[0].tolist()) == sorted(hot.tolist())
    st = res["stage_stats"]
    for m in range(4):
        n = int(off[m + 1] - off[m])
        assert st["requests"][m] == (1 if n else 0)       # at most one bulk request per owner
        assert st["rows"][m] == n and st["bytes"][m] == n * rb
        assert st["delta_rows"][m] == n                   # empty previous cache
    L = len(fanout)
    F = helpers.segments(res["frontier_ids"], res["frontier_off"], L, W)
    for b in range(W):
        ids = F[L][b]
        out = res["outs"][b]
        for i, u in enumerate(ids):
            assert np.array_equal(out[i, :rb], full[u, :rb])   # every gathered row is the source row
        gs = res["gather_stats"][b]
        remote = [u for u in ids if helpers.owner_of(kind, 4, rs, u) != local]
        assert gs["hits"] + gs["misses"] == len(remote)        # hits + misses = requests
        assert gs["local"] + gs["hits"] + gs["misses"] == len(ids) == gs["rows"]
        assert gs["misses"] == 0                               # union hot set covers the window


def test_zero_budget_is_pure_on_demand_fetch():
    rng = np.random.default_rng(8)
    row_ptr, col_idx = helpers.random_graph(300, 2000, rng)
    W, fanout = 3, (3, 3)
    res, part, feat, full, cache, slot_of, rs = _window(row_ptr, col_idx, 0, 0, W, fanout, rng,
                                                        n_hot=0)
    assert len(res["hot_ids"]) == 0 and res["stage_stats"]["requests_total"] == 0
    L = len(fanout)
    F = helpers.segments(res["frontier_ids"], res["frontier_off"], L, W)
    for b in range(W):
        ids = F[L][b]
        gs = res["gather_stats"][b]
        owners = [helpers.owner_of(0, 4, rs, u) for u in ids]
        remote = [u for u, m in zip(ids, owners) if m != 0]
        assert gs["hits"] == 0 and gs["misses"] == len(remote)
        for m in range(4):
            n_m = sum(1 for o in owners if o == m) if m != 0 else 0
            assert gs["miss_rows"][m] == n_m
            assert gs["miss_requests"][m] == (1 if n_m else 0)    # indicator of Eq. (2)
        rb = feat.row_bytes
        for i, u in enumerate(ids):
            assert np.array_equal(res["outs"][b][i, :rb], full[u, :rb])


def test_budget_between_misses_and_hits():
    rng = np.random.default_rng(9)
    row_ptr, col_idx = helpers.random_graph(300, 2000, rng)
    W, fanout = 4, (3, 3)
    res, part, feat, full, cache, slot_of, rs = _window(row_ptr, col_idx, 0, 0, W, fanout, rng,
                                                        n_hot=20)
    hot = set(res["hot_ids"].tolist())
    assert len(hot) == 20
    L = len(fanout)
    F = helpers.segments(res["frontier_ids"], res["frontier_off"], L, W)
    for b in range(W):
        ids = F[L][b]
        gs = res["gather_stats"][b]
        remote = [u for u in ids if u % 4 != 0]
        assert gs["hits"] == sum(1 for u in remote if u in hot)
        assert gs["misses"] == sum(1 for u in remote if u not in hot)   # M_b = N_b \ H_k
        rb = feat.row_bytes
        for i, u in enumerate(ids):
            assert np.array_equal(res["outs"][b][i, :rb], full[u, :rb])


def test_w1_degenerates_to_per_batch_fetch():
    rng = np.random.default_rng(31)
    row_ptr, col_idx = helpers.random_graph(500, 4000, rng)
    N = 500
    fanout = (4, 2)
    part, feat, full, shards, rs = make_world(row_ptr, col_idx, 0, 4, 0, 32, 32, rng)
    seeds, soff = random_seeds(N, 6, 8, rng)
    cache = np.zeros((N, 32), dtype=np.uint8)
    slot_of = np.full(N, -1, dtype=np.int32)
    prev = None
    total_bulk = 0
    for b in range(6):
        so = np.array([0, soff[b + 1] - soff[b]], dtype=np.int64)
        s = seeds[soff[b]:soff[b + 1]]
        win = ggref.run_window(row_ptr, col_idx, s, so, fanout, 4, 0, b, part, feat, cache, 32,
                               slot_of, prev)
        # on-demand reference: no cache at all
        ids = win["frontier_ids"][win["frontier_off"][2]:win["frontier_off"][3]]
        empty = np.full(N, -1, dtype=np.int32)
        out = np.zeros((len(ids), 32), dtype=np.uint8)
        od = ggref.gather_batch(ids, part, feat, cache[:0], 32, empty, out, 32)
        assert win["hot_ids"].tolist() == sorted(u for u in ids.tolist() if u % 4 != 0)
        assert win["stage_stats"]["rows"] == od["miss_rows"]
        assert win["stage_stats"]["requests"] == od["miss_requests"]
        assert np.array_equal(win["outs"][0], out)
        total_bulk += win["stage_stats"]["requests_total"]
        prev = win["bucket_ids"]
    assert total_bulk <= 6 * 3


def test_restaging_reports_the_rebuild_delta_and_clears_stale_slots():
    rng = np.random.default_rng(41)
    row_ptr, col_idx = helpers.random_graph(400, 3000, rng)
    N = 400
    part, feat, full, shards, rs = make_world(row_ptr, col_idx, 1, 4, 0, 16, 16, rng)
    cache = np.zeros((N, 16), dtype=np.uint8)
    slot_of = np.full(N, -1, dtype=np.int32)
    prev = None
    for k in range(4):
        seeds, soff = random_seeds(N, 3, 6, rng)
        win = ggref.run_window(row_ptr, col_idx, seeds, soff, (3, 2), 8, 0, 3 * k, part, feat,
                               cache, 16, slot_of, prev)
        hot = win["bucket_ids"].tolist()
        # slot_of holds exactly the current hot set (cache == H_k)
        assert sorted(np.nonzero(slot_of >= 0)[0].tolist()) == sorted(hot)
        prev_set = set() if prev is None else set(prev.tolist())
        off = win["owner_off"]
        for m in range(4):
            seg = hot[off[m]:off[m + 1]]
            assert win["stage_stats"]["delta_rows"][m] == len(set(seg) - prev_set)
        assert win["stage_stats"]["invalidated"] == len(prev_set)
        prev = win["bucket_ids"]


@pytest.mark.parametrize("kind,local", [(ggref.PART_RANGE, 0), (ggref.PART_MOD, -1)])
def test_delta_staging_requests_only_the_set_difference(kind, local):
    """Sec. IV-A, Eq. (1): with the previous cache as a source only
    Delta_{k,m} = (H_k in owner m) minus H_{k-1} is requested from owner m;
    rows already cached are copied from the previous cache.  Ground truth is
    the unsharded feature matrix and Python set algebra."""
    rng = np.random.default_rng(43)
    N = 500
    row_ptr, col_idx = helpers.random_graph(N, 4000, rng)
    part, feat, full, shards, rs = make_world(row_ptr, col_idx, kind, 4, local, 20, 32, rng)
    caches = [np.zeros((N, 32), dtype=np.uint8) for _ in range(2)]
    slot_of = np.full(N, -1, dtype=np.int32)
    prev = None
    for k in range(5):
        seeds, soff = random_seeds(N, 3, 5, rng)
        fids, foff, _, _ = ggref.sample_window(row_ptr, col_idx, seeds, soff, (3, 2), 5, 0, 3 * k)
        hot, _ = ggref.build_hotset(fids, foff, 3, 2, part, -1)
        bucket, owner_off = ggref.bucket_by_owner(hot, part)
        cache, src = caches[k % 2], (caches[(k - 1) % 2] if k else None)
        full_cache = np.zeros_like(cache)
        full_slot = slot_of.copy()
        ref = ggref.stage_bulk(bucket, owner_off, part, feat, full_cache, 32, full_slot, prev)
        st = ggref.stage_bulk(bucket, owner_off, part, feat, cache, 32, slot_of, prev,
                              src_cache=src, src_slot_of=slot_of if src is not None else None)
        prev_set = set() if prev is None else set(prev.tolist())
        H = bucket.tolist()
        for m in range(4):
            seg = H[owner_off[m]:owner_off[m + 1]]
            delta = set(seg) - prev_set
            assert st["rows"][m] == st["delta_rows"][m] == len(delta)
            assert st["requests"][m] == (1 if delta else 0)
            assert st["bytes"][m] == 20 * len(delta)
        assert st["retained"] == len(set(H) & prev_set)
        assert st["rows_total"] == len(H)
        # the cache holds the rows of H_k, equal to a full restage's cache
        for s_, u in enumerate(H):
            assert slot_of[u] == s_
            assert np.array_equal(cache[s_, :20], full[u, :20])
        assert np.array_equal(cache[:len(H), :20], full_cache[:len(H), :20])
        assert np.array_equal(slot_of, full_slot)
        assert ref["delta_rows"] == st["delta_rows"]
        prev = bucket


@pytest.mark.parametrize("kind,local", [(ggref.PART_MOD, 0), (ggref.PART_RANGE, 2),
                                        (ggref.PART_RANGE, -1)])
def test_inplace_staging_keeps_cached_rows_and_fills_lowest_free_slots(kind, local):
    """Algorithm 1 WarmCache(H_{k+1} minus C) on one persistent cache: a node
    the previous window cached keeps its slot and its bytes are not
    touched; only Delta_{k,m} = (H_k in owner m) minus H_{k-1} is requested,
    one request per owner with a non-empty delta, and the delta takes the
    lowest slots the previous window does not hold, in bucket order.  Ground
    truth: Python sets, sorted lists and the unsharded feature matrix."""
    rng = np.random.default_rng(47)
    N = 500
    row_ptr, col_idx = helpers.random_graph(N, 4000, rng)
    part, feat, full, shards, rs = make_world(row_ptr, col_idx, kind, 4, local, 20, 32, rng)
    cache_rows = N
    cache = np.zeros((cache_rows, 32), dtype=np.uint8)
    remaps = [np.full(N, -1, dtype=np.int32) for _ in range(2)]
    held = [None, None]                    # hot set each remap last held
    prev = None
    for k in range(6):
        seeds, soff = random_seeds(N, 3, 5, rng)
        fids, foff, _, _ = ggref.sample_window(row_ptr, col_idx, seeds, soff, (3, 2), 5, 0, 3 * k)
        hot, _ = ggref.build_hotset(fids, foff, 3, 2, part, -1)
        bucket, owner_off = ggref.bucket_by_owner(hot, part)
        cur, old = remaps[k % 2], (remaps[(k - 1) % 2] if k else None)
        before = cache.copy()
        old_map = None if old is None else old.copy()
        cleared = held[k % 2]
        st = ggref.stage_inplace(bucket, owner_off, part, feat, cache, 32, cur, old,
                                 clear_ids=cleared)
        held[k % 2] = bucket.copy()
        H = bucket.tolist()
        prev_set = set() if prev is None else set(prev)
        taken = set() if old_map is None else {int(x) for x in old_map if x >= 0}
        free = [x for x in range(cache_rows) if x not in taken]
        delta = [u for u in H if u not in prev_set]          # bucket order
        for j, u in enumerate(delta):
            assert cur[u] == free[j]
        for u in H:
            if u in prev_set:
                assert cur[u] == old_map[u]
                assert np.array_equal(cache[cur[u]], before[cur[u]])   # not rewritten
            assert np.array_equal(cache[cur[u], :20], full[u, :20])
        mask = np.ones(N, bool)
        mask[H] = False
        assert np.all(cur[mask] == -1)
        assert len({int(cur[u]) for u in H}) == len(H)
        for m in range(4):
            seg = set(H[owner_off[m]:owner_off[m + 1]]) - prev_set
            assert st["rows"][m] == st["delta_rows"][m] == len(seg)
            assert st["requests"][m] == (1 if seg else 0)
            assert st["bytes"][m] == 20 * len(seg)
        assert st["retained"] == len(set(H) & prev_set)
        assert st["rows_total"] == len(H)
        assert st["invalidated"] == (0 if cleared is None else len(cleared))
        if k == 0:                      # a first window takes slot = bucket position
            assert [int(cur[u]) for u in H] == list(range(len(H)))
        prev = H


def test_inplace_staging_capacity_is_the_union_of_two_windows():
    """The free slots run out exactly when the cache is smaller than the
    union of the previous and the current hot set."""
    rng = np.random.default_rng(53)
    N = 300
    row_ptr, col_idx = helpers.random_graph(N, 2000, rng)
    part, feat, full, shards, rs = make_world(row_ptr, col_idx, ggref.PART_MOD, 4, 0, 8, 8, rng)
    hs = []
    for k in range(2):
        seeds, soff = random_seeds(N, 2, 4, rng)
        fids, foff, _, _ = ggref.sample_window(row_ptr, col_idx, seeds, soff, (2, 2), 1, 0, 2 * k)
        hot, _ = ggref.build_hotset(fids, foff, 2, 2, part, -1)
        hs.append(ggref.bucket_by_owner(hot, part))
    union = len(set(hs[0][0].tolist()) | set(hs[1][0].tolist()))
    assert union > len(hs[1][0])
    for rows, ok in [(union, True), (union - 1, False)]:
        cache = np.zeros((rows, 8), dtype=np.uint8)
        r0, r1 = np.full(N, -1, np.int32), np.full(N, -1, np.int32)
        ggref.stage_inplace(hs[0][0], hs[0][1], part, feat, cache, 8, r0, None)
        if ok:
            ggref.stage_inplace(hs[1][0], hs[1][1], part, feat, cache, 8, r1, r0)
            assert max(int(r1[u]) for u in hs[1][0]) < rows
        else:
            with pytest.raises(ggref.OracleError, match="-2"):
                ggref.stage_inplace(hs[1][0], hs[1][1], part, feat, cache, 8, r1, r0)


def _expected_inplace(H, old_map, cache_rows):
    """Slots of the hot set H (bucket order) under in-place staging, from
    the definition: a node the previous remap holds keeps its slot; the
    delta takes, in bucket order, the ascending slots the previous remap
    does not hold; delta rows past the last free slot stay uncached (-1)."""
    taken = set() if old_map is None else {int(x) for x in old_map if x >= 0}
    free = [x for x in range(cache_rows) if x not in taken]
    want, j = {}, 0
    for u in H:
        if old_map is not None and old_map[u] >= 0:
            want[u] = int(old_map[u])
        elif j < len(free):
            want[u] = free[j]
            j += 1
        else:
            want[u] = -1
    return want


@pytest.mark.parametrize("short_by", [1, 7])
def test_inplace_staging_after_running_out_of_slots(short_by):
    """Reading R22: a cache smaller than the union of two windows' hot sets
    leaves the delta rows past the last free slot uncached (their remap
    entries -1, served as misses) and the call reports the shortfall; the
    next window then treats every slot the short window did fill as taken,
    so none of its delta rows lands on a row it keeps, and the nodes left
    out are part of its delta.  Three consecutive windows against the
    definition (Python sets and sorted lists) and the unsharded matrix."""
    rng = np.random.default_rng(59)
    N = 300
    row_ptr, col_idx = helpers.random_graph(N, 2000, rng)
    part, feat, full, shards, rs = make_world(row_ptr, col_idx, ggref.PART_MOD, 4, 0, 8, 16, rng)
    hs = []
    for k in range(3):
        seeds, soff = random_seeds(N, 2, 4, rng)
        fids, foff, _, _ = ggref.sample_window(row_ptr, col_idx, seeds, soff, (2, 2), 1, 0, 2 * k)
        hot, _ = ggref.build_hotset(fids, foff, 2, 2, part, -1)
        hs.append(ggref.bucket_by_owner(hot, part))
    union01 = len(set(hs[0][0].tolist()) | set(hs[1][0].tolist()))
    rows = union01 - short_by
    assert rows >= len(hs[0][0]) and rows >= len(hs[2][0])
    cache = np.zeros((rows, 16), dtype=np.uint8)
    remaps = [np.full(N, -1, np.int32), np.full(N, -1, np.int32)]
    held = [None, None]
    shorts = []
    for k in range(3):
        bucket, owner_off = hs[k]
        cur, old = remaps[k % 2], (remaps[(k - 1) % 2].copy() if k else None)
        before = cache.copy()
        H = bucket.tolist()
        want = _expected_inplace(H, old, rows)
        st, short = ggref.stage_inplace(bucket, owner_off, part, feat, cache, 16, cur, old,
                                        clear_ids=held[k % 2], allow_short=True)
        held[k % 2] = bucket.copy()
        shorts.append(short)
        assert short == (min(want.values()) < 0)
        for u in H:
            assert cur[u] == want[u], (k, u)
            if want[u] >= 0:
                assert np.array_equal(cache[want[u], :8], full[u, :8])
            if old is not None and old[u] >= 0:
                assert np.array_equal(cache[old[u]], before[old[u]])      # kept, not rewritten
        mask = np.ones(N, bool)
        mask[H] = False
        assert np.all(cur[mask] == -1)
        for m in range(4):
            seg = H[owner_off[m]:owner_off[m + 1]]
            delta = [u for u in seg if old is None or old[u] < 0]
            placed = [u for u in delta if want[u] >= 0]
            assert st["delta_rows"][m] == len(delta)
            assert st["rows"][m] == len(placed)
            assert st["bytes"][m] == 8 * len(placed)
            assert st["requests"][m] == (1 if placed else 0)
        assert st["retained"] == sum(1 for u in H if old is not None and old[u] >= 0)
        assert st["rows_total"] == len(H)
    assert shorts[0] is False and shorts[1] is True


def test_paper_consolidation_example():
    """Sec. IV-C: W = 16 batches over three remote owners turn up to
    16 x 3 = 48 per-batch requests into 3 bulk transfers."""
    with open(os.path.join(GOLDEN, "consolidation_w16.json")) as f:
        g = json.load(f)
    W, P = g["W"], g["num_parts"]
    # Complete graph on 8 nodes, owners by id mod 4: every batch's receptive
    # field reaches every owner.
    row_ptr, col_idx = helpers.csr_from_edges(8, [(i, j) for i in range(8) for j in range(8)
                                                  if i != j])
    rng = np.random.default_rng(0)
    part, feat, full, shards, rs = make_world(row_ptr, col_idx, 0, P, 0, 16, 16, rng)
    seeds = np.arange(W, dtype=np.int32) % 8
    soff = np.arange(W + 1, dtype=np.int64)
    cache = np.zeros((8, 16), dtype=np.uint8)
    slot_of = np.full(8, -1, dtype=np.int32)
    win = ggref.run_window(row_ptr, col_idx, seeds, soff, [7], 0, 0, 0, part, feat, cache, 16,
                           slot_of)
    nocache = ggref.run_window(row_ptr, col_idx, seeds, soff, [7], 0, 0, 0, part, feat,
                               np.zeros((8, 16), np.uint8), 16, np.full(8, -1, np.int32),
                               n_hot=0)
    per_batch = sum(sum(gs["miss_requests"]) for gs in nocache["gather_stats"])
    assert per_batch == g["per_batch_requests"]
    assert win["stage_stats"]["requests_total"] == g["bulk_requests"]
    assert sum(sum(gs["miss_requests"]) for gs in win["gather_stats"]) == 0


def test_oracle_reports_capacity_and_range_errors():
    row_ptr, col_idx = GRAPHS["path"](None)
    with pytest.raises(ggref.OracleError):
        ggref.sample_window(row_ptr, col_idx, np.array([12], np.int32),
                            np.array([0, 1], np.int64), [2], 0, 0, 0)
    with pytest.raises(ggref.OracleError):
        ggref.sample_window(row_ptr, col_idx, np.array([1], np.int32),
                            np.array([0, 1], np.int64), [2], 0, 0, 0, frontier_cap=1,
                            nbr_cap=100)
