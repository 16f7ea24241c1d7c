"""Pins of the oracle's trace simulator (Sec. IV-A simulation; Sec. IV-B,
Eqs. (1)-(3)): hand-worked traces, special cases that reduce to plain
counting, the paper's consolidation example and brute force on tiny
traces."""
import json
import os

import numpy as np
import pytest

from oracle import ggref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

# Owners by id mod 4, owner 0 local.  Batches (N_b, ascending):
#   b0 = {1, 2, 3, 5}   remote owners: 1->1, 2->2, 3->3, 5->1
#   b1 = {2, 3, 6}      2->2, 3->3, 6->2
#   b2 = {1, 7}         1->1, 7->3
IDS = np.array([1, 2, 3, 5, 2, 3, 6, 1, 7], np.int32)
OFF = np.array([0, 4, 7, 9], np.int64)
PART = ggref.make_part(4, ggref.PART_MOD, 0, 16)
# eps_init 1, eps_row 0.01 per row, lam_init 1 ms, lam_row 10 us per row,
# 1 GB/s ceiling, 400-byte rows, 30 W idle.
COEF = ggref.sim_coeffs(4, 1.0, 0.01, 1e-3, 1e-5, 1e9, 400, 30.0)


def test_hand_worked_w1_union():
    # W = 1, union hot set: every window caches its whole remote set.
    #   k0: H = {1,2,3,5}, C = {}     -> Delta: owner1 {1,5}, owner2 {2}, owner3 {3}: 3 events, 4 rows
    #   k1: H = {2,3,6},   C = k0     -> Delta {6} (owner 2): 1 event, 1 row
    #   k2: H = {1,7},     C = k1     -> Delta {1} (owner 1), {7} (owner 3): 2 events, 2 rows
    # E_rebuild = 6 * 1 + 7 * 0.01 = 6.07.  Event durations (the slowest
    # owner; 4 rows at 1 GB/s take 1.6 us): 1.02 ms, 1.01 ms, 1.01 ms.
    a = ggref.simulate_epoch(IDS, OFF, 1, -1, PART, COEF)
    assert (a["windows"], a["batches"]) == (3, 3)
    assert (a["rebuild_events"], a["rebuild_rows"]) == (6, 7)
    assert (a["miss_events"], a["miss_rows"], a["remote_rows"], a["hits"]) == (0, 0, 9, 9)
    assert a["e_rebuild"] == pytest.approx(6.07, rel=1e-14)
    assert a["e_miss"] == 0.0
    assert a["t_stall"] == pytest.approx(3.04e-3, rel=1e-14)
    assert a["e_stall"] == pytest.approx(30 * 3.04e-3, rel=1e-14)
    assert a["e_phy"] == pytest.approx(6.07 + 30 * 3.04e-3, rel=1e-14)


def test_hand_worked_w2_budget_two():
    # W = 2, n_hot = 2.
    #   k0 = b0, b1: remote freq 1:1 2:2 3:2 5:1 6:1 -> H = {2, 3}
    #      Delta {2} (owner 2), {3} (owner 3): 2 events, 2 rows
    #      b0 misses {1, 5} (owner 1, 2 rows): 1 event; b1 misses {6} (owner 2): 1 event
    #   k1 = b2: freq 1:1 7:1 -> H = {1, 7}; Delta = {1, 7}: 2 events, 2 rows; no misses
    a = ggref.simulate_epoch(IDS, OFF, 2, 2, PART, COEF)
    assert (a["rebuild_events"], a["rebuild_rows"]) == (4, 4)
    assert (a["miss_events"], a["miss_rows"]) == (2, 3)
    assert (a["remote_rows"], a["hits"]) == (9, 6)
    assert a["e_rebuild"] == pytest.approx(4.04, rel=1e-14)
    assert a["e_miss"] == pytest.approx(2.03, rel=1e-14)
    # durations: 1.01 (k0 rebuild) + 1.02 (b0) + 1.01 (b1) + 1.01 (k1 rebuild) ms
    assert a["t_stall"] == pytest.approx(4.05e-3, rel=1e-14)
    assert a["e_phy"] == pytest.approx(4.04 + 2.03 + 30 * 4.05e-3, rel=1e-14)


def test_bandwidth_ceiling_decides_long_events():
    # A 400 B/s ceiling makes each row take 1 s at aggregate bandwidth, more
    # than any single owner's 0.5 s per row: every event lasts its total rows.
    c = ggref.sim_coeffs(4, 1.0, 0.01, 0.0, 0.5, 400.0, 400, 1.0)
    a = ggref.simulate_epoch(IDS, OFF, 1, -1, PART, c)
    assert a["t_stall"] == 7.0 and a["e_stall"] == 7.0
    # With no payload latency and an unlimited link, each event lasts one
    # initiation: three rebuild events (one per window).
    c = ggref.sim_coeffs(4, 1.0, 0.01, 1.0, 0.0, 1e300, 400, 2.0)
    a = ggref.simulate_epoch(IDS, OFF, 1, -1, PART, c)
    assert a["t_stall"] == 3.0 and a["e_stall"] == 6.0


def test_energy_terms_count_events_and_rows():
    for W in (1, 2, 3):
        for n_hot in (-1, 0, 1, 3):
            ev = ggref.simulate_epoch(IDS, OFF, W, n_hot, PART,
                                      ggref.sim_coeffs(4, 1.0, 0.0, 0.0, 0.0, 1.0, 0.0, 0.0))
            rows = ggref.simulate_epoch(IDS, OFF, W, n_hot, PART,
                                        ggref.sim_coeffs(4, 0.0, 1.0, 0.0, 0.0, 1.0, 0.0, 0.0))
            assert ev["e_rebuild"] == ev["rebuild_events"] and ev["e_miss"] == ev["miss_events"]
            assert rows["e_rebuild"] == rows["rebuild_rows"]
            assert rows["e_miss"] == rows["miss_rows"]
            assert ev["t_stall"] == 0.0 and ev["e_phy"] == ev["e_rebuild"] + ev["e_miss"]
            assert ev["hits"] + ev["miss_rows"] == ev["remote_rows"] == 9


def _random_trace(rng, N, n_batches, max_b):
    ids, off = [], [0]
    for _ in range(n_batches):
        nb = np.unique(rng.integers(0, N, size=rng.integers(0, max_b + 1)))
        ids.extend(nb.tolist())
        off.append(len(ids))
    return np.array(ids, np.int32), np.array(off, np.int64)


def _batch_sets(ids, off):
    return [set(ids[off[b]:off[b + 1]].tolist()) for b in range(len(off) - 1)]


@pytest.mark.parametrize("kind,local", [(ggref.PART_MOD, 0), (ggref.PART_RANGE, 2),
                                        (ggref.PART_MOD, -1)])
def test_zero_budget_is_pure_on_demand_fetch(kind, local):
    # n_hot = 0: nothing is cached, so there is no rebuild and every remote
    # (batch, owner) pair with a node is one on-demand request (the per-batch
    # fetch of the paper's baseline).
    rng = np.random.default_rng(1)
    N, P = 40, 4
    part = ggref.make_part(P, kind, local, N, [0, 7, 19, 30, 40] if kind == ggref.PART_RANGE else None)
    ids, off = _random_trace(rng, N, 11, 9)
    own = lambda u: ggref.owner(part, u)   # noqa: E731
    pairs = sum(len({own(u) for u in s if own(u) != local}) for s in _batch_sets(ids, off))
    remote = sum(sum(1 for u in s if own(u) != local) for s in _batch_sets(ids, off))
    for W in (1, 3, 11, 20):
        a = ggref.simulate_epoch(ids, off, W, 0, part, COEF)
        assert a["rebuild_events"] == 0 and a["rebuild_rows"] == 0 and a["e_rebuild"] == 0.0
        assert a["miss_events"] == pairs and a["miss_rows"] == remote and a["hits"] == 0


def test_union_hot_set_never_misses_and_w1_restages_each_batch():
    rng = np.random.default_rng(2)
    N = 64
    part = ggref.make_part(4, ggref.PART_MOD, 1, N)
    ids, off = _random_trace(rng, N, 9, 12)
    sets = _batch_sets(ids, off)
    own = lambda u: ggref.owner(part, u)   # noqa: E731
    for W in (1, 2, 4, 9):
        a = ggref.simulate_epoch(ids, off, W, -1, part, COEF)
        assert a["miss_events"] == 0 and a["hits"] == a["remote_rows"]
    # W = 1: the delta of batch b is its remote set minus batch b-1's.
    a = ggref.simulate_epoch(ids, off, 1, -1, part, COEF)
    prev, ev, rows = set(), 0, 0
    for s in sets:
        r = {u for u in s if own(u) != 1}
        d = r - prev
        ev += len({own(u) for u in d})
        rows += len(d)
        prev = r
    assert (a["rebuild_events"], a["rebuild_rows"]) == (ev, rows)
    # One window over the whole epoch: one bulk request per owner present.
    a = ggref.simulate_epoch(ids, off, 9, -1, part, COEF)
    allr = {u for s in sets for u in s if own(u) != 1}
    assert a["rebuild_events"] == len({own(u) for u in allr}) and a["rebuild_rows"] == len(allr)


def test_brute_force_budgets_on_tiny_traces():
    # Top-n_hot by (frequency desc, id asc), deltas against the previous
    # window's hot set and per-batch misses, counted with Python sets.
    rng = np.random.default_rng(3)
    N = 30
    part = ggref.make_part(3, ggref.PART_MOD, 0, N)
    own = lambda u: ggref.owner(part, u)   # noqa: E731
    for trial in range(20):
        ids, off = _random_trace(rng, N, int(rng.integers(1, 9)), 10)
        sets = _batch_sets(ids, off)
        for W in (1, 2, 3, 5):
            for n_hot in (0, 1, 2, 5, -1):
                prev = set()
                rb_ev = rb_rows = m_ev = m_rows = 0
                for k in range(0, len(sets), W):
                    win = sets[k:k + W]
                    freq = {}
                    for s in win:
                        for u in s:
                            if own(u) != 0:
                                freq[u] = freq.get(u, 0) + 1
                    order = sorted(freq, key=lambda u: (-freq[u], u))
                    hot = set(order if n_hot < 0 else order[:n_hot])
                    d = hot - prev
                    rb_ev += len({own(u) for u in d})
                    rb_rows += len(d)
                    for s in win:
                        m = {u for u in s if own(u) != 0} - hot
                        m_ev += len({own(u) for u in m})
                        m_rows += len(m)
                    prev = hot
                a = ggref.simulate_epoch(ids, off, W, n_hot, part, COEF)
                assert (a["rebuild_events"], a["rebuild_rows"], a["miss_events"],
                        a["miss_rows"]) == (rb_ev, rb_rows, m_ev, m_rows), (trial, W, n_hot)


def test_paper_consolidation_example_in_the_simulator():
    """Sec. IV-C: W = 16 batches over three remote owners: 48 per-batch
    requests, or 3 bulk transfers when the window is cached."""
    with open(os.path.join(GOLDEN, "consolidation_w16.json")) as f:
        g = json.load(f)
    W, P = g["W"], g["num_parts"]
    part = ggref.make_part(P, ggref.PART_MOD, 0, 64)
    rng = np.random.default_rng(4)
    ids, off = [], [0]
    for b in range(W):             # every batch reaches every owner
        s = sorted({int(x) for x in rng.integers(0, 64, 20)} | {4 * b % 64 + m for m in range(4)})
        ids += s
        off.append(len(ids))
    ids, off = np.array(ids, np.int32), np.array(off, np.int64)
    on_demand = ggref.simulate_epoch(ids, off, W, 0, part, COEF)
    windowed = ggref.simulate_epoch(ids, off, W, -1, part, COEF)
    assert on_demand["miss_events"] == g["per_batch_requests"]
    assert windowed["rebuild_events"] == g["bulk_requests"] and windowed["miss_events"] == 0
    # initiation paid 3 times instead of 48
    c = ggref.sim_coeffs(P, 1.0, 0.0, 0.0, 0.0, 1.0, 0.0, 0.0)
    assert ggref.simulate_epoch(ids, off, W, 0, part, c)["e_phy"] == 48.0
    assert ggref.simulate_epoch(ids, off, W, -1, part, c)["e_phy"] == 3.0


def test_simulator_rejects_bad_arguments():
    with pytest.raises(ggref.OracleError):
        ggref.simulate_epoch(IDS, OFF, 0, -1, PART, COEF)
    with pytest.raises(ggref.OracleError):
        ggref.simulate_epoch(IDS, OFF, 1, -1, PART,
                             ggref.sim_coeffs(4, 1.0, 0.0, 0.0, 0.0, 0.0, 400, 0.0))


def test_top_fraction_budget_hand_worked():
    # One window, owners by id mod 4, owner 0 local: b0 = {1,2,3}, b1 = {1,5},
    # b2 = {1,6}.  7 remote requests over U = 5 distinct nodes; freq(1) = 3,
    # every other node 1.
    ids = np.array([1, 2, 3, 1, 5, 1, 6], np.int32)
    off = np.array([0, 3, 5, 7], np.int64)
    # top 10%: ceil(0.5) = 1 node -> {1}, which serves 3 of the 7 requests
    a = ggref.simulate_epoch(ids, off, 3, -1, PART, COEF, hot_frac=(1, 10))
    assert (a["hits"], a["remote_rows"], a["rebuild_rows"], a["miss_rows"]) == (3, 7, 1, 4)
    # top 40%: exactly 2 nodes -> {1, 2} (ties by smaller id): 4 of 7
    a = ggref.simulate_epoch(ids, off, 3, -1, PART, COEF, hot_frac=(2, 5))
    assert (a["hits"], a["rebuild_rows"]) == (4, 2)
    hot, freq = ggref.build_hotset(ids, off, 3, 0, PART, -1, hot_frac=(2, 5))
    assert hot.tolist() == [1, 2] and freq.tolist() == [3, 1]
    # top 41%: ceil(2.05) = 3 nodes -> {1, 2, 3}
    hot, _ = ggref.build_hotset(ids, off, 3, 0, PART, -1, hot_frac=(41, 100))
    assert hot.tolist() == [1, 2, 3]
    # 0 and 1: nothing cached / the whole union
    assert ggref.simulate_epoch(ids, off, 3, -1, PART, COEF, hot_frac=(0, 7))["hits"] == 0
    assert ggref.simulate_epoch(ids, off, 3, -1, PART, COEF, hot_frac=(7, 7))["hits"] == 7


def test_top_fraction_budget_brute_force():
    rng = np.random.default_rng(5)
    N = 50
    part = ggref.make_part(4, ggref.PART_MOD, 2, N)
    own = lambda u: ggref.owner(part, u)   # noqa: E731
    for trial in range(15):
        ids, off = _random_trace(rng, N, int(rng.integers(1, 7)), 14)
        sets = _batch_sets(ids, off)
        for num, den in ((1, 10), (1, 4), (3, 7), (1, 1), (0, 3)):
            for W in (1, 2, 6):
                hits = remote = 0
                for k in range(0, len(sets), W):
                    win = sets[k:k + W]
                    freq = {}
                    for s in win:
                        for u in s:
                            if own(u) != 2:
                                freq[u] = freq.get(u, 0) + 1
                    n = -(-len(freq) * num // den)          # ceil(U * num / den)
                    hot = set(sorted(freq, key=lambda u: (-freq[u], u))[:n])
                    for s in win:
                        r = {u for u in s if own(u) != 2}
                        remote += len(r)
                        hits += len(r & hot)
                a = ggref.simulate_epoch(ids, off, W, -1, part, COEF, hot_frac=(num, den))
                assert (a["hits"], a["remote_rows"]) == (hits, remote), (trial, num, den, W)


def test_relative_budget_argument_checks():
    for n_hot, frac in ((3, (1, 10)), (-1, (11, 10)), (-1, (-1, 10)), (-1, (1, 1 << 32))):
        with pytest.raises(ggref.OracleError):
            ggref.build_hotset(IDS, OFF, 3, 0, PART, n_hot, hot_frac=frac)
