"""GPU parity: the HIP path through the C ABI against the CPU oracle, byte
for byte (the path moves ids and opaque feature bytes only, so the
tolerance is exact equality)."""
import numpy as np
import pytest

import synth
from tests import helpers

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util  # noqa: F401  (loads libgg)
    yield


def world(*a, **k):
    from tests.gpu_util import World
    return World(*a, **k)


def log(m):
    print(m, flush=True)


def test_tiny_window_matches_oracle():
    log("tiny: mod-4 owners, fanout [10,5], W=4")
    w = world(synth.instance("tiny"))
    w.run_and_compare(0)


@pytest.mark.parametrize("n_hot", [0, 1, 100, 2000, 10**7])
def test_tiny_hot_budget_and_miss_path(n_hot):
    log(f"tiny: n_hot={n_hot}")
    w = world(synth.instance("tiny"), n_hot=n_hot)
    w.run_and_compare(0)


def test_tiny_all_owners_remote():
    log("tiny: local_owner=-1")
    w = world(synth.instance("tiny"), local_owner=-1)
    w.run_and_compare(0)


def test_small_consecutive_windows_restage_and_invalidate():
    log("small: range owners, 3 consecutive windows, W=4")
    w = world(synth.instance("small"))
    for k in range(3):
        r = w.run_and_compare(k)
        assert r["stage"]["invalidated"] == (0 if k == 0 else len(prev))
        prev = r["hot"]


@pytest.mark.parametrize("W", [1, 3, 7])
def test_small_window_sizes(W):
    log(f"small: W={W}")
    w = world(synth.instance("small"), W=W)
    w.run_and_compare(0)
    w.run_and_compare(1)


@pytest.mark.parametrize("n_hot", [-1, 0, 1, 2000])
def test_hot_set_in_multi_pass_chunks(n_hot):
    """The hot set's chunks span several 256-word passes once a graph has
    more than 4096 of them; tuning hot_max_chunks = 2 forces that layout on
    the small graph, with and without a budget."""
    log(f"small: hot set in two chunks of several passes, n_hot={n_hot}")
    from paper_2606_02916_amd import gg
    w = world(synth.instance("small"), n_hot=n_hot, tuning=gg.make_tuning(hot_max_chunks=2))
    w.run_and_compare(0)
    w.run_and_compare(1)


@pytest.mark.parametrize("tile", [1, 4, 16])
@pytest.mark.parametrize("n_hot", [-1, 300])
def test_fewer_rows_per_wave_step(tile, n_hot):
    """Tuning tile_rows shrinks the rows a wavefront copies per step in the
    stage and the gather (1 = one row per wavefront step), the variants the
    benchmark's ablation times: same bytes, with and without misses."""
    log(f"small: {tile} rows per wave step, n_hot={n_hot}")
    from paper_2606_02916_amd import gg
    w = world(synth.instance("small"), n_hot=n_hot, tuning=gg.make_tuning(tile_rows=tile))
    w.run_and_compare(0)
    w.run_and_compare(1)


@pytest.mark.parametrize("frac", [(1, 10), (1, 3), (0, 1), (1, 1), (999, 1000)])
def test_relative_budget_window_matches_oracle(frac):
    log(f"small: hot set = top {frac[0]}/{frac[1]} of the window's remote nodes, 2 windows")
    w = world(synth.instance("small"), hot_frac=frac)
    w.run_and_compare(0)
    w.run_and_compare(1)


def test_small_budget_misses_across_windows():
    log("small: n_hot=3000 over two windows")
    w = world(synth.instance("small"), n_hot=3000)
    w.run_and_compare(0)
    w.run_and_compare(1)


def test_ragged_and_empty_batches():
    log("tiny: ragged batch sizes with an empty batch")
    inst = synth.instance("tiny")
    w = world(inst, W=5, batch=1000)
    sizes = [1, 0, 65, 257, 1000]
    seeds = np.random.default_rng(2).integers(0, inst.wl.num_nodes, sum(sizes)).astype(np.int32)
    so = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    w.run_and_compare(0, seeds=seeds, so=so, b0=3)


@pytest.mark.parametrize("sizes", [[16384, 3, 0], [16385, 700, 1]])
def test_seed_batches_at_and_past_the_fused_level0_limit(sizes):
    """Level 0 is built in one launch for batches of up to 16,384 seeds and
    by a clearing pass plus atomic marks beyond; duplicated seeds either
    way (batches larger than the graph's 10,000 nodes)."""
    log(f"tiny: seed batches of {sizes}")
    inst = synth.instance("tiny")
    w = world(inst, W=len(sizes), batch=max(sizes))
    seeds = np.random.default_rng(5).integers(0, inst.wl.num_nodes, sum(sizes)).astype(np.int32)
    so = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    w.run_and_compare(0, seeds=seeds, so=so, b0=7)


def test_fanout_above_every_degree_is_the_bfs_ball():
    log("hand graph: fanout above max degree")
    rng = np.random.default_rng(3)
    row_ptr, col_idx = helpers.random_graph(3000, 20000, rng)
    maxdeg = int(np.diff(row_ptr).max())
    assert maxdeg < 32
    wl = synth.Workload("hand", 3000, col_idx.shape[0], False, 64, synth.PART_MOD, 4, 1, 16, "fp32",
                        "normal", (maxdeg + 1, maxdeg + 1), 40, 2, "perm_all", n_windows=1)
    inst = synth.Instance(wl, row_ptr, col_idx, *synth.seed_batches(wl),
                          [synth.shard_features(wl, m) for m in range(4)], None)
    w = world(inst)
    r = w.run_and_compare(0)
    L, W = 2, 2
    for b in range(W):
        s = inst.batch_off
        want = helpers.bfs_ball(row_ptr, col_idx, inst.seeds[s[b]:s[b + 1]], L)
        got = r["fids"][r["foff"][L * W + b]:r["foff"][L * W + b + 1]].tolist()
        assert got == want


def test_unaligned_rows_use_the_word_path():
    log("tiny: 44-byte rows at a 44-byte stride, 4-byte copy path")
    inst = synth.instance("tiny")
    rng = np.random.default_rng(5)
    shards = [rng.integers(0, 256, size=(s.shape[0], 44), dtype=np.uint8) for s in inst.shards]
    w = world(inst, shards=shards, row_bytes=44, stride=44, cache_stride=44)
    w.run_and_compare(0)


def test_row_with_tail_words():
    log("tiny: 1 KB + 12 byte rows at a 16-byte-aligned stride (vector path with tail)")
    inst = synth.instance("tiny")
    rng = np.random.default_rng(6)
    shards = [rng.integers(0, 256, size=(s.shape[0], 1040), dtype=np.uint8) for s in inst.shards]
    w = world(inst, shards=shards, row_bytes=1036, stride=1040)
    w.run_and_compare(0)


@pytest.mark.parametrize("rows", [(4, 4), (4, 16), (16, 16), (20, 20), (20, 32), (100, 100),
                                  (100, 112), (1204, 1204), (1204, 1216)])
def test_row_widths_with_one_chunk_or_one_tail_word(rows):
    """Row widths whose copy geometry has a divisor of 1: one 16-byte chunk
    per row (16 and 20 bytes), one 4-byte tail word (4, 20, 100 and 1,204
    bytes on the vector path) or one word per row (4 bytes on the word
    path), with strides that are and are not multiples of 16.  Through
    k_stage_rows and both gathers with a budget that leaves misses
    (k_gather_finish), then through in-place staging (k_inplace_rows) over
    two windows with the union."""
    rb, stride = rows
    log(f"tiny: {rb}-byte rows at stride {stride}")
    inst = synth.instance("tiny")
    rng = np.random.default_rng(rb * 7 + stride)
    shards = [rng.integers(0, 256, size=(s.shape[0], stride), dtype=np.uint8)
              for s in inst.shards]
    w = world(inst, shards=shards, row_bytes=rb, stride=stride, n_hot=700)
    r = w.run_and_compare(0)
    assert sum(sum(g["miss_rows"]) for g in [w.pipe.gather_stats_dict(b)
                                            for b in range(r["Wk"])]) > 0
    w = world(inst, shards=shards, row_bytes=rb, stride=stride, W=2, inplace=True)
    for k in range(2):
        w.run_and_compare(k)


@pytest.mark.parametrize("tile", [None, 64])
@pytest.mark.parametrize("n_hot", [0, 700, -1])
def test_wide_rows_with_misses(n_hot, tile):
    """2,408-byte rows at a 2,416-byte stride (by default eight rows per
    staging step and two per gather step; tuning tile_rows = 64 makes both
    64) through both gathers and the miss path: with n_hot = 0 every remote
    row is a miss, with 700 some are."""
    log(f"tiny: 2408-byte rows, tile {tile or 'default'}, n_hot={n_hot}, consecutive windows")
    from paper_2606_02916_amd import gg
    inst = synth.instance("tiny")
    rng = np.random.default_rng(8)
    shards = [rng.integers(0, 256, size=(s.shape[0], 2416), dtype=np.uint8) for s in inst.shards]
    w = world(inst, shards=shards, row_bytes=2408, stride=2416, n_hot=n_hot, W=2,
              tuning=gg.make_tuning(tile_rows=tile) if tile else None)
    for k in range(2):
        w.run_and_compare(k)


@pytest.mark.parametrize("fields", [
    dict(mark_slices_max=-1, bytemap_max_mb=-1), dict(mark_slices_max=-1, bytemap_max_mb=1),
    dict(mark_slices_max=-1),
    dict(gather_loads=2, gather_blocks=8), dict(gather_loads=4), dict(gather_loads=8, tile_rows=3),
    dict(stage_blocks=1, tile_rows=7), dict(stage_blocks=3, emit_blocks=1, hot_max_chunks=1),
    dict(sample_order=1), dict(sample_order=2), dict(sample_order=2, sample_tile_runs=1),
    dict(sample_order=2, sample_tile_runs=64),
    dict(sample_order=1, bytemap_max_mb=-1, mark_slices_max=-1),
    dict(sample_order=2, mark_slices_max=-1),
    dict(mark_min_slots=-1), dict(mark_min_slots=10**9), dict(mark_block=256),
    dict(mark_block=1024, mark_min_slots=-1, sample_order=2)])
def test_launch_tuning_leaves_results_unchanged(fields):
    """Launch tuning changes only how the work is spread: the sampler's
    marks through LDS (in blocks of 256 or 1,024 lanes, at every hop or at
    the last only), by atomic ORs (as on the 111M-node graph) or, at the
    last hop, into the byte map; the sampler in
    node tiles at the last hop or at every hop (sized per hop, or fixed at
    256 or 16,384 ids); gathers with 2, 4 or 8 loads in flight and few
    blocks (many tiles per wave), staging by one or three blocks, one
    hot-set chunk and one free-list block.  Full restage, then in-place staging over three
    windows, each against the oracle with a budget that leaves misses."""
    log(f"small: tuning {fields}")
    from paper_2606_02916_amd import gg
    tune = gg.make_tuning(**fields)
    inst = synth.instance("small")
    w = world(inst, n_hot=3000, tuning=tune)
    w.run_and_compare(0)
    w = world(inst, n_hot=3000, inplace=True, tuning=tune)
    for k in range(3):
        w.run_and_compare(k)


@pytest.mark.parametrize("fields", [
    dict(), dict(mark_slices_max=-1), dict(mark_slices_max=-1, bytemap_max_mb=-1),
    dict(sample_order=1), dict(sample_order=1, mark_slices_max=-1)])
def test_sample_window_in_two_parts_across_streams(fields):
    """gg_sample_window_part: the bits part on one stream, then (after an
    event) the last level's compaction on another; the bit sets are final
    after the first part (marked through LDS, or the byte map folded in,
    when either is used), and after the second every output equals the
    oracle's."""
    log(f"small: sampling in two parts on two streams, tuning {fields}")
    import torch as T
    from oracle import ggref
    from paper_2606_02916_amd import gg
    tune = gg.make_tuning(**fields)
    w = world(synth.instance("small"), tuning=tune)
    p = w.pipe
    L = len(w.fanout)
    s1, s2 = T.cuda.Stream(), T.cuda.Stream()
    for k in range(2):
        seeds, so, b0 = w.window_inputs(k)
        sd = T.from_numpy(seeds).to(w.dev)
        p.frontier_ids.fill_(-7)
        T.cuda.synchronize()
        args = (p.csr, sd, so, len(so) - 1, list(w.fanout), L, 0, 0, b0, p.wsample)
        gg.gg_sample_window_part(*args, gg.GG_SAMPLE_PART_BITS, p.status, p.ws, stream=s1,
                                 tuning=tune)
        ev = T.cuda.Event()
        ev.record(s1)
        s2.wait_event(ev)
        gg.gg_sample_window_part(*args, gg.GG_SAMPLE_PART_LAST, p.status, p.ws, stream=s2,
                                 tuning=tune)
        T.cuda.synchronize()
        assert p.read_status() == 0
        Wk = len(so) - 1
        fids, foff, nids, noff = ggref.sample_window(w.inst.row_ptr, w.inst.col_idx, seeds, so,
                                                     w.fanout, 0, 0, b0)
        g_fids, g_foff, g_nids, g_noff = p.sample_outputs(Wk)
        assert np.array_equal(g_foff, foff) and np.array_equal(g_fids, fids)
        assert np.array_equal(g_noff, noff) and np.array_equal(g_nids, nids)
        from tests.gpu_util import check_bits
        bits = p.frontier_bits[:Wk * p.wpb].cpu().numpy().view(np.uint32)
        check_bits(bits, p.wpb, Wk, lambda b: fids[foff[L * Wk + b]:foff[L * Wk + b + 1]])
    with pytest.raises(gg.GGError):
        gg.gg_sample_window_part(*args, 3, p.status, p.ws, tuning=tune)


@pytest.mark.parametrize("n_hot", [-1, 200])
def test_every_limit_at_once(n_hot):
    """The ABI's limits together: W = 64 batches (of 16 seeds), L = 4 hops
    with a fan-out of 32 at the first (the widest Floyd network), and 64
    owners by node id mod 64 with local owner 5; with the union and with a
    budget (the miss path over 64 owners)."""
    log(f"tiny graph: W=64, L=4, fanout [32,3,2,1], 64 owners (mod), local 5, n_hot={n_hot}")
    import dataclasses
    base = synth.instance("tiny")
    wl = dataclasses.replace(base.wl, name="tiny_limits", num_parts=64, local_owner=5,
                             fanout=(32, 3, 2, 1), batch_size=16, W=64)
    shards = [synth.shard_features(wl, m) for m in range(wl.num_parts)]
    inst = synth.Instance(wl, base.row_ptr, base.col_idx, *synth.seed_batches(wl), shards, None)
    w = world(inst, n_hot=n_hot)
    r = w.run_and_compare(0)
    assert r["Wk"] == 64


def test_repeat_runs_are_identical():
    log("small: determinism across two pipelines")
    inst = synth.instance("small")
    a = world(inst)
    b = world(inst)
    ra = a.run_and_compare(0)
    rb = b.run_and_compare(0)
    assert np.array_equal(ra["fids"], rb["fids"])


def test_capacity_overflow_is_flagged_and_clamped():
    log("tiny: frontier capacity too small -> status bit, no out-of-bounds writes")
    import torch as T
    from paper_2606_02916_amd import gg
    w = world(synth.instance("tiny"))
    p = w.pipe
    guard = 4096
    small = T.full((1000 + guard,), 0x7EADBEEF, dtype=T.int32, device=w.dev)
    ws = gg.make_wsample(small[:1000], p.frontier_off, p.nbr_ids, p.nbr_off, p.frontier_bits,
                         p.need)
    seeds, so, b0 = w.window_inputs(0)
    sd = T.from_numpy(seeds).to(w.dev)
    gg.gg_sample_window(p.csr, sd, so, len(so) - 1, list(w.fanout), len(w.fanout), 0, 0, b0, ws,
                        p.status, p.ws)
    T.cuda.synchronize()
    assert p.read_status() & gg.DEV_CAPACITY
    assert int(p.need[0].item()) > 1000
    assert bool((small[1000:] == 0x7EADBEEF).all())
    assert int(p.frontier_off.max().item()) <= 1000


@pytest.mark.parametrize("frac", [0.3, 0.8])
def test_slot_overflow_leaves_the_same_sets_under_every_marking(frac):
    """Neighbour slots too few for the window (a capacity of 30m + 1, a
    multiple of no fan-out, so an entry straddles it): the status bit is
    raised, nothing is written past the capacity, and marks through LDS
    (which read the written slots of complete entries only), atomic ORs and
    the last hop's byte map leave the same bit sets, lists and offsets."""
    log(f"small: neighbour-slot capacity {frac} of the need, three ways of marking")
    import torch as T
    from paper_2606_02916_amd import gg
    w = world(synth.instance("small"))
    p = w.pipe
    N, L = w.inst.wl.num_nodes, len(w.fanout)
    seeds, so, b0 = w.window_inputs(0)
    sd = T.from_numpy(seeds).to(w.dev)
    Wk = len(so) - 1
    gg.gg_sample_window(p.csr, sd, so, Wk, list(w.fanout), L, 0, 0, b0, p.wsample, p.status,
                        p.ws)
    T.cuda.synchronize()
    assert p.read_status() == 0
    need = int(p.need[1].item())
    ncap = int(need * frac) // 30 * 30 + 1
    assert 0 < ncap < need and all(ncap % k for k in w.fanout)
    guard = 4096
    outs = []
    for fields in (dict(), dict(mark_slices_max=-1), dict(mark_slices_max=-1, bytemap_max_mb=-1)):
        tune = gg.make_tuning(**fields)
        ws = T.empty(gg.gg_ws_sample(N, Wk, tune), dtype=T.uint8, device=w.dev)
        nb = T.full((ncap + guard,), 0x7EADBEEF, dtype=T.int32, device=w.dev)
        wsm = gg.make_wsample(p.frontier_ids, p.frontier_off, nb[:ncap], p.nbr_off,
                              p.frontier_bits, p.need)
        p.frontier_ids.fill_(-7)
        p.status.zero_()
        gg.gg_sample_window(p.csr, sd, so, Wk, list(w.fanout), L, 0, 0, b0, wsm, p.status, ws,
                            tuning=tune)
        T.cuda.synchronize()
        assert p.read_status() & gg.DEV_CAPACITY, fields
        assert bool((nb[ncap:] == 0x7EADBEEF).all()), fields
        foff = p.frontier_off[:(L + 1) * Wk + 1].cpu().numpy()
        outs.append((p.frontier_bits[:Wk * p.wpb].cpu().numpy(), foff,
                     p.frontier_ids[:int(foff[-1])].cpu().numpy(),
                     p.nbr_off[:L * Wk + 1].cpu().numpy(), nb[:ncap].cpu().numpy(),
                     p.need.cpu().numpy()))
    for o in outs[1:]:
        for x, y in zip(outs[0], o):
            assert np.array_equal(x, y)


@pytest.mark.parametrize("mark_block", [256, 1024])
def test_marks_from_unaligned_slots_match_oracle(mark_block):
    """Neighbour slots at an address that is not 16-byte aligned (a C
    caller's buffer, one int32 past an aligned one): the mark pass reads
    them one at a time instead of in 16-byte groups.  Every hop marks
    through LDS; the window's frontiers, slots and bit sets against the
    oracle."""
    log(f"small: LDS marks from unaligned neighbour slots, {mark_block}-lane blocks")
    import torch as T
    from oracle import ggref
    from paper_2606_02916_amd import gg
    from tests.gpu_util import check_bits
    tune = gg.make_tuning(mark_min_slots=-1, mark_min_batches=-1, mark_block=mark_block)
    w = world(synth.instance("small"), tuning=tune)
    p = w.pipe
    L = len(w.fanout)
    seeds, so, b0 = w.window_inputs(0)
    sd = T.from_numpy(seeds).to(w.dev)
    Wk = len(so) - 1
    nb = T.full((p.nbr_ids.numel() + 1,), 0x7EADBEEF, dtype=T.int32, device=w.dev)
    assert nb[1:].data_ptr() % 16 == 4
    wsm = gg.make_wsample(p.frontier_ids, p.frontier_off, nb[1:], p.nbr_off, p.frontier_bits,
                          p.need)
    gg.gg_sample_window(p.csr, sd, so, Wk, list(w.fanout), L, 0, 0, b0, wsm, p.status, p.ws,
                        tuning=tune)
    T.cuda.synchronize()
    assert p.read_status() == 0
    fids, foff, nids, noff = ggref.sample_window(w.inst.row_ptr, w.inst.col_idx, seeds, so,
                                                 w.fanout, 0, 0, b0)
    g_foff = p.frontier_off[:(L + 1) * Wk + 1].cpu().numpy()
    g_noff = p.nbr_off[:L * Wk + 1].cpu().numpy()
    assert np.array_equal(g_foff, foff) and np.array_equal(g_noff, noff)
    assert np.array_equal(p.frontier_ids[:int(foff[-1])].cpu().numpy(), fids)
    assert np.array_equal(nb[1:1 + int(noff[-1])].cpu().numpy(), nids)
    bits = p.frontier_bits.view(T.int32)[:Wk * p.wpb].cpu().numpy().view(np.uint32)
    check_bits(bits, p.wpb, Wk, lambda b: fids[foff[L * Wk + b]:foff[L * Wk + b + 1]])


@pytest.mark.timeout(900)
@pytest.mark.parametrize("fields", [dict(), dict(mark_slice_chunks=3, mark_slices_max=16,
                                                mark_block=256, mark_min_slots=-1)])
def test_large_sparse_full_window_matches_oracle(fields):
    """Window 0 of the 2.45M-node graph against the oracle; with the second
    tuning every hop marks through LDS slices of 3 chunks (13 slices per
    batch, the last one of 2 chunks)."""
    log(f"large_sparse: 2.45M nodes, 62M edges, fanout [15,10,5], batch 1024, W=16, window 0, "
        f"tuning {fields}")
    from paper_2606_02916_amd import gg
    w = world(synth.instance("large_sparse"), tuning=gg.make_tuning(**fields))
    w.run_and_compare(0)


def rows_from_shards(inst, ids, rb):
    """Feature rows of `ids` read straight from the owners' shards (range
    book): ground truth independent of any cache."""
    rs = inst.range_start
    out = np.empty((len(ids), rb), dtype=np.uint8)
    owner = np.searchsorted(np.asarray(rs), ids, side="right") - 1
    for m in range(len(rs) - 1):
        sel = owner == m
        out[sel] = inst.shards[m][ids[sel] - rs[m], :rb]
    return out


@pytest.mark.timeout(1500)
@pytest.mark.parametrize("name", ["large_sparse", "dense_mid", "papers_share"])
def test_lookahead_as_benchmarked(name):
    """The benchmark's launch configuration: the look-ahead driver with its
    default buffer sets (three with every shard in HBM; two on the
    Papers100M share, whose remote shards sit in pinned host memory) and
    streams (staging on the fetch stream and the gather on a third stream on
    that share and on the 2.45M-node graph, whose build is the longer
    chain; staging after the build on the 233K-node graph) and only
    a gather end event per window, over four consecutive windows (window
    k+1 is enqueued before window k is read).  Every window against the
    oracle element by element: every batch's frontiers, neighbour slots and
    bit set, the hot set, buckets, staging statistics, the whole remap,
    every staged row, gather statistics and every gathered row; the gathered
    rows also against the owners' shards directly."""
    log(f"{name}: look-ahead driver as benchmarked, windows 0-3 against the oracle")
    import torch as T
    from paper_2606_02916_amd import LookaheadPipeline
    from tests.gpu_util import LookaheadOracle
    inst, rp_d, ci_d, sh_d = synth.torch_instance(name, "cuda:0")
    wl = inst.wl
    assert wl.part_kind == synth.PART_RANGE and wl.local_owner == 0
    P, L, W = wl.num_parts, len(wl.fanout), wl.W
    dev = T.device("cuda:0")
    look = LookaheadPipeline(rp_d, ci_d, P, wl.part_kind, wl.local_owner, inst.range_start, sh_d,
                             [s.shape[0] for s in inst.shards], wl.row_bytes, wl.row_stride, W,
                             wl.fanout, wl.batch_size, device=dev)
    host = wl.remote_on_host
    assert look.nsets == (2 if host else 3)
    assert look.stage_apart == (host or name == "large_sparse")
    assert (look.stage_stream is look.build_stream) != look.stage_apart
    orc = LookaheadOracle(inst, look)
    seeds_d = T.from_numpy(inst.seeds).to(dev)
    boff, rb = inst.batch_off, wl.row_bytes

    def check(k, Wk, bufs, b0, b1):
        look.gathered_event(k).synchronize()
        log(f"{name}: checking window {k} ({Wk} batches)")
        seeds = inst.seeds[boff[b0]:boff[b1]]
        r = orc.check(k, Wk, bufs, seeds, boff[b0:b1 + 1] - boff[b0], b0)
        fids, foff = r["fids"], r["foff"]
        allN = fids[int(foff[L * Wk]):]
        got = bufs.win_out[:len(allN), :rb].cpu().numpy()
        assert np.array_equal(got, rows_from_shards(inst, allN, rb)), f"window {k} rows"
        for b in range(Wk):
            gs = bufs.gather_stats_dict(b)
            assert gs["misses"] == 0 and gs["local"] + gs["hits"] == gs["rows"]

    pending = None
    for k in range(4):
        b0, b1 = synth.window_batches(boff, W, k)
        Wk, bufs = look.window(seeds_d[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0], b0,
                               gather_events=(None, T.cuda.Event(enable_timing=True)))
        if pending is not None:
            check(*pending)
        pending = (k, Wk, bufs, b0, b1)
    check(*pending)
    assert look.read_status() == 0


@pytest.mark.parametrize("split,host", [(True, False), (False, False), (True, True)])
def test_lookahead_split_sampling_matches_oracle(split, host):
    """The look-ahead driver with the last level's compaction on the gather
    stream (split) or on the build stream, with shards in device memory and
    with the remote shards in pinned host memory: five consecutive windows
    of the small graph against the oracle, element by element."""
    log(f"small: look-ahead, split_last={split}, host shards={host}, windows 0-4")
    import torch as T
    from paper_2606_02916_amd import LookaheadPipeline
    from tests.gpu_util import LookaheadOracle
    inst = synth.instance("small")
    wl = inst.wl
    dev = T.device("cuda:0")
    rp_d, ci_d = T.from_numpy(inst.row_ptr).to(dev), T.from_numpy(inst.col_idx).to(dev)
    sh_d = [T.from_numpy(sh).to(dev) if (m == wl.local_owner or not host)
            else T.from_numpy(sh).pin_memory() for m, sh in enumerate(inst.shards)]
    look = LookaheadPipeline(rp_d, ci_d, wl.num_parts, wl.part_kind, wl.local_owner,
                             inst.range_start, sh_d, [x.shape[0] for x in inst.shards],
                             wl.row_bytes, wl.row_stride, wl.W, wl.fanout, wl.batch_size,
                             device=dev, split_last=split)
    assert look.split_last == split
    orc = LookaheadOracle(inst, look)
    boff = inst.batch_off
    seeds_d = T.from_numpy(inst.seeds).to(dev)
    pending = None
    for k in range(min(5, synth.n_windows(boff, wl.W))):
        b0, b1 = synth.window_batches(boff, wl.W, k)
        Wk, bufs = look.window(seeds_d[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0], b0,
                               gather_events=(None, T.cuda.Event()))
        if pending is not None:
            pk, pW, pb, pb0, pb1 = pending
            look.gathered_event(pk).synchronize()
            orc.check(pk, pW, pb, inst.seeds[boff[pb0]:boff[pb1]], boff[pb0:pb1 + 1] - boff[pb0],
                      pb0)
        pending = (k, Wk, bufs, b0, b1)
    pk, pW, pb, pb0, pb1 = pending
    look.gathered_event(pk).synchronize()
    orc.check(pk, pW, pb, inst.seeds[boff[pb0]:boff[pb1]], boff[pb0:pb1 + 1] - boff[pb0], pb0)
    assert look.read_status() == 0


@pytest.mark.parametrize("fields", [dict(bytemap_max_mb=1, mark_slices_max=-1), dict()])
def test_short_last_window_takes_the_byte_map(fields):
    """Workspaces sized for W = 20 batches of the small graph serve the
    epoch's 4-batch last window, which takes the byte map where the 20-batch
    window does not: with a 1 MB limit (1.3 MB of map for 20 batches: atomic
    marks; 256 KB for 4), and by default (LDS marks from 8 batches on: the
    20-batch window marks through LDS, the 4-batch one into the map).  The
    sequential driver and the look-ahead driver (split sampling) over both
    windows, against the oracle."""
    log(f"small: W=20 (windows of 20 and 4 batches), tuning {fields}")
    import torch as T
    from paper_2606_02916_amd import LookaheadPipeline, gg
    from tests.gpu_util import LookaheadOracle
    tune = gg.make_tuning(**fields)
    inst = synth.instance("small")
    wl, W = inst.wl, 20
    boff = inst.batch_off
    assert synth.n_windows(boff, W) == 2 and len(boff) - 1 == 24
    per_batch = gg.gg_bits_words(wl.num_nodes) * 32
    assert 4 * per_batch <= 1 << 20 < W * per_batch
    # the 20-batch workspace holds the 4-batch window's map
    assert gg.gg_ws_sample(wl.num_nodes, W, tune) >= 4 * per_batch
    w = world(inst, W=W, n_hot=3000, tuning=tune)
    for k in range(2):
        w.run_and_compare(k)
    dev = T.device("cuda:0")
    rp_d, ci_d = T.from_numpy(inst.row_ptr).to(dev), T.from_numpy(inst.col_idx).to(dev)
    sh_d = [T.from_numpy(sh).to(dev) for sh in inst.shards]
    look = LookaheadPipeline(rp_d, ci_d, wl.num_parts, wl.part_kind, wl.local_owner,
                             inst.range_start, sh_d, [x.shape[0] for x in inst.shards],
                             wl.row_bytes, wl.row_stride, W, wl.fanout, wl.batch_size,
                             device=dev, tuning=tune)
    assert look.split_last
    orc = LookaheadOracle(inst, look)
    seeds_d = T.from_numpy(inst.seeds).to(dev)
    for k in range(2):
        b0, b1 = synth.window_batches(boff, W, k)
        Wk, bufs = look.window(seeds_d[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0], b0)
        look.gathered_event(k).synchronize()
        orc.check(k, Wk, bufs, inst.seeds[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0], b0)
    assert look.read_status() == 0


@pytest.mark.timeout(900)
def test_dense_mid_full_window_matches_oracle():
    log("dense_mid: 233K nodes, 114M edges, fp32x602 (stride 2416), fanout [25,10], W=8, window 0")
    w = world(synth.instance("dense_mid"))
    w.run_and_compare(0)


@pytest.mark.parametrize("flags", [0, 1])
@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("order", ["ascending", "shuffled", "one_descent"])
def test_bucket_by_owner_direct(kind, order, flags):
    """flags=1 is GG_BUCKET_OWNER_ORDERED: under a range book an input out of
    owner order must raise GG_DEV_ORDER instead of being bucketed."""
    log(f"bucket_by_owner: kind={kind} order={order} flags={flags}")
    import torch as T
    from oracle import ggref
    from paper_2606_02916_amd import gg
    rng = np.random.default_rng(17)
    N, P = 500_000, 5
    rs = [0, 70_000, 70_000, 300_000, 420_001, N]
    ids = np.sort(rng.choice(N, size=123_457, replace=False)).astype(np.int32)
    if order == "shuffled":
        rng.shuffle(ids)
    elif order == "one_descent":
        ids[[1000, 60_000]] = ids[[60_000, 1000]]
    part_ref = ggref.make_part(P, kind, 0, N, rs if kind == 1 else None)
    want, want_off = ggref.bucket_by_owner(ids, part_ref)
    dev = T.device("cuda:0")
    cap = ids.shape[0] + 1000
    hot = T.zeros(cap, dtype=T.int32, device=dev)
    hot[:ids.shape[0]] = T.from_numpy(ids).to(dev)
    cnt = T.tensor([ids.shape[0], ids.shape[0]], dtype=T.int64, device=dev)
    out = T.full((cap,), -7, dtype=T.int32, device=dev)
    off = T.zeros(P + 1, dtype=T.int64, device=dev)
    status = T.zeros(1, dtype=T.int32, device=dev)
    ws = T.empty(gg.gg_ws_bucket(cap, P), dtype=T.uint8, device=dev)
    part = gg.make_part(P, kind, 0, N, rs if kind == 1 else None)
    gg.gg_bucket_by_owner(hot, cnt, cap, part, out, off, status, ws, flags=flags)
    T.cuda.synchronize()
    if flags and kind == 1 and order != "ascending":
        assert int(status.item()) == gg.DEV_ORDER
        return
    assert int(status.item()) == 0
    assert np.array_equal(off.cpu().numpy(), want_off)
    assert np.array_equal(out[:ids.shape[0]].cpu().numpy(), want)
    assert np.all(out[ids.shape[0]:].cpu().numpy() == -7)


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("W,nwin", [(1, 2), (2, 2), (4, 2), (8, 2), (16, 1), (32, 1)])
def test_wsweep_batch4096_matches_oracle(W, nwin):
    """The W sweep at batch 4096 on the large sparse graph: window 0 (and
    window 1 where W <= 8) of every W against the oracle, every
    intermediate element by element (sampling, bit sets, hot set, buckets,
    staged cache, remap, statistics, per-batch and whole-window gathers)."""
    log(f"wsweep graph: batch 4096, W={W}, windows 0..{nwin - 1}, full compare")
    w = world(synth.instance("wsweep"), W=W)
    for k in range(nwin):
        r = w.run_and_compare(k)
        assert r["Wk"] == W


@pytest.mark.timeout(1800)
def test_papers_share_windows_match_oracle():
    """The Papers100M-shaped share (111M nodes, 1.6B edges, fp16 x 128; the
    three remote shards in pinned host memory, read over PCIe) through the
    sequential driver, windows 0 and 1: every intermediate against the
    oracle element by element (all 16 batches' frontiers and neighbour
    slots, bit sets, hot set, frequencies, buckets, owner offsets, staging
    statistics, the whole remap, every cache row, every gathered row of the
    per-batch and whole-window gathers)."""
    log("papers_share: 111M nodes, 1.6B edges, fp16x128, remote shards in pinned host memory, "
        "W=16, windows 0 and 1 against the oracle")
    inst, rp_d, ci_d, sh_d = synth.torch_instance("papers_share", "cuda:0")
    assert all(not sh_d[m].is_cuda for m in (1, 2, 3)) and sh_d[0].is_cuda
    w = world(inst, tensors=(rp_d, ci_d, sh_d))
    for k in range(2):
        log(f"papers_share: window {k}")
        r = w.run_and_compare(k)
        assert r["stage"]["requests"] == [0, 1, 1, 1]


@pytest.mark.parametrize("name,n_hot,W", [("small", -1, None), ("small", 3000, None),
                                          ("tiny", -1, 1)])
def test_delta_staging_matches_oracle(name, n_hot, W):
    log(f"{name}: delta staging over consecutive windows, n_hot={n_hot}, W={W}")
    w = world(synth.instance(name), n_hot=n_hot, W=W, delta=True)
    nwin = synth.n_windows(w.inst.batch_off, w.W)
    for k in range(min(nwin, 4)):
        r = w.run_and_compare(k)
        st = r["stage"]
        if k > 0:
            assert st["retained"] > 0
            assert st["rows"] == st["delta_rows"]          # only the delta is requested
            assert st["retained"] + sum(st["rows"]) == st["rows_total"]


def test_window_graph_replays_match_eager():
    """A whole sequential window captured into a HIP graph and replayed
    three times, with eager GPU work, host synchronisation and a refill of
    the seeds between replays: after every replay the sampled frontiers and
    neighbour slots, hot set, buckets, remap, statistics and every gathered
    row equal an eager run of the same seeds (at the captured batch index)."""
    log("small: window graph replays against eager windows")
    import torch as T
    from paper_2606_02916_amd import FetchPipeline
    inst = synth.instance("small")
    wl = inst.wl
    dev = T.device("cuda:0")
    boff, W, L, rb = inst.batch_off, wl.W, len(wl.fanout), wl.row_bytes
    wins = []
    for k in range(2):
        b0, b1 = synth.window_batches(boff, W, k)
        wins.append((inst.seeds[boff[b0]:boff[b1]].copy(), boff[b0:b1 + 1] - boff[b0], b0))
    assert np.array_equal(wins[0][1], wins[1][1])
    so, b0 = wins[0][1], wins[0][2]
    rp = T.from_numpy(inst.row_ptr).to(dev)
    ci = T.from_numpy(inst.col_idx).to(dev)
    sh = [T.from_numpy(x).to(dev) for x in inst.shards]

    def make():
        return FetchPipeline(rp, ci, wl.num_parts, wl.part_kind, wl.local_owner,
                             inst.range_start, sh, [x.shape[0] for x in inst.shards], rb,
                             wl.row_stride, W, wl.fanout, wl.batch_size, device=dev)

    def snapshot(p, Wk):
        fids, foff, nids, noff = p.sample_outputs(Wk)
        hot, freq, cnt, bucket, owner_off = p.hot_outputs(0)
        n = int(foff[(L + 1) * Wk] - foff[L * Wk])
        return dict(fids=fids, foff=foff, nids=nids, noff=noff, hot=hot, freq=freq,
                    bucket=bucket, owner_off=owner_off, remap=p.slot_of.cpu().numpy(),
                    rows=p.win_out[:n, :rb].cpu().numpy(), stage=p.stage_stats_dict(),
                    gather=[p.gather_stats_dict(b) for b in range(Wk)])

    gpipe, epipe = make(), make()
    seeds_buf = T.from_numpy(wins[0][0]).to(dev)
    graph, Wk = gpipe.capture_window(seeds_buf, so, b0)
    T.cuda.synchronize()
    for rep, k in enumerate([0, 1, 0]):
        seeds_buf.copy_(T.from_numpy(wins[k][0]).to(dev))
        graph.replay()
        T.cuda.synchronize()
        got = snapshot(gpipe, Wk)
        epipe.reset_cache()
        epipe.window(T.from_numpy(wins[k][0]).to(dev), so, b0)
        T.cuda.synchronize()
        want = snapshot(epipe, Wk)
        for key in want:
            if isinstance(want[key], np.ndarray):
                assert np.array_equal(got[key], want[key]), (rep, key)
            else:
                assert got[key] == want[key], (rep, key)
        x = T.arange(1 << 20, device=dev, dtype=T.float32)     # eager work between replays
        assert float((x * 2).max()) == 2.0 * ((1 << 20) - 1)
    assert gpipe.read_status() == 0 and epipe.read_status() == 0


@pytest.mark.parametrize("name,n_hot,W,rows", [("small", -1, None, None), ("small", 3000, None, None),
                                               ("tiny", -1, 1, None), ("tiny", 700, 2, (2408, 2416)),
                                               ("tiny", -1, 4, (1036, 1040)), ("tiny", 0, 2, None)])
def test_inplace_staging_matches_oracle(name, n_hot, W, rows):
    """Delta staging into one persistent cache over consecutive windows:
    the remap, every staged row at its slot (retained rows keep theirs, the
    delta takes the lowest free slots in bucket order), the statistics and
    every gathered row equal the oracle's; with 2,408-byte rows (tail
    words), an unaligned 1,036-byte row (the 4-byte path) and budgets that
    leave misses."""
    log(f"{name}: in-place staging over consecutive windows, n_hot={n_hot}, W={W}, rows={rows}")
    inst = synth.instance(name)
    kw = {}
    if rows:
        rng = np.random.default_rng(11)
        kw = dict(shards=[rng.integers(0, 256, size=(sh.shape[0], rows[1]), dtype=np.uint8)
                          for sh in inst.shards], row_bytes=rows[0], stride=rows[1])
    w = world(inst, n_hot=n_hot, W=W, inplace=True, **kw)
    nwin = synth.n_windows(w.inst.batch_off, w.W)
    for k in range(min(nwin, 5)):
        r = w.run_and_compare(k)
        st = r["stage"]
        if k > 0 and n_hot != 0:
            assert st["retained"] > 0
        assert st["retained"] + sum(st["rows"]) == st["rows_total"]


@pytest.mark.parametrize("emit_blocks", [1, 2])
def test_inplace_free_list_blocks_take_several_chunks(emit_blocks):
    """The free list of the persistent cache is emitted by at most a fixed
    number of blocks that stride over the 8,192-slot chunks below the
    previous extent; tuning emit_blocks = 1 or 2 makes every block take
    several chunks on the small graph, whose extent passes two chunks."""
    log(f"small: in-place staging, free list emitted by {emit_blocks} block(s)")
    from paper_2606_02916_amd import gg
    w = world(synth.instance("small"), inplace=True,
              tuning=gg.make_tuning(emit_blocks=emit_blocks))
    nwin = synth.n_windows(w.inst.batch_off, w.W)
    ext = []
    for k in range(min(nwin, 5)):
        w.run_and_compare(k)
        # window k's occupancy map starts with its extent (int64)
        ext.append(int(w.pipe.occs[k % 2][:8].cpu().numpy().view(np.int64)[0]))
    assert max(ext[:-1]) > 2 * 8192, ext


@pytest.mark.parametrize("short_by", [1, 40])
def test_inplace_staging_out_of_slots_leaves_misses(short_by):
    """A persistent cache short of two windows' hot sets: the second staging
    raises GG_DEV_CAPACITY and leaves the delta rows past the last free slot
    out of the remap, and the gathers still return every row, those through
    the miss path.  The third window must treat every slot the short window
    filled as taken (the occupancy extent covers the whole cache), so none of
    its delta rows lands on a row it keeps.  All three windows against the
    oracle: remaps, every staged row, statistics, every gathered row."""
    log(f"small: in-place staging with a cache {short_by} slot(s) short of two windows, "
        "three windows")
    from oracle import ggref
    inst = synth.instance("small")
    wl = inst.wl
    L = len(wl.fanout)
    part = ggref.make_part(wl.num_parts, wl.part_kind, wl.local_owner, wl.num_nodes,
                           inst.range_start)
    hot = []
    for k in range(2):
        b0, b1 = synth.window_batches(inst.batch_off, wl.W, k)
        boff = inst.batch_off
        seeds, so = inst.seeds[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0]
        fids, foff, _, _ = ggref.sample_window(inst.row_ptr, inst.col_idx, seeds, so, wl.fanout,
                                               0, 0, b0)
        hot.append(ggref.build_hotset(fids, foff, len(so) - 1, L, part, -1)[0])
    union = len(set(hot[0].tolist()) | set(hot[1].tolist()))
    rows = union - short_by
    assert rows >= len(hot[0])
    w = world(inst, inplace=True, cache_rows=rows)
    shorts = [w.run_and_compare(k)["short"] for k in range(3)]
    assert shorts[:2] == [False, True], shorts
    # the short window's occupancy extent covers the whole cache
    assert int(w.pipe.occs[1][:8].cpu().numpy().view(np.int64)[0]) == rows


@pytest.mark.parametrize("name,n_hot,W,nsets,host,gev,rows", [
    ("small", -1, None, 2, False, None, None), ("small", 3000, None, 2, False, "both", None),
    ("tiny", -1, 1, 2, False, None, None), ("small", -1, None, None, False, "end", None),
    ("tiny", 2000, 1, 3, False, "end", None), ("small", 3000, None, 4, False, "both", None),
    ("small", -1, None, None, True, "both", None), ("small", 3000, None, 3, True, "end", None),
    ("small", 3000, None, None, "apart", "end", None), ("tiny", -1, 1, 2, "apart", "both", None),
    ("tiny", 700, 2, None, False, "end", (1036, 1040)),
    ("small", 3000, None, None, False, "end", (2408, 2416))])
def test_lookahead_pipeline_equals_sequential(name, n_hot, W, nsets, host, gev, rows):
    """The look-ahead driver against the sequential delta-staging driver,
    window by window: with shards in device memory (staging on the build
    stream, or on a stream of its own: "apart") and with the remote shards
    in pinned host memory (staging on the fetch stream, gathers on a third
    stream); without gather events,
    with both, and with only the end event, which then also releases the
    buffer set (the benchmark's configuration).  Rows of 1,036 and 2,408
    bytes give the look-ahead's gather (four loads, tiles of as many rows
    as fit in 8 KB) tiles of 7 and 3 rows, where the sequential driver's
    gather takes 4 and 2."""
    log(f"{name}: look-ahead pipeline vs sequential delta windows, n_hot={n_hot}, W={W}, "
        f"nsets={nsets}, host shards={host}, gather events={gev}, rows={rows}")
    import torch as T
    from paper_2606_02916_amd import LookaheadPipeline
    inst = synth.instance(name)
    wl = inst.wl
    apart = host == "apart"
    host = host is True
    kw = {}
    if rows:
        rng = np.random.default_rng(13)
        kw = dict(shards=[rng.integers(0, 256, size=(sh.shape[0], rows[1]), dtype=np.uint8)
                          for sh in inst.shards], row_bytes=rows[0], stride=rows[1])
    seq = world(inst, n_hot=n_hot, W=W, delta=True, **kw)
    W = seq.W
    rb = seq.row_bytes
    dev = seq.dev
    shards = seq.shards_d
    if host:
        shards = [s if m == wl.local_owner else s.cpu().pin_memory()
                  for m, s in enumerate(seq.shards_d)]
    look = LookaheadPipeline(seq.row_ptr_d, seq.col_idx_d, wl.num_parts, wl.part_kind,
                             wl.local_owner, inst.range_start, shards,
                             [s.shape[0] for s in inst.shards], rb, seq.stride, W,
                             wl.fanout, wl.batch_size, n_hot=n_hot, device=dev, nsets=nsets,
                             stage_apart=True if apart else None)
    assert look.stage_apart == (host or apart)
    assert (look.stage_stream is look.fetch_stream) == look.stage_apart
    assert (look.gather_stream is look.fetch_stream) != look.stage_apart
    nsets = look.nsets
    mk = lambda: T.cuda.Event(enable_timing=True)  # noqa: E731
    seeds_d = T.from_numpy(inst.seeds).to(dev)
    boff = inst.batch_off
    nwin = synth.n_windows(boff, W)
    L = len(wl.fanout)
    expected = []
    for k in range(nwin):
        r = seq.run_and_compare(k)
        expected.append((np.concatenate(r["outs"])[:, :rb], r["stage"]))

    def read(k, Wk, bufs):
        look.gathered_event(k).synchronize()
        foff = bufs.frontier_off[:(L + 1) * Wk + 1].cpu().numpy()
        n = int(foff[-1] - foff[L * Wk])
        return bufs.win_out[:n, :rb].cpu().numpy(), bufs.stage_stats_dict()

    got, pending = [], None
    for k in range(nwin):
        b0, b1 = synth.window_batches(boff, W, k)
        ge = None if gev is None else (None if gev == "end" else mk(), mk())
        # the seeds were uploaded on the caller's stream, which only the
        # first window has to wait for
        Wk, bufs = look.window(seeds_d[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0], b0,
                               gather_events=ge, after_caller=k == 0)
        if ge is not None:
            assert (look.gathered_event(k) is ge[1])
        if pending is not None:                 # read window k-1 while k is in flight
            got.append(read(*pending))
        pending = (k, Wk, bufs)
    got.append(read(*pending))
    assert look.read_status() == 0
    assert len(got) == nwin
    for k in range(nwin):
        assert np.array_equal(got[k][0], expected[k][0]), f"window {k} rows"
        # each buffer set's remap is cleared of the window nsets back, so the
        # cleared-entry count differs from the one-remap driver's
        g_st, e_st = dict(got[k][1]), dict(expected[k][1])
        assert g_st.pop("invalidated") == (expected[k - nsets][1]["rows_total"]
                                           if k >= nsets else 0)
        e_st.pop("invalidated")
        assert g_st == e_st, f"window {k} staging statistics"


def _oracle_trace(inst):
    """The epoch's N_b from the oracle sampler, batch by batch (N_b does not
    depend on W)."""
    from oracle import ggref
    wl = inst.wl
    L = len(wl.fanout)
    boff = inst.batch_off
    nb = boff.shape[0] - 1
    ids, off = [], [0]
    for b0 in range(0, nb, 4):
        b1 = min(nb, b0 + 4)
        so = boff[b0:b1 + 1] - boff[b0]
        fids, foff, _, _ = ggref.sample_window(inst.row_ptr, inst.col_idx,
                                               inst.seeds[boff[b0]:boff[b1]], so, wl.fanout,
                                               0, 0, b0)
        Wk = b1 - b0
        for b in range(Wk):
            s = L * Wk + b
            ids.append(fids[foff[s]:foff[s + 1]])
            off.append(off[-1] + int(foff[s + 1] - foff[s]))
    return np.concatenate(ids).astype(np.int32), np.array(off, np.int64)


SIM_COEF = dict(eps_init=0.025, eps_row=1.6e-5, lam_init=5e-4, lam_row=3.2e-7,
                bw_bytes_per_s=1.25e9, row_bytes=400.0, p_idle=30.0)


@pytest.mark.parametrize("name,W,n_hot,driver,frac", [
    ("tiny", 1, -1, "seq", None), ("tiny", 2, 2000, "seq", None), ("tiny", 4, 0, "seq", None),
    ("small", 1, 3000, "seq", None), ("small", 4, 3000, "delta", None),
    ("small", 8, -1, "seq", None), ("small", 3, 0, "seq", None),
    ("small", 4, 3000, "lookahead", None), ("small", 2, 20000, "lookahead", None),
    ("small", 4, -1, "seq", (1, 10)), ("small", 16, -1, "lookahead", (1, 10)),
    ("tiny", 3, -1, "seq", (7, 9)), ("small", 1, -1, "delta", (0, 5))])
def test_simulator_counts_match_oracle(name, W, n_hot, driver, frac):
    log(f"{name}: simulator z(W), E_phy(W) over the epoch, W={W}, n_hot={n_hot}, {driver}, "
        f"relative budget {frac}")
    import torch as T
    from oracle import ggref
    from paper_2606_02916_amd import LookaheadPipeline, gg
    inst = synth.instance(name)
    wl = inst.wl
    w = world(inst, W=W, n_hot=n_hot, delta=driver == "delta", hot_frac=frac)
    P = wl.num_parts
    coeffs = gg.make_sim_coeffs(P, **SIM_COEF)
    acc = T.zeros(gg.SIM_ACC_BYTES, dtype=T.uint8, device=w.dev)
    boff = inst.batch_off
    nwin = synth.n_windows(boff, W)
    seeds_d = T.from_numpy(inst.seeds).to(w.dev)
    if driver == "lookahead":
        pipe = LookaheadPipeline(w.row_ptr_d, w.col_idx_d, P, wl.part_kind, wl.local_owner,
                                 inst.range_start, w.shards_d, [s.shape[0] for s in inst.shards],
                                 wl.row_bytes, wl.row_stride, W, wl.fanout, wl.batch_size,
                                 n_hot=n_hot, device=w.dev, hot_frac=frac)
    else:
        pipe = w.pipe
    for k in range(nwin):
        b0, b1 = synth.window_batches(boff, W, k)
        pipe.window(seeds_d[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0], b0,
                    sim=(coeffs, acc))
    assert pipe.read_status() == 0
    T.cuda.synchronize()
    got = gg.sim_acc_from_bytes(acc.cpu().numpy().tobytes())
    ids, off = _oracle_trace(inst)
    part = ggref.make_part(P, wl.part_kind, wl.local_owner, wl.num_nodes, inst.range_start)
    ref = ggref.simulate_epoch(ids, off, W, n_hot, part, ggref.sim_coeffs(P, **SIM_COEF),
                               hot_frac=frac)
    # integer counts exactly; the fp64 energies are formed in the same order
    # without fused multiply-adds on both sides, so they agree bit for bit
    assert got == ref
    if n_hot == 0 or (frac is not None and frac[0] == 0):
        assert got["rebuild_events"] == 0 and got["hits"] == 0
    if n_hot < 0 and frac is None:
        assert got["miss_events"] == 0


def _sage_layers(rng, dims):
    """Random GraphSAGE weights, scaled by 1/sqrt(d_in); ReLU on all but the
    last layer."""
    L = len(dims) - 1
    return [((rng.standard_normal((dims[j], dims[j + 1])) / np.sqrt(dims[j])).astype(np.float32),
             (rng.standard_normal((dims[j], dims[j + 1])) / np.sqrt(dims[j])).astype(np.float32),
             (0.1 * rng.standard_normal(dims[j + 1])).astype(np.float32), j < L - 1)
            for j in range(L)]


def _sage_tolerance(layers, fanout, ab):
    """Rounding bound of the fp32 kernels against the fp64 oracle: per layer
    at most K + k + 5 roundings (a K-term product, a mean of up to k rows,
    the reciprocal and its product, the self term and the bias), each of
    relative size 2^-24 of the magnitudes the absolute-value pass bounds;
    doubled for second-order terms."""
    L = len(layers)
    n = sum(layers[j][0].shape[0] + fanout[L - 1 - j] + 5 for j in range(L))
    return 2.0 * n * 2.0 ** -24 * ab


def _run_consumer(w, layers, x_dtype, stride, Wk):
    import torch as T
    from paper_2606_02916_amd import SageConsumer
    lt = [(T.from_numpy(a).to(w.dev), T.from_numpy(b).to(w.dev), T.from_numpy(c).to(w.dev), r)
          for a, b, c, r in layers]
    cons = SageConsumer(w.pipe.geo, lt, x_dtype=x_dtype, device=w.dev)
    out = cons.forward(w.pipe.buf, Wk, w.pipe.win_out, stride, w.pipe.status)
    T.cuda.synchronize()
    assert w.pipe.read_status() == 0
    return out.cpu().numpy()


@pytest.mark.parametrize("name,hidden,fp16,W", [
    ("tiny", [16, 41], False, None), ("small", [16, 16, 47], False, None),
    ("tiny", [128, 7], True, None), ("small", [40, 100, 3], False, 2),
    ("tiny", [1, 1], False, 1)])
def test_sage_consumer_matches_oracle(name, hidden, fp16, W):
    log(f"{name}: GraphSAGE consumer, dims {hidden}, fp16={fp16}, W={W}")
    from oracle import ggref
    inst = synth.instance(name)
    wl = inst.wl
    kw = {}
    d_in = wl.feat_dim
    stride = wl.row_stride
    if fp16:   # the same values rounded to fp16, 2-byte elements
        kw["shards"] = [np.ascontiguousarray(
            s[:, :wl.row_bytes].view(np.float32).astype(np.float16)).view(np.uint8)
            for s in inst.shards]
        kw["row_bytes"] = kw["stride"] = stride = 2 * d_in
    w = world(inst, W=W, **kw)
    r = w.run_and_compare(0)
    Wk, fan = r["Wk"], list(wl.fanout)
    rng = np.random.default_rng(len(hidden) * 100 + hidden[0])
    layers = _sage_layers(rng, [d_in] + hidden)
    x = np.concatenate(r["outs"])          # the oracle's own gathered rows
    dt = 1 if fp16 else 0
    ref, ab = ggref.sage_forward(r["fids"], r["foff"], r["nids"], r["noff"], Wk, fan, x, dt,
                                 stride, layers)
    got = _run_consumer(w, layers, dt, stride, Wk)[:ref.shape[0]]
    tol = _sage_tolerance(layers, fan, ab)
    err = np.abs(got.astype(np.float64) - ref)
    assert np.all(err <= tol), (float(np.max(err - tol)), float(np.max(err)))
    assert ref.shape[0] == int(r["foff"][Wk] - r["foff"][0])


@pytest.mark.timeout(900)
def test_sage_consumer_large_sparse_window_sampled_batches():
    """The consumer over a whole 16-batch window of the 2.45M-node graph, as
    the benchmark lays it out; the oracle recomputes two of the batches from
    its own sampling and the feature shards."""
    log("large_sparse: GraphSAGE consumer over a full window, batches 0 and 11 checked")
    import torch as T
    from oracle import ggref
    inst = synth.instance("large_sparse")
    wl = inst.wl
    w = world(inst)
    pipe, dev = w.pipe, w.dev
    boff = inst.batch_off
    b0, b1 = synth.window_batches(boff, wl.W, 3)
    seeds_d = T.from_numpy(inst.seeds[boff[b0]:boff[b1]]).to(dev)
    Wk = pipe.window(seeds_d, boff[b0:b1 + 1] - boff[b0], b0)
    rng = np.random.default_rng(7)
    layers = _sage_layers(rng, [wl.feat_dim, 16, 16, 47])
    from paper_2606_02916_amd import SageConsumer
    lt = [(T.from_numpy(a).to(dev), T.from_numpy(b).to(dev), T.from_numpy(c).to(dev), r_)
          for a, b, c, r_ in layers]
    cons = SageConsumer(pipe.geo, lt, device=dev)
    out = cons.forward(pipe.buf, Wk, pipe.win_out, wl.row_stride, pipe.status)
    T.cuda.synchronize()
    assert pipe.read_status() == 0
    foff_g = pipe.frontier_off[:(len(wl.fanout) + 1) * Wk + 1].cpu().numpy()
    got_all = out.cpu().numpy()
    part = ggref.make_part(wl.num_parts, wl.part_kind, wl.local_owner, wl.num_nodes,
                           inst.range_start)
    L = len(wl.fanout)
    for b in (0, 11):
        g = b0 + b
        so = np.array([0, boff[g + 1] - boff[g]], np.int64)
        fids, foff, nids, noff = ggref.sample_window(inst.row_ptr, inst.col_idx,
                                                     inst.seeds[boff[g]:boff[g + 1]], so,
                                                     wl.fanout, 0, 0, g)
        ids = fids[foff[L]:foff[L + 1]]
        x = np.stack([inst.shards[ggref.owner(part, int(u))][ggref.row(part, int(u))]
                      for u in ids])
        ref, ab = ggref.sage_forward(fids, foff, nids, noff, 1, wl.fanout, x, 0, wl.row_stride,
                                     layers)
        got = got_all[foff_g[b] - foff_g[0]:foff_g[b + 1] - foff_g[0]]
        assert got.shape == ref.shape
        tol = _sage_tolerance(layers, list(wl.fanout), ab)
        assert np.all(np.abs(got.astype(np.float64) - ref) <= tol), b
