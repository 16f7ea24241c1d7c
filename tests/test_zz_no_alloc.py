"""The no-allocation gather (gg_gather_batch_noalloc) against the workspace
gather (gg_gather_batch) through the C ABI, byte for byte: gathered rows and
per-batch statistics, on two calls in a row (a whole window with misses,
then a smaller one: a single batch with the look-ahead's flag), so the
second call runs on the scratch the first one left behind."""
import numpy as np
import pytest

import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def log(m):
    print(m, flush=True)


def test_noalloc_gather_matches_the_workspace_gather():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_02916_amd import gg
    from tests.gpu_util import World
    log("small: no-allocation gather against gg_gather_batch, two calls, the second smaller")
    w = World(synth.instance("small"), n_hot=3000)      # a budget: the miss path runs too
    r = w.run_and_compare(0)                             # the window, checked against the oracle
    p, Wk, L = w.pipe, r["Wk"], len(w.fanout)
    foff = r["foff"]
    rb, st = w.row_bytes, w.stride
    assert Wk >= 2
    calls = [(0, Wk, 0), (1, 1, gg.GG_GATHER_SHARED)]    # (first batch, batches, flags)
    misses = []
    for first, nseg, flags in calls:
        n = int(foff[L * Wk + first + nseg] - foff[L * Wk + first])
        log(f"batches {first}..{first + nseg - 1} ({n} rows), flags {flags}")
        bounds = p.frontier_off.data_ptr() + 8 * (L * Wk + first)
        outs, stats = [], []
        for fn in ("ws", "noalloc"):
            out = torch.full((n, st), 0xA5, dtype=torch.uint8, device=w.dev)
            stt = torch.full((nseg, gg.GATHER_STATS_BYTES), 0x5A, dtype=torch.uint8,
                             device=w.dev)
            args = (p.frontier_ids, bounds, nseg, n, p.part, p.feat, p.staged_cache(),
                    p.cache_stride, p.cache_rows, p.slot_of, out, st, stt.data_ptr(), p.status)
            if fn == "ws":
                gg.gg_gather_batch(*args, p.ws, flags=flags)
            else:
                gg.gg_gather_batch_noalloc(*args, flags=flags)
            torch.cuda.synchronize()
            assert p.read_status() == 0
            outs.append(out[:, :rb].cpu().numpy())
            stats.append([gg.gather_stats_from_bytes(stt[b].cpu().numpy().tobytes(), w.P)
                          for b in range(nseg)])
        assert np.array_equal(outs[1], outs[0])
        assert stats[1] == stats[0]
        # and the rows are the oracle's (run_and_compare kept them)
        want = np.concatenate([o[:, :rb] for o in r["outs"][first:first + nseg]])
        assert np.array_equal(outs[1], want)
        misses.append(sum(s_["misses"] for s_ in stats[1]))
    assert misses[0] > 0 and misses[1] > 0               # the finish kernel read the scratch
