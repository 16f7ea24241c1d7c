"""The README's example of driving the look-ahead pipeline, executed as
written on the large_sparse workload: in every window, every gathered row of
the first and the last batch must equal its node's row of the feature
matrix."""
import os
import textwrap

import numpy as np
import pytest

import synth
from tests import helpers

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _example():
    """The README's code block, from its imports to its status check, with
    a call to _check after the line that takes the window's rows."""
    text = open(os.path.join(helpers.ROOT, "README.md")).read()
    start = text.index("    import torch\n    from paper_2606_02916_amd import LookaheadPipeline")
    end = text.index("\n", text.index("look.read_status() == 0", start))
    lines = textwrap.dedent(text[start:end]).split("\n")
    at = next(i for i, ln in enumerate(lines) if ln.lstrip().startswith("x = bufs.win_out"))
    indent = lines[at][:len(lines[at]) - len(lines[at].lstrip())]
    lines.insert(at + 1, indent + "_check(k, Wk, bufs, off, x)")
    return "\n".join(lines)


def test_readme_example_runs_as_written():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print("large_sparse: the README's look-ahead example", flush=True)
    dev = torch.device("cuda:0")
    inst, row_ptr, col_idx, shards = synth.torch_instance("large_sparse", dev)
    wl = inst.wl
    assert (wl.num_parts, wl.local_owner, wl.row_bytes, wl.row_stride, wl.W, wl.batch_size) == \
        (4, 0, 400, 400, 16, 1024) and list(wl.fanout) == [15, 10, 5]
    seeds_d = torch.from_numpy(inst.seeds).to(dev)
    boff = inst.batch_off
    windows = []
    for k in range(synth.n_windows(boff, wl.W)):
        b0, b1 = synth.window_batches(boff, wl.W, k)
        windows.append((seeds_d[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0], b0))
    feats = np.concatenate(inst.shards)          # the range book's owners in id order
    seen = []

    def _check(k, Wk, bufs, off, x):
        fid = bufs.frontier_ids.cpu().numpy()
        for b in (0, Wk - 1):
            lo, hi = int(off[b] - off[0]), int(off[b + 1] - off[0])
            ids = fid[int(off[b]):int(off[b + 1])]
            assert hi > lo
            assert np.array_equal(x[lo:hi, :wl.row_bytes].cpu().numpy(),
                                  feats[ids, :wl.row_bytes]), (k, b)
        seen.append(k)

    ns = {"row_ptr": row_ptr, "col_idx": col_idx, "range_start": inst.range_start,
          "shards": shards, "windows": windows, "_check": _check}
    exec(compile(_example(), "README.md", "exec"), ns)
    assert seen == list(range(len(windows)))
