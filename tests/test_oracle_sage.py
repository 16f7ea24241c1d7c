"""Pins of the oracle's GraphSAGE consumer (mean aggregator) over sampled
blocks: a hand-worked path, and the special case that reduces to dense
full-graph GraphSAGE (fan-out above every degree samples every neighbour,
so the seeds' outputs equal the whole-graph layer equations evaluated with
numpy matrix products)."""
import numpy as np
import pytest

from oracle import ggref
from tests import helpers


def _window(row_ptr, col_idx, seeds_per_batch, fanout, batch0=0):
    seeds = np.concatenate([np.asarray(s, np.int32) for s in seeds_per_batch])
    off = np.concatenate([[0], np.cumsum([len(s) for s in seeds_per_batch])]).astype(np.int64)
    return ggref.sample_window(row_ptr, col_idx, seeds, off, fanout, 7, 0, batch0)


def _x_rows(fids, foff, W, L, feats, dtype):
    """The window's N_b rows back to back, as the gather lays them out."""
    ids = fids[foff[L * W]:foff[(L + 1) * W]]
    vals = feats[ids].astype(np.float16 if dtype == 1 else np.float32)
    return np.ascontiguousarray(vals).view(np.uint8), vals.dtype.itemsize * feats.shape[1]


def test_hand_worked_path():
    # Path 0 - 1 - 2, one batch with seed 1, one layer with 1x1 identity
    # weights: out(1) = x1 + mean(x0, x2) = 10 + (1 + 100) / 2 = 60.5.
    rp, ci = helpers.csr_from_edges(3, [(0, 1), (1, 0), (1, 2), (2, 1)])
    fids, foff, nids, noff = _window(rp, ci, [[1]], [5])
    feats = np.array([[1.0], [10.0], [100.0]])
    x, st = _x_rows(fids, foff, 1, 1, feats, 0)
    one, zero = np.ones((1, 1)), np.zeros(1)
    out, ab = ggref.sage_forward(fids, foff, nids, noff, 1, [5], x, 0, st,
                                 [(one, one, zero, False)])
    assert out.tolist() == [[60.5]] and ab.tolist() == [[60.5]]
    # W_neigh = -1 and a bias of 2: 10 - 50.5 + 2 = -38.5, and ReLU gives 0
    out, ab = ggref.sage_forward(fids, foff, nids, noff, 1, [5], x, 0, st,
                                 [(one, -one, 2 * np.ones(1), True)])
    assert out.tolist() == [[0.0]] and ab.tolist() == [[62.5]]
    # an isolated seed aggregates nothing: out = x_self
    rp, ci = helpers.csr_from_edges(2, [])
    fids, foff, nids, noff = _window(rp, ci, [[1]], [3])
    x, st = _x_rows(fids, foff, 1, 1, np.array([[0.0], [4.0]]), 0)
    out, _ = ggref.sage_forward(fids, foff, nids, noff, 1, [3], x, 0, st,
                                [(one, 5 * one, zero, False)])
    assert out.tolist() == [[4.0]]


def _dense_sage(row_ptr, col_idx, feats, layers):
    """Whole-graph GraphSAGE with the mean aggregator: H' = act(H Ws +
    D^-1 A H Wn + b), A counting multi-edges and self loops, rows of
    isolated nodes aggregating zero."""
    N = row_ptr.shape[0] - 1
    A = np.zeros((N, N))
    for u in range(N):
        for v in col_idx[row_ptr[u]:row_ptr[u + 1]]:
            A[u, v] += 1
    deg = A.sum(axis=1)
    Dinv = np.where(deg > 0, 1.0 / np.maximum(deg, 1), 0.0)
    H = feats.astype(np.float64)
    for ws, wn, b, relu in layers:
        H = H @ ws.astype(np.float64) + (Dinv[:, None] * (A @ H)) @ wn.astype(np.float64) + b
        if relu:
            H = np.maximum(H, 0)
    return H


@pytest.mark.parametrize("L,dtype", [(1, 0), (2, 0), (3, 0), (2, 1)])
def test_full_fanout_equals_dense_graphsage(L, dtype):
    rng = np.random.default_rng(10 + L + dtype)
    N = 60
    row_ptr, col_idx = helpers.random_graph(N, 240, rng)      # with self loops / multi-edges
    maxdeg = int(np.max(np.diff(row_ptr)))
    fanout = [maxdeg] * L
    dims = [7, 5, 6, 3][:L + 1]
    layers = [(rng.standard_normal((dims[j], dims[j + 1])).astype(np.float32),
               rng.standard_normal((dims[j], dims[j + 1])).astype(np.float32),
               rng.standard_normal(dims[j + 1]).astype(np.float32), j < L - 1) for j in range(L)]
    # fp16-exact values for the fp16 case
    feats = np.round(rng.standard_normal((N, dims[0])) * 8) / 8
    batches = [rng.choice(N, size=4, replace=False) for _ in range(3)]
    fids, foff, nids, noff = _window(row_ptr, col_idx, batches, fanout)
    x, st = _x_rows(fids, foff, 3, L, feats, dtype)
    out, ab = ggref.sage_forward(fids, foff, nids, noff, 3, fanout, x, dtype, st, layers)
    ref = _dense_sage(row_ptr, col_idx, feats, layers)
    seeds = fids[foff[0]:foff[3]]
    np.testing.assert_allclose(out, ref[seeds], rtol=1e-12, atol=1e-12)
    assert np.all(np.abs(out) <= ab * (1 + 1e-12))


def test_zero_weights_give_the_bias():
    rng = np.random.default_rng(3)
    row_ptr, col_idx = helpers.random_graph(40, 200, rng)
    fids, foff, nids, noff = _window(row_ptr, col_idx, [[1, 2, 3], [4]], [3, 2])
    x, st = _x_rows(fids, foff, 2, 2, rng.standard_normal((40, 4)), 0)
    z = lambda a, b: np.zeros((a, b), np.float32)   # noqa: E731
    b2 = np.array([-1.0, 2.0], np.float32)
    out, ab = ggref.sage_forward(fids, foff, nids, noff, 2, [3, 2], x, 0, st,
                                 [(z(4, 3), z(4, 3), np.ones(3), True), (z(3, 2), z(3, 2), b2, True)])
    assert out.shape == (4, 2) and np.all(out == [0.0, 2.0]) and np.all(ab == [1.0, 2.0])


def test_argument_checks():
    rp, ci = helpers.csr_from_edges(3, [(0, 1), (1, 0)])
    fids, foff, nids, noff = _window(rp, ci, [[1]], [2])
    x, st = _x_rows(fids, foff, 1, 1, np.ones((3, 2)), 0)
    w = np.ones((2, 2), np.float32)
    with pytest.raises(ggref.OracleError):            # d_in of layer 2 != d_out of layer 1
        ggref.sage_forward(fids, foff, nids, noff, 1, [2, 2], x, 0, st,
                           [(w, w, np.zeros(2), True), (np.ones((3, 1)), np.ones((3, 1)),
                                                        np.zeros(1), False)])
    with pytest.raises(ggref.OracleError):            # stride shorter than a row
        ggref.sage_forward(fids, foff, nids, noff, 1, [2], x, 0, 4, [(w, w, np.zeros(2), False)])
