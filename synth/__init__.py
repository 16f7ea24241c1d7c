"""Seeded synthetic workloads for the per-window feature-fetch path.

This package builds inputs only: R-MAT power-law graphs in CSR form, the
partition book, feature shards and the per-batch seed lists.  It holds none
of the method's arithmetic and is shared by the oracle side and the HIP side
of every test and benchmark.

The five workloads stand in for the paper's datasets (Reddit, OGBN-Products
and OGBN-Papers100M, Sec. VI-A), with their node and edge counts, on R-MAT
graphs with (a, b, c) = (0.57, 0.19, 0.19).
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# SYNTH_LIB lets the sanitizer test tier load an instrumented build.
LIB_PATH = os.environ.get("SYNTH_LIB") or os.path.join(_HERE, "libsynth.so")

PART_MOD = 0
PART_RANGE = 1
MASTER_SEED = 0

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"synthetic-input library not built: {LIB_PATH}")
        L = C.CDLL(LIB_PATH)
        P = C.c_void_p
        L.synth_permutation.argtypes = [C.c_int64, C.c_uint64, C.c_uint64, P]
        L.synth_permutation.restype = None
        L.synth_rmat_csr.argtypes = [C.c_int64, C.c_int64, C.c_double, C.c_double, C.c_double,
                                     C.c_uint64, C.c_int, P, P]
        L.synth_rmat_csr.restype = C.c_int
        L.synth_features.argtypes = [C.c_int64, C.c_int64, C.c_int32, C.c_int32, C.c_int32,
                                     C.c_int64, C.c_uint64, P]
        L.synth_features.restype = None
        _lib = L
    return _lib


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    num_nodes: int
    num_edges: int
    relabel: bool
    row_ptr_bits: int
    part_kind: int
    num_parts: int
    local_owner: int
    feat_dim: int
    feat_dtype: str          # "fp32" | "fp16"
    feat_dist: str           # "normal" | "uniform"
    fanout: tuple
    batch_size: int
    W: int
    seed_rule: str           # "perm_all" | "train_split" | "owner0"
    train_frac: float = 1.0
    n_windows: int = 0       # owner0 / perm_all: windows of seeds generated
    remote_on_host: bool = False

    @property
    def elem_bytes(self):
        return 4 if self.feat_dtype == "fp32" else 2

    @property
    def row_bytes(self):
        return self.feat_dim * self.elem_bytes

    @property
    def row_stride(self):
        return (self.row_bytes + 15) // 16 * 16

    def range_start(self):
        P, N = self.num_parts, self.num_nodes
        return [m * N // P for m in range(P)] + [N]


WORKLOADS = {
    # 10,000-node R-MAT, owners by node id mod 4, fp32 x 64, fanout [10,5],
    # batch 256, W = 4, one window.
    "tiny": Workload("tiny", 10_000, 100_000, False, 32, PART_MOD, 4, 0, 64, "fp32", "normal",
                     (10, 5), 256, 4, "perm_all", n_windows=1),
    # Reddit-shaped: 233,000 nodes, 114M edges, fp32 x 602, fanout [25,10],
    # batch 1024, W = 8, one epoch over a 66% training split.
    "dense_mid": Workload("dense_mid", 233_000, 114_000_000, True, 64, PART_RANGE, 4, 0, 602,
                          "fp32", "normal", (25, 10), 1024, 8, "train_split", train_frac=0.66),
    # OGBN-Products-shaped: 2.45M nodes, 62M edges, fp32 x 100 ~ U(-1,1),
    # fanout [15,10,5], batch 1024, W = 16, one epoch over an 8% split.
    "large_sparse": Workload("large_sparse", 2_450_000, 62_000_000, True, 64, PART_RANGE, 4, 0,
                             100, "fp32", "uniform", (15, 10, 5), 1024, 16, "train_split",
                             train_frac=0.08),
    # The same graph at batch 4096 for the window-size sweep.
    "wsweep": Workload("wsweep", 2_450_000, 62_000_000, True, 64, PART_RANGE, 4, 0, 100, "fp32",
                       "uniform", (15, 10, 5), 4096, 16, "train_split", train_frac=0.08),
    # One GPU's share of a 4-way split of a Papers100M-shaped graph:
    # 111M nodes, 1.6B edges, fp16 x 128; local shard in HBM, the three
    # remote shards in pinned host memory.
    "papers_share": Workload("papers_share", 111_000_000, 1_600_000_000, True, 64, PART_RANGE, 4,
                             0, 128, "fp16", "normal", (15, 10, 5), 1024, 16, "owner0",
                             n_windows=5, remote_on_host=True),
}

# A small graph for tests that must finish in seconds on the CPU oracle but
# still span several tiles and a ragged tail on the GPU.
WORKLOADS["small"] = Workload("small", 60_001, 700_000, True, 64, PART_RANGE, 4, 0, 100, "fp32",
                              "uniform", (15, 10, 5), 512, 4, "train_split", train_frac=0.2)


def rmat_csr(num_nodes, num_edges, seed=MASTER_SEED, relabel=True, row_ptr_bits=64,
             a=0.57, b=0.19, c=0.19):
    row_ptr = np.empty(num_nodes + 1, dtype=np.int64)
    col_idx = np.empty(num_edges, dtype=np.int32)
    rc = lib().synth_rmat_csr(num_nodes, num_edges, a, b, c, seed, int(relabel),
                              row_ptr.ctypes.data, col_idx.ctypes.data)
    if rc != 0:
        raise RuntimeError("R-MAT generation ran out of candidates")
    if row_ptr_bits == 32:
        assert num_edges < 2**31
        row_ptr = row_ptr.astype(np.int32)
    return row_ptr, col_idx


def permutation(n, seed, stream):
    out = np.empty(n, dtype=np.int64)
    lib().synth_permutation(n, seed, stream, out.ctypes.data)
    return out


def features(u_begin, u_end, dim, dtype, dist, stride, seed=MASTER_SEED, out=None):
    """Feature rows of nodes [u_begin, u_end) as a uint8 array (rows x stride)."""
    n = u_end - u_begin
    if out is None:
        out = np.empty((n, stride), dtype=np.uint8)
    assert out.shape == (n, stride) and out.flags.c_contiguous
    if n:
        lib().synth_features(u_begin, u_end, dim, 0 if dtype == "fp32" else 1,
                             0 if dist == "normal" else 1, stride, seed, out.ctypes.data)
    return out


def seed_batches(wl: Workload, epoch=0, seed=MASTER_SEED):
    """All seed batches of one epoch: (seeds int32, batch_off int64[n_batches+1])."""
    N, B = wl.num_nodes, wl.batch_size
    if wl.seed_rule == "perm_all":
        n = min(N, wl.n_windows * wl.W * B)
        seeds = permutation(N, seed, 11)[:n]
    elif wl.seed_rule == "train_split":
        n_train = int(wl.train_frac * N)
        train = permutation(N, seed, 11)[:n_train]
        order = permutation(n_train, seed, 1000 + epoch)
        seeds = train[order]
    elif wl.seed_rule == "owner0":
        lo, hi = wl.range_start()[0], wl.range_start()[1]
        n = min(hi - lo, wl.n_windows * wl.W * B)
        seeds = lo + permutation(hi - lo, seed, 11)[:n]
    else:
        raise ValueError(wl.seed_rule)
    n = seeds.shape[0]
    nb = (n + B - 1) // B
    off = np.minimum(np.arange(nb + 1, dtype=np.int64) * B, n)
    return seeds.astype(np.int32), off


def window_batches(batch_off, W, k):
    """Global batch range [b0, b1) of window k (the last window may be short)."""
    nb = batch_off.shape[0] - 1
    b0 = k * W
    return b0, min(nb, b0 + W)


def n_windows(batch_off, W):
    nb = batch_off.shape[0] - 1
    return (nb + W - 1) // W


@dataclasses.dataclass
class Instance:
    wl: Workload
    row_ptr: np.ndarray
    col_idx: np.ndarray
    seeds: np.ndarray
    batch_off: np.ndarray
    shards: list          # per owner: uint8 array (rows x stride)
    range_start: list


def shard_rows(wl: Workload, m):
    if wl.part_kind == PART_MOD:
        N, P = wl.num_nodes, wl.num_parts
        return (N - m + P - 1) // P
    rs = wl.range_start()
    return rs[m + 1] - rs[m]


def shard_features(wl: Workload, m, out=None):
    """Owner m's feature shard: rows in owner-local order."""
    stride = wl.row_stride
    if wl.part_kind == PART_RANGE:
        rs = wl.range_start()
        return features(rs[m], rs[m + 1], wl.feat_dim, wl.feat_dtype, wl.feat_dist, stride,
                        out=out)
    full = features(0, wl.num_nodes, wl.feat_dim, wl.feat_dtype, wl.feat_dist, stride)
    sh = np.ascontiguousarray(full[m::wl.num_parts])
    if out is not None:
        out[...] = sh
        return out
    return sh


def full_features(wl: Workload):
    """The unsharded feature matrix (row u = node u); ground truth for tests."""
    return features(0, wl.num_nodes, wl.feat_dim, wl.feat_dtype, wl.feat_dist, wl.row_stride)


_cache = {}
GEN_VERSION = 2


def _disk_cache(name, what, make):
    """Arrays of a workload, memoised under $SYNTH_CACHE_DIR when it is set
    (the generator is deterministic, so a cached copy equals a fresh one)."""
    d = os.environ.get("SYNTH_CACHE_DIR")
    if not d:
        return make()
    path = os.path.join(d, f"{name}.v{GEN_VERSION}.{what}.npz")
    if os.path.exists(path):
        with np.load(path) as z:
            return [z[k] for k in sorted(z.files, key=lambda k: int(k[1:]))]
    arrs = make()
    os.makedirs(d, exist_ok=True)
    tmp = path + ".tmp.npz"
    np.savez(tmp, **{f"a{i}": a for i, a in enumerate(arrs)})
    os.replace(tmp, path)
    return arrs


def _progress(msg):
    import sys
    import time
    print(f"[synth {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def instance(name, with_features=True, host_alloc=None):
    """Generates (or returns the memoised) workload `name`.

    host_alloc(m, rows, stride) -> uint8 array: when given, the shards of
    remote owners of a workload that keeps them in host memory are written
    straight into the arrays it returns (e.g. views of pinned host tensors).
    """
    key = (name, with_features, host_alloc is not None)
    if key in _cache:
        return _cache[key]
    wl = WORKLOADS[name]
    gname = "large_sparse" if name == "wsweep" else name
    big = wl.num_edges > 500_000_000
    if big:
        _progress(f"{name}: R-MAT {wl.num_nodes} nodes, {wl.num_edges} edges")
    make_csr = lambda: list(rmat_csr(wl.num_nodes, wl.num_edges, relabel=wl.relabel,  # noqa: E731
                                     row_ptr_bits=wl.row_ptr_bits))
    row_ptr, col_idx = make_csr() if big else _disk_cache(gname, "csr", make_csr)
    seeds, boff = seed_batches(wl)
    shards = []
    if with_features:
        if wl.remote_on_host and host_alloc is not None:
            for m in range(wl.num_parts):
                rows = shard_rows(wl, m)
                out = None if m == wl.local_owner else host_alloc(m, rows, wl.row_stride)
                if big:
                    _progress(f"{name}: features of owner {m} ({rows} rows)")
                shards.append(shard_features(wl, m, out=out))
        elif big:
            for m in range(wl.num_parts):
                _progress(f"{name}: features of owner {m}")
                shards.append(shard_features(wl, m))
        else:
            shards = _disk_cache(gname, "feat", lambda: [shard_features(wl, m)
                                                         for m in range(wl.num_parts)])
    if big:
        _progress(f"{name}: ready")
    inst = Instance(wl, row_ptr, col_idx, seeds, boff, shards,
                    wl.range_start() if wl.part_kind == PART_RANGE else None)
    _cache[key] = inst
    return inst


def torch_instance(name, device):
    """The workload with its CSR and feature shards as torch tensors:
    device tensors, except the remote shards of a workload that keeps them
    in host memory, which stay pinned host tensors (read by the GPU through
    their device address).  Returns (inst, row_ptr_d, col_idx_d, shards_d)."""
    import torch
    wl = WORKLOADS[name]
    pinned = {}

    def alloc(m, rows, stride):
        t = torch.empty((rows, stride), dtype=torch.uint8, pin_memory=True)
        pinned[m] = t
        return t.numpy()

    key = ("torch", name)
    if key in _cache:
        return _cache[key]
    inst = instance(name, host_alloc=alloc if wl.remote_on_host else None)
    if wl.remote_on_host and not pinned:
        raise RuntimeError("host-resident shards were generated without pinned memory")
    dev = torch.device(device)
    row_ptr_d = torch.from_numpy(inst.row_ptr).to(dev)
    col_idx_d = torch.from_numpy(inst.col_idx).to(dev)
    shards_d = [pinned[m] if m in pinned else torch.from_numpy(inst.shards[m]).to(dev)
                for m in range(wl.num_parts)]
    res = (inst, row_ptr_d, col_idx_d, shards_d)
    _cache[key] = res
    return res
