"""ctypes wrapper of the CPU oracle (``libggref.so``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``.  The product path never imports
this module.  All arrays are numpy arrays on the host.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

MAX_PARTS = 64
PART_MOD = 0
PART_RANGE = 1
ERR_CAPACITY = -2   # GGREF_ERR_CAPACITY

_HERE = os.path.dirname(os.path.abspath(__file__))
# GGREF_LIB lets the oracle's own mutation tests load a deliberately broken
# build of it; nothing else sets it.
LIB_PATH = os.environ.get("GGREF_LIB") or os.path.join(_HERE, "libggref.so")


class Csr(C.Structure):
    _fields_ = [("num_nodes", C.c_int64), ("num_edges", C.c_int64), ("row_ptr", C.c_void_p),
                ("row_ptr_bits", C.c_int32), ("pad_", C.c_int32), ("col_idx", C.c_void_p)]


class Part(C.Structure):
    _fields_ = [("num_parts", C.c_int32), ("kind", C.c_int32), ("local_owner", C.c_int32),
                ("pad_", C.c_int32), ("num_nodes", C.c_int64),
                ("range_start", C.c_int64 * (MAX_PARTS + 1))]


class Feat(C.Structure):
    _fields_ = [("row_bytes", C.c_int32), ("num_parts", C.c_int32),
                ("shard", C.c_void_p * MAX_PARTS), ("row_stride", C.c_int64 * MAX_PARTS),
                ("shard_rows", C.c_int64 * MAX_PARTS)]


class StageStats(C.Structure):
    _fields_ = [("rows_total", C.c_int64), ("requests_total", C.c_int64),
                ("invalidated", C.c_int64), ("retained", C.c_int64),
                ("requests", C.c_int64 * MAX_PARTS), ("rows", C.c_int64 * MAX_PARTS),
                ("bytes", C.c_int64 * MAX_PARTS), ("delta_rows", C.c_int64 * MAX_PARTS)]


class GatherStats(C.Structure):
    _fields_ = [("rows", C.c_int64), ("local", C.c_int64), ("hits", C.c_int64),
                ("misses", C.c_int64), ("miss_requests", C.c_int64 * MAX_PARTS),
                ("miss_rows", C.c_int64 * MAX_PARTS)]


class SimCoeffs(C.Structure):
    _fields_ = [("eps_init", C.c_double * MAX_PARTS), ("eps_row", C.c_double * MAX_PARTS),
                ("lam_init", C.c_double * MAX_PARTS), ("lam_row", C.c_double * MAX_PARTS),
                ("bw_bytes_per_s", C.c_double), ("row_bytes", C.c_double),
                ("p_idle", C.c_double)]


class SimAcc(C.Structure):
    _fields_ = [("windows", C.c_int64), ("batches", C.c_int64),
                ("rebuild_events", C.c_int64), ("rebuild_rows", C.c_int64),
                ("miss_events", C.c_int64), ("miss_rows", C.c_int64),
                ("remote_rows", C.c_int64), ("hits", C.c_int64),
                ("e_rebuild", C.c_double), ("e_miss", C.c_double), ("t_stall", C.c_double),
                ("e_stall", C.c_double), ("e_phy", C.c_double)]


class SageLayer(C.Structure):
    _fields_ = [("d_in", C.c_int32), ("d_out", C.c_int32), ("relu", C.c_int32),
                ("w_self", C.c_void_p), ("w_neigh", C.c_void_p), ("bias", C.c_void_p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"oracle library not built: {LIB_PATH}")
        L = C.CDLL(LIB_PATH)
        P = C.c_void_p
        i64, i32, u64 = C.c_int64, C.c_int32, C.c_uint64
        L.ggref_philox4x32_10.argtypes = [P, P, P]
        L.ggref_philox4x32_10.restype = None
        L.ggref_bounded.argtypes = [C.c_uint32, u64]
        L.ggref_bounded.restype = u64
        L.ggref_floyd.argtypes = [i64, i32, P, P]
        L.ggref_floyd.restype = C.c_int
        L.ggref_owner.argtypes = [P, i64]
        L.ggref_owner.restype = i32
        L.ggref_row.argtypes = [P, i64]
        L.ggref_row.restype = i64
        L.ggref_sample_window.argtypes = [P, P, P, i32, P, i32, u64, i32, i64, P, i64, P, P,
                                          i64, P, P]
        L.ggref_sample_window.restype = C.c_int
        L.ggref_build_hotset.argtypes = [P, P, i32, i32, P, i64, i64, i64, P, P, i64, P]
        L.ggref_build_hotset.restype = C.c_int
        L.ggref_bucket_by_owner.argtypes = [P, i64, P, P, P]
        L.ggref_bucket_by_owner.restype = C.c_int
        L.ggref_stage_bulk.argtypes = [P, P, P, P, P, i64, i64, P, P, i64, P, P, P]
        L.ggref_stage_bulk.restype = C.c_int
        L.ggref_stage_inplace.argtypes = [P, P, P, P, P, i64, i64, P, P, i64, P, P]
        L.ggref_stage_inplace.restype = C.c_int
        L.ggref_gather_batch.argtypes = [P, i64, P, P, P, i64, i64, P, P, i64, P]
        L.ggref_gather_batch.restype = C.c_int
        L.ggref_simulate_epoch.argtypes = [P, P, i64, i32, i64, i64, i64, P, P, P]
        L.ggref_simulate_epoch.restype = C.c_int
        L.ggref_sage_forward.argtypes = [P, P, P, P, i32, i32, P, P, i32, i64, P, P, P]
        L.ggref_sage_forward.restype = C.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


class OracleError(RuntimeError):
    pass


def _check(rc, what):
    if rc != 0:
        raise OracleError(f"{what} failed with code {rc}")


def make_part(num_parts, kind, local_owner, num_nodes, range_start=None):
    p = Part()
    p.num_parts = num_parts
    p.kind = kind
    p.local_owner = local_owner
    p.num_nodes = num_nodes
    if range_start is not None:
        for i, v in enumerate(range_start):
            p.range_start[i] = int(v)
    return p


def make_feat(row_bytes, shards, strides):
    """shards: list of 2-D uint8 views (rows x stride bytes), one per owner."""
    f = Feat()
    f.row_bytes = row_bytes
    f.num_parts = len(shards)
    for m, (s, st) in enumerate(zip(shards, strides)):
        f.shard[m] = s.ctypes.data if s.size else None
        f.row_stride[m] = st
        f.shard_rows[m] = s.shape[0]
    return f


def make_csr(row_ptr, col_idx):
    g = Csr()
    g.num_nodes = row_ptr.shape[0] - 1
    g.num_edges = col_idx.shape[0]
    g.row_ptr = row_ptr.ctypes.data
    g.row_ptr_bits = 64 if row_ptr.dtype == np.int64 else 32
    g.col_idx = col_idx.ctypes.data
    return g


def philox(ctr, key):
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().ggref_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def bounded(r, bound):
    return int(lib().ggref_bounded(int(r), int(bound)))


def floyd(d, k, t):
    t = np.ascontiguousarray(t, dtype=np.int64)
    pos = np.zeros(k, dtype=np.int64)
    _check(lib().ggref_floyd(d, k, _p(t), _p(pos)), "ggref_floyd")
    return pos


def owner(part, u):
    return int(lib().ggref_owner(C.byref(part), int(u)))


def row(part, u):
    return int(lib().ggref_row(C.byref(part), int(u)))


def sample_window(row_ptr, col_idx, seeds, seed_off, fanout, rng_seed, epoch, batch0,
                  frontier_cap=None, nbr_cap=None):
    """Returns (frontier_ids, frontier_off, nbr_ids, nbr_off) as numpy arrays."""
    g = make_csr(row_ptr, col_idx)
    seeds = np.ascontiguousarray(seeds, dtype=np.int32)
    seed_off = np.ascontiguousarray(seed_off, dtype=np.int64)
    fan = np.ascontiguousarray(fanout, dtype=np.int32)
    W = seed_off.shape[0] - 1
    L = fan.shape[0]
    need = np.zeros(2, dtype=np.int64)
    fcap = 0 if frontier_cap is None else frontier_cap
    ncap = 0 if nbr_cap is None else nbr_cap
    for _ in range(2):
        fids = np.zeros(max(fcap, 1), dtype=np.int32)
        foff = np.zeros((L + 1) * W + 1, dtype=np.int64)
        nids = np.zeros(max(ncap, 1), dtype=np.int32)
        noff = np.zeros(L * W + 1, dtype=np.int64)
        rc = lib().ggref_sample_window(C.byref(g), _p(seeds), _p(seed_off), W, _p(fan), L,
                                       C.c_uint64(rng_seed), epoch, batch0, _p(fids), fcap,
                                       _p(foff), _p(nids), ncap, _p(noff), _p(need))
        if rc == -2 and frontier_cap is None and nbr_cap is None:
            fcap, ncap = int(need[0]), int(need[1])
            continue
        _check(rc, "ggref_sample_window")
        return fids[:need[0]], foff, nids[:need[1]], noff
    raise OracleError("sample_window capacity loop")


def build_hotset(frontier_ids, frontier_off, W, L, part, n_hot=-1, hot_frac=None):
    """hot_frac = (num, den): the top ceil(U * num / den) of the window's U
    distinct remote nodes (n_hot must then be -1)."""
    num, den = hot_frac if hot_frac is not None else (0, 0)
    cap = max(1, int(frontier_ids.shape[0]))
    hot = np.zeros(cap, dtype=np.int32)
    freq = np.zeros(cap, dtype=np.int32)
    cnt = np.zeros(1, dtype=np.int64)
    fids = np.ascontiguousarray(frontier_ids, dtype=np.int32)
    foff = np.ascontiguousarray(frontier_off, dtype=np.int64)
    _check(lib().ggref_build_hotset(_p(fids), _p(foff), W, L, C.byref(part), n_hot, num, den,
                                    _p(hot), _p(freq), cap, _p(cnt)), "ggref_build_hotset")
    n = int(cnt[0])
    return hot[:n], freq[:n]


def bucket_by_owner(hot_ids, part):
    hot_ids = np.ascontiguousarray(hot_ids, dtype=np.int32)
    out = np.zeros(max(1, hot_ids.shape[0]), dtype=np.int32)
    off = np.zeros(part.num_parts + 1, dtype=np.int64)
    _check(lib().ggref_bucket_by_owner(_p(hot_ids), hot_ids.shape[0], C.byref(part), _p(out),
                                       _p(off)), "ggref_bucket_by_owner")
    return out[:hot_ids.shape[0]], off


def stage_bulk(bucket_ids, owner_off, part, feat, cache, cache_stride, slot_of, prev_ids=None,
               src_cache=None, src_slot_of=None):
    """cache: uint8 array (rows x cache_stride); slot_of: int32[N], updated
    in place.  prev_ids: remap entries to clear.  src_cache / src_slot_of:
    the cache rows may be taken from (delta staging)."""
    st = StageStats()
    bucket_ids = np.ascontiguousarray(bucket_ids, dtype=np.int32)
    owner_off = np.ascontiguousarray(owner_off, dtype=np.int64)
    prev = None if prev_ids is None else np.ascontiguousarray(prev_ids, dtype=np.int32)
    npre = 0 if prev is None else prev.shape[0]
    _check(lib().ggref_stage_bulk(_p(bucket_ids), _p(owner_off), C.byref(part), C.byref(feat),
                                  _p(cache), cache_stride, cache.shape[0], _p(slot_of), _p(prev),
                                  npre, _p(src_cache), _p(src_slot_of), C.byref(st)),
           "ggref_stage_bulk")
    return stats_dict(st, part.num_parts)


def stage_inplace(bucket_ids, owner_off, part, feat, cache, cache_stride, slot_of, prev_slot_of,
                  clear_ids=None, allow_short=False):
    """Delta staging into one persistent cache: cache (rows x cache_stride,
    uint8) and slot_of (int32[N], this window's remap) are updated in place;
    prev_slot_of is the previous window's remap (None for a first window);
    clear_ids: entries of slot_of to clear first.  When the free slots run
    out the call raises, unless allow_short: it then returns (stats, True)
    with the delta rows left over uncached, and (stats, False) otherwise."""
    st = StageStats()
    bucket_ids = np.ascontiguousarray(bucket_ids, dtype=np.int32)
    owner_off = np.ascontiguousarray(owner_off, dtype=np.int64)
    clr = None if clear_ids is None else np.ascontiguousarray(clear_ids, dtype=np.int32)
    ncl = 0 if clr is None else clr.shape[0]
    rc = lib().ggref_stage_inplace(_p(bucket_ids), _p(owner_off), C.byref(part), C.byref(feat),
                                   _p(cache), cache_stride, cache.shape[0], _p(slot_of),
                                   _p(clr), ncl, _p(prev_slot_of), C.byref(st))
    short = rc == ERR_CAPACITY
    if not (allow_short and short):
        _check(rc, "ggref_stage_inplace")
    d = stats_dict(st, part.num_parts)
    return (d, short) if allow_short else d


def gather_batch(in_ids, part, feat, cache, cache_stride, slot_of, out, out_stride):
    gs = GatherStats()
    in_ids = np.ascontiguousarray(in_ids, dtype=np.int32)
    _check(lib().ggref_gather_batch(_p(in_ids), in_ids.shape[0], C.byref(part), C.byref(feat),
                                    _p(cache), cache_stride, cache.shape[0], _p(slot_of), _p(out),
                                    out_stride, C.byref(gs)), "ggref_gather_batch")
    return stats_dict(gs, part.num_parts)


def sim_coeffs(P, eps_init, eps_row, lam_init, lam_row, bw_bytes_per_s, row_bytes, p_idle):
    """Coefficients of the analytical model; per-owner terms are scalars
    (the same for every owner) or sequences of P values."""
    c = SimCoeffs()
    for name, v in (("eps_init", eps_init), ("eps_row", eps_row), ("lam_init", lam_init),
                    ("lam_row", lam_row)):
        vals = list(v) if hasattr(v, "__len__") else [v] * P
        arr = getattr(c, name)
        for m in range(P):
            arr[m] = float(vals[m])
    c.bw_bytes_per_s, c.row_bytes, c.p_idle = float(bw_bytes_per_s), float(row_bytes), float(p_idle)
    return c


def simulate_epoch(trace_ids, trace_off, W, n_hot, part, coeffs, hot_frac=None):
    """The trace simulator for window size W over the epoch's N_b (batch b
    at trace_ids[trace_off[b]:trace_off[b+1]], ascending): event counts and
    the energies of Eqs. (1)-(3)."""
    num, den = hot_frac if hot_frac is not None else (0, 0)
    ids = np.ascontiguousarray(trace_ids, dtype=np.int32)
    off = np.ascontiguousarray(trace_off, dtype=np.int64)
    acc = SimAcc()
    _check(lib().ggref_simulate_epoch(_p(ids), _p(off), off.shape[0] - 1, W, n_hot, num, den,
                                      C.byref(part), C.byref(coeffs), C.byref(acc)),
           "ggref_simulate_epoch")
    return sim_dict(acc)


def sage_forward(frontier_ids, frontier_off, nbr_ids, nbr_off, W, fanout, x, x_dtype, x_stride,
                 layers):
    """GraphSAGE (mean aggregator) over a window's sampled blocks.  x: the
    window's N_b rows back to back as a uint8 array of rows at x_stride
    bytes; x_dtype 0 = fp32, 1 = fp16; layers: list of (w_self [d_in, d_out],
    w_neigh, bias [d_out], relu).  Returns (out, out_abs) over the rows of
    F_0 of all batches."""
    L = len(fanout)
    fids = np.ascontiguousarray(frontier_ids, dtype=np.int32)
    foff = np.ascontiguousarray(frontier_off, dtype=np.int64)
    nids = np.ascontiguousarray(nbr_ids, dtype=np.int32)
    noff = np.ascontiguousarray(nbr_off, dtype=np.int64)
    fan = np.ascontiguousarray(fanout, dtype=np.int32)
    xb = np.ascontiguousarray(x)
    keep = []
    arr = (SageLayer * L)()
    for j, (ws, wn, b, relu) in enumerate(layers):
        ws = np.ascontiguousarray(ws, dtype=np.float32)
        wn = np.ascontiguousarray(wn, dtype=np.float32)
        b = np.ascontiguousarray(b, dtype=np.float32)
        keep += [ws, wn, b]
        arr[j].d_in, arr[j].d_out, arr[j].relu = ws.shape[0], ws.shape[1], int(bool(relu))
        arr[j].w_self, arr[j].w_neigh, arr[j].bias = ws.ctypes.data, wn.ctypes.data, b.ctypes.data
    n0 = int(foff[W] - foff[0])
    d = int(arr[L - 1].d_out)
    out = np.zeros((n0, d), dtype=np.float64)
    oab = np.zeros((n0, d), dtype=np.float64)
    _check(lib().ggref_sage_forward(_p(fids), _p(foff), _p(nids), _p(noff), W, L, _p(fan),
                                    _p(xb), x_dtype, x_stride, arr, _p(out), _p(oab)),
           "ggref_sage_forward")
    return out, oab


def sim_dict(acc):
    return {name: (float(getattr(acc, name)) if typ is C.c_double else int(getattr(acc, name)))
            for name, typ in acc._fields_}


def stats_dict(st, P):
    d = {}
    for name, typ in st._fields_:
        v = getattr(st, name)
        if name == "pad_":
            continue
        d[name] = [int(x) for x in v][:P] if hasattr(v, "__len__") else int(v)
    return d


def run_window(row_ptr, col_idx, seeds, seed_off, fanout, rng_seed, epoch, batch0, part, feat,
               cache, cache_stride, slot_of, prev_ids=None, n_hot=-1, out_stride=None,
               keep_outputs=True):
    """One window of the path, step by step: sample, hot set, owner buckets,
    bulk stage, then one gather per batch.  slot_of is updated in place;
    returns every intermediate (numpy arrays) and the per-batch outputs."""
    W = len(seed_off) - 1
    L = len(fanout)
    row_bytes = feat.row_bytes
    out_stride = out_stride or cache_stride
    fids, foff, nids, noff = sample_window(row_ptr, col_idx, seeds, seed_off, fanout, rng_seed,
                                           epoch, batch0)
    hot, freq = build_hotset(fids, foff, W, L, part, n_hot)
    bucket, owner_off = bucket_by_owner(hot, part)
    sst = stage_bulk(bucket, owner_off, part, feat, cache, cache_stride, slot_of, prev_ids)
    outs, gstats = [], []
    for b in range(W):
        s = L * W + b
        ids = fids[foff[s]:foff[s + 1]]
        out = np.zeros((ids.shape[0], out_stride), dtype=np.uint8)
        gstats.append(gather_batch(ids, part, feat, cache, cache_stride, slot_of, out,
                                   out_stride))
        outs.append(out if keep_outputs else None)
    return dict(frontier_ids=fids, frontier_off=foff, nbr_ids=nids, nbr_off=noff, hot_ids=hot,
                hot_freq=freq, bucket_ids=bucket, owner_off=owner_off, stage_stats=sst,
                outs=outs, gather_stats=gstats, row_bytes=row_bytes)
