"""ctypes binding of libgg (include/gg.h): argument marshalling only.

Every function keeps the C name and argument order.  Device buffers are
torch tensors on a ROCm device (or pinned host tensors for shards kept in
host memory); they are passed by data pointer, and the stream defaults to
torch's current stream.  Every step of the path runs in libgg's kernels;
if the library is missing this module raises on import.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

MAX_PARTS = 64
MAX_LAYERS = 4
MAX_W = 64
MAX_FANOUT = 32
PART_MOD = 0
PART_RANGE = 1

GG_OK = 0
GG_ERR_ARG = 1
GG_ERR_CAPACITY = 2
GG_ERR_HIP = 3
GG_ERR_UNSUPPORTED = 4

GG_BUCKET_OWNER_ORDERED = 1
GG_GATHER_SHARED = 1

DEV_CAPACITY = 1
DEV_BAD_ID = 2
DEV_BAD_ROW = 4
DEV_BAD_DEGREE = 8
DEV_ORDER = 16

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgg.so")


class gg_csr_t(C.Structure):
    _fields_ = [("num_nodes", C.c_int64), ("num_edges", C.c_int64), ("row_ptr", C.c_void_p),
                ("row_ptr_bits", C.c_int32), ("pad_", C.c_int32), ("col_idx", C.c_void_p)]


class gg_part_t(C.Structure):
    _fields_ = [("num_parts", C.c_int32), ("kind", C.c_int32), ("local_owner", C.c_int32),
                ("pad_", C.c_int32), ("num_nodes", C.c_int64),
                ("range_start", C.c_int64 * (MAX_PARTS + 1))]


class gg_feat_t(C.Structure):
    _fields_ = [("row_bytes", C.c_int32), ("num_parts", C.c_int32),
                ("shard", C.c_void_p * MAX_PARTS), ("row_stride", C.c_int64 * MAX_PARTS),
                ("shard_rows", C.c_int64 * MAX_PARTS)]


class gg_wsample_t(C.Structure):
    _fields_ = [("frontier_ids", C.c_void_p), ("frontier_cap", C.c_int64),
                ("frontier_off", C.c_void_p), ("nbr_ids", C.c_void_p), ("nbr_cap", C.c_int64),
                ("nbr_off", C.c_void_p), ("frontier_bits", C.c_void_p), ("need", C.c_void_p)]


class gg_stage_stats_t(C.Structure):
    _fields_ = [("rows_total", C.c_int64), ("requests_total", C.c_int64),
                ("invalidated", C.c_int64), ("retained", C.c_int64),
                ("requests", C.c_int64 * MAX_PARTS), ("rows", C.c_int64 * MAX_PARTS),
                ("bytes", C.c_int64 * MAX_PARTS), ("delta_rows", C.c_int64 * MAX_PARTS)]


class gg_gather_stats_t(C.Structure):
    _fields_ = [("rows", C.c_int64), ("local", C.c_int64), ("hits", C.c_int64),
                ("misses", C.c_int64), ("miss_requests", C.c_int64 * MAX_PARTS),
                ("miss_rows", C.c_int64 * MAX_PARTS)]


class gg_sim_coeffs_t(C.Structure):
    _fields_ = [("eps_init", C.c_double * MAX_PARTS), ("eps_row", C.c_double * MAX_PARTS),
                ("lam_init", C.c_double * MAX_PARTS), ("lam_row", C.c_double * MAX_PARTS),
                ("bw_bytes_per_s", C.c_double), ("row_bytes", C.c_double),
                ("p_idle", C.c_double)]


class gg_sim_acc_t(C.Structure):
    _fields_ = [("windows", C.c_int64), ("batches", C.c_int64),
                ("rebuild_events", C.c_int64), ("rebuild_rows", C.c_int64),
                ("miss_events", C.c_int64), ("miss_rows", C.c_int64),
                ("remote_rows", C.c_int64), ("hits", C.c_int64),
                ("e_rebuild", C.c_double), ("e_miss", C.c_double), ("t_stall", C.c_double),
                ("e_stall", C.c_double), ("e_phy", C.c_double)]


class gg_tuning_t(C.Structure):
    _fields_ = [("tile_rows", C.c_int32), ("gather_blocks", C.c_int32),
                ("gather_loads", C.c_int32), ("stage_blocks", C.c_int32),
                ("stage_host_blocks", C.c_int32), ("emit_blocks", C.c_int32),
                ("hot_max_chunks", C.c_int32), ("bytemap_max_mb", C.c_int32),
                ("sample_order", C.c_int32), ("sample_tile_runs", C.c_int32),
                ("mark_slices_max", C.c_int32), ("mark_slice_chunks", C.c_int32),
                ("mark_block", C.c_int32), ("mark_min_slots", C.c_int32),
                ("mark_min_batches", C.c_int32)]


TUNING_FIELDS = tuple(name for name, _ in gg_tuning_t._fields_)
GG_SAMPLE_BATCH_ORDER, GG_SAMPLE_TILES_LAST, GG_SAMPLE_TILES_ALL = 0, 1, 2


class gg_sage_layer_t(C.Structure):
    _fields_ = [("d_in", C.c_int32), ("d_out", C.c_int32), ("relu", C.c_int32),
                ("w_self", C.c_void_p), ("w_neigh", C.c_void_p), ("bias", C.c_void_p)]


GG_F32, GG_F16 = 0, 1
STAGE_STATS_BYTES = C.sizeof(gg_stage_stats_t)
GATHER_STATS_BYTES = C.sizeof(gg_gather_stats_t)
SIM_ACC_BYTES = C.sizeof(gg_sim_acc_t)

# Every function include/gg.h declares, with its ctypes signature.
_P, _I32, _I64, _U64, _SZ = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_size_t
SIGNATURES = {
    "gg_bits_words": (_I64, [_I64]),
    "gg_sample_caps": (C.c_int, [_I64, _I32, _I64, _P, _I32, _P, _P]),
    "gg_ws_sample": (_SZ, [_I64, _I32, _P]),
    "gg_ws_hotset": (_SZ, [_I64, _I32, _P]),
    "gg_ws_bucket": (_SZ, [_I64, _I32]),
    "gg_ws_stage": (_SZ, [_I64, _I32]),
    "gg_ws_stage_inplace": (_SZ, [_I64, _I64, _I32]),
    "gg_ws_gather": (_SZ, [_I64, _I32, _I32, _P]),
    "gg_sample_window": (C.c_int, [_P, _P, _P, _I32, _P, _I32, _U64, _I32, _I64, _P, _P, _P, _P,
                                   _SZ, _P]),
    "gg_sample_window_part": (C.c_int, [_P, _P, _P, _I32, _P, _I32, _U64, _I32, _I64, _P, _I32,
                                        _P, _P, _P, _SZ, _P]),
    "gg_build_hotset": (C.c_int, [_P, _I32, _P, _I64, _I64, _I64, _P, _P, _I64, _P, _P, _P, _P,
                                  _SZ, _P]),
    "gg_bucket_by_owner": (C.c_int, [_P, _P, _I64, _P, _I32, _P, _P, _P, _P, _SZ, _P]),
    "gg_stage_bulk": (C.c_int, [_P, _P, _I64, _P, _P, _P, _I64, _I64, _P, _P, _P, _P, _P, _P, _P,
                                _P, _P, _SZ, _P]),
    "gg_stage_inplace": (C.c_int, [_P, _P, _I64, _P, _P, _P, _I64, _I64, _P, _P, _P, _P, _P,
                                   _P, _P, _P, _P, _P, _SZ, _P]),
    "gg_gather_batch": (C.c_int, [_P, _P, _I32, _I64, _P, _P, _P, _I64, _I64, _P, _P, _I64, _I32,
                                  _P, _P, _P, _P, _SZ, _P]),
    "gg_gather_batch_noalloc": (C.c_int, [_P, _P, _I32, _I64, _P, _P, _P, _I64, _I64, _P, _P,
                                          _I64, _I32, _P, _P, _P, _P]),
    "gg_sim_accumulate": (C.c_int, [_P, _P, _I32, _P, _P, _P, _P]),
    "gg_ws_sage": (_SZ, [_I64, _I32, _I64, _I32, _P]),
    "gg_sage_forward": (C.c_int, [_P, _I64, _I32, _I32, _P, _P, _I32, _I64, _I64, _P, _P, _I64, _P,
                                  _P, _SZ, _P]),
    "gg_read_status": (C.c_int, [_P, _P, _P]),
    "gg_status_string": (C.c_char_p, [_I32]),
    "gg_last_error": (C.c_char_p, []),
    "gg_version": (C.c_int, []),
}

if not os.path.exists(LIB_PATH):
    raise ImportError(f"libgg is not built ({LIB_PATH}); run __graft_entry__.build()")
# torch first: libgg must bind to the HIP runtime torch loads (its own copy),
# since it is handed torch's streams; loaded first, libgg would bring in the
# system runtime and torch a second one.
import torch  # noqa: E402,F401

lib = C.CDLL(LIB_PATH)
for _name, (_res, _args) in SIGNATURES.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args


class GGError(RuntimeError):
    pass


def check(rc, what):
    if rc != GG_OK:
        msg = lib.gg_last_error().decode()
        raise GGError(f"{what}: {lib.gg_status_string(rc).decode()} ({msg})")
    return rc


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def make_tuning(**fields):
    """A gg_tuning_t with the given fields set (the rest 0: library
    defaults), or None when no field is given."""
    if not fields:
        return None
    t = gg_tuning_t()
    for k, v in fields.items():
        if k not in TUNING_FIELDS:
            raise GGError(f"unknown tuning field {k!r}")
        setattr(t, k, int(v))
    return t


def _tune(tuning):
    return None if tuning is None else C.byref(tuning)


def make_csr(row_ptr, col_idx, num_nodes=None):
    g = gg_csr_t()
    g.num_nodes = row_ptr.numel() - 1 if num_nodes is None else num_nodes
    g.num_edges = col_idx.numel()
    g.row_ptr = row_ptr.data_ptr()
    g.row_ptr_bits = 64 if row_ptr.element_size() == 8 else 32
    g.col_idx = col_idx.data_ptr()
    return g


def make_part(num_parts, kind, local_owner, num_nodes, range_start=None):
    p = gg_part_t()
    p.num_parts = num_parts
    p.kind = kind
    p.local_owner = local_owner
    p.num_nodes = num_nodes
    if range_start is not None:
        for i, v in enumerate(range_start):
            p.range_start[i] = int(v)
    return p


def make_feat(row_bytes, shards, strides, rows):
    """shards: tensors (device, or pinned host used through its device address)."""
    f = gg_feat_t()
    f.row_bytes = row_bytes
    f.num_parts = len(shards)
    for m, (s, st, r) in enumerate(zip(shards, strides, rows)):
        f.shard[m] = s.data_ptr() if (s is not None and r > 0) else None
        f.row_stride[m] = st
        f.shard_rows[m] = r
    return f


def make_wsample(frontier_ids, frontier_off, nbr_ids, nbr_off, frontier_bits, need):
    w = gg_wsample_t()
    w.frontier_ids = frontier_ids.data_ptr()
    w.frontier_cap = frontier_ids.numel()
    w.frontier_off = frontier_off.data_ptr()
    w.nbr_ids = nbr_ids.data_ptr()
    w.nbr_cap = nbr_ids.numel()
    w.nbr_off = nbr_off.data_ptr()
    w.frontier_bits = frontier_bits.data_ptr()
    w.need = need.data_ptr()
    return w


def gg_bits_words(num_nodes):
    return int(lib.gg_bits_words(num_nodes))


def gg_sample_caps(num_nodes, W, max_batch, fanout):
    fan = np.ascontiguousarray(fanout, dtype=np.int32)
    fc, nc = C.c_int64(0), C.c_int64(0)
    check(lib.gg_sample_caps(num_nodes, W, max_batch, fan.ctypes.data, len(fan), C.byref(fc),
                             C.byref(nc)), "gg_sample_caps")
    return fc.value, nc.value


def gg_ws_sample(num_nodes, W, tuning=None):
    return int(lib.gg_ws_sample(num_nodes, W, _tune(tuning)))


def gg_ws_hotset(num_nodes, W, tuning=None):
    return int(lib.gg_ws_hotset(num_nodes, W, _tune(tuning)))


def gg_ws_bucket(cap, num_parts):
    return int(lib.gg_ws_bucket(cap, num_parts))


def gg_ws_stage(cap, num_parts):
    return int(lib.gg_ws_stage(cap, num_parts))


def gg_ws_gather(n_cap, nseg, num_parts, tuning=None):
    return int(lib.gg_ws_gather(n_cap, nseg, num_parts, _tune(tuning)))


def gg_sample_window(csr, seeds, seed_off, W, fanout, L, rng_seed, epoch, batch0, out, status, ws,
                     stream=None, tuning=None):
    so = np.ascontiguousarray(seed_off, dtype=np.int64)
    fan = np.ascontiguousarray(fanout, dtype=np.int32)
    if seeds is not None and hasattr(seeds, "numel") and seeds.numel() < int(so[-1]):
        raise GGError(f"gg_sample_window: seed_off ends at {int(so[-1])} but only "
                      f"{seeds.numel()} seeds were given")
    return check(lib.gg_sample_window(C.byref(csr), _ptr(seeds), so.ctypes.data, W,
                                      fan.ctypes.data, L, C.c_uint64(rng_seed), epoch, batch0,
                                      C.byref(out), _tune(tuning), _ptr(status), _ptr(ws),
                                      ws.numel(), _stream(stream)), "gg_sample_window")


GG_SAMPLE_PART_BITS, GG_SAMPLE_PART_LAST = 1, 2


def gg_sample_window_part(csr, seeds, seed_off, W, fanout, L, rng_seed, epoch, batch0, out, part,
                          status, ws, stream=None, tuning=None):
    """One part of gg_sample_window (GG_SAMPLE_PART_BITS, then
    GG_SAMPLE_PART_LAST with the same arguments and workspace)."""
    so = np.ascontiguousarray(seed_off, dtype=np.int64)
    fan = np.ascontiguousarray(fanout, dtype=np.int32)
    return check(lib.gg_sample_window_part(C.byref(csr), _ptr(seeds), so.ctypes.data, W,
                                           fan.ctypes.data, L, C.c_uint64(rng_seed), epoch,
                                           batch0, C.byref(out), part, _tune(tuning),
                                           _ptr(status), _ptr(ws), ws.numel(), _stream(stream)),
                 "gg_sample_window_part")


def gg_build_hotset(frontier_bits, W, part, n_hot, hot_ids, hot_freq, cap, hot_count, status, ws,
                    stream=None, hot_frac=None, tuning=None):
    """hot_frac = (num, den): budget ceil(U * num / den) of the window's U
    distinct remote nodes (n_hot must then be -1)."""
    num, den = hot_frac if hot_frac is not None else (0, 0)
    return check(lib.gg_build_hotset(_ptr(frontier_bits), W, C.byref(part), n_hot, num, den,
                                     _ptr(hot_ids), _ptr(hot_freq), cap, _ptr(hot_count),
                                     _tune(tuning), _ptr(status), _ptr(ws), ws.numel(),
                                     _stream(stream)), "gg_build_hotset")


def gg_bucket_by_owner(hot_ids, hot_count, cap, part, bucket_ids, owner_off, status, ws,
                       stream=None, flags=0):
    """flags = GG_BUCKET_OWNER_ORDERED when hot_ids is known to be in owner
    order (the ascending output of gg_build_hotset under a range book)."""
    return check(lib.gg_bucket_by_owner(_ptr(hot_ids), _ptr(hot_count), cap, C.byref(part), flags,
                                        _ptr(bucket_ids), _ptr(owner_off), _ptr(status), _ptr(ws),
                                        ws.numel(), _stream(stream)), "gg_bucket_by_owner")


def gg_stage_bulk(bucket_ids, owner_off, cap, part, feat, cache, cache_stride, cache_rows, slot_of,
                  clear_ids, clear_count, src_cache, src_slot_of, stats, status, ws, stream=None,
                  tuning=None):
    return check(lib.gg_stage_bulk(_ptr(bucket_ids), _ptr(owner_off), cap, C.byref(part),
                                   C.byref(feat), _ptr(cache), cache_stride, cache_rows,
                                   _ptr(slot_of), _ptr(clear_ids), _ptr(clear_count),
                                   _ptr(src_cache), _ptr(src_slot_of), _ptr(stats),
                                   _tune(tuning), _ptr(status), _ptr(ws), ws.numel(),
                                   _stream(stream)), "gg_stage_bulk")


def gg_ws_stage_inplace(cap, cache_rows, num_parts):
    return int(lib.gg_ws_stage_inplace(cap, cache_rows, num_parts))


def gg_stage_inplace(bucket_ids, owner_off, cap, part, feat, cache, cache_stride, cache_rows,
                     slot_of, clear_ids, clear_count, prev_slot_of, occ_prev, occ, stats, status,
                     ws, stream=None, tuning=None):
    return check(lib.gg_stage_inplace(_ptr(bucket_ids), _ptr(owner_off), cap, C.byref(part),
                                      C.byref(feat), _ptr(cache), cache_stride, cache_rows,
                                      _ptr(slot_of), _ptr(clear_ids), _ptr(clear_count),
                                      _ptr(prev_slot_of), _ptr(occ_prev), _ptr(occ), _ptr(stats),
                                      _tune(tuning), _ptr(status), _ptr(ws), ws.numel(),
                                      _stream(stream)), "gg_stage_inplace")


def occ_bytes(cache_rows):
    """Bytes of a cache occupancy buffer (gg_stage_inplace): a 16-byte
    header and one byte per slot, rounded up to a multiple of 32."""
    return 16 + (int(cache_rows) + 31) // 32 * 32


def gg_gather_batch(in_ids, bounds_ptr, nseg, n_cap, part, feat, cache, cache_stride, cache_rows,
                    slot_of, out, out_stride, stats_ptr, status, ws, stream=None, flags=0,
                    tuning=None):
    """bounds_ptr and stats_ptr are raw device addresses (e.g. an offset into
    frontier_off, or into an array of nseg statistics structures).  flags =
    GG_GATHER_SHARED when other streams sample on the device meanwhile."""
    return check(lib.gg_gather_batch(_ptr(in_ids), bounds_ptr, nseg, n_cap, C.byref(part),
                                     C.byref(feat), _ptr(cache), cache_stride, cache_rows,
                                     _ptr(slot_of), _ptr(out), out_stride, flags, stats_ptr,
                                     _tune(tuning), _ptr(status), _ptr(ws), ws.numel(),
                                     _stream(stream)), "gg_gather_batch")


GATHER_SCRATCH_BYTES = 1 << 20


def gg_gather_batch_noalloc(in_ids, bounds_ptr, nseg, n_cap, part, feat, cache, cache_stride,
                            cache_rows, slot_of, out, out_stride, stats_ptr, status, stream=None,
                            flags=0, tuning=None):
    """gg_gather_batch without a workspace: the library's per-GPU scratch
    array holds the call's block statistics (calls overlapping on one GPU
    race)."""
    return check(lib.gg_gather_batch_noalloc(_ptr(in_ids), bounds_ptr, nseg, n_cap,
                                             C.byref(part), C.byref(feat), _ptr(cache),
                                             cache_stride, cache_rows, _ptr(slot_of), _ptr(out),
                                             out_stride, flags, stats_ptr, _tune(tuning),
                                             _ptr(status), _stream(stream)),
                 "gg_gather_batch_noalloc")


def make_sim_coeffs(P, eps_init, eps_row, lam_init, lam_row, bw_bytes_per_s, row_bytes, p_idle):
    """Coefficients of the analytical energy model; each per-owner term is a
    scalar (every owner alike) or a sequence of P values."""
    c = gg_sim_coeffs_t()
    for name, v in (("eps_init", eps_init), ("eps_row", eps_row), ("lam_init", lam_init),
                    ("lam_row", lam_row)):
        vals = list(v) if hasattr(v, "__len__") else [v] * P
        arr = getattr(c, name)
        for m in range(P):
            arr[m] = float(vals[m])
    c.bw_bytes_per_s, c.row_bytes, c.p_idle = float(bw_bytes_per_s), float(row_bytes), float(p_idle)
    return c


def gg_sim_accumulate(stage_stats, gather_stats_ptr, nseg, part, coeffs, acc, stream=None):
    """gather_stats_ptr is the device address of nseg gather statistics."""
    return check(lib.gg_sim_accumulate(_ptr(stage_stats), gather_stats_ptr, nseg, C.byref(part),
                                       C.byref(coeffs), _ptr(acc), _stream(stream)),
                 "gg_sim_accumulate")


def sim_acc_from_bytes(buf):
    a = gg_sim_acc_t.from_buffer_copy(bytes(buf))
    return {name: (float(getattr(a, name)) if typ is C.c_double else int(getattr(a, name)))
            for name, typ in a._fields_}


def make_sage_layers(layers):
    """layers: sequence of (w_self [d_in, d_out], w_neigh, bias or None,
    relu) with fp32 device tensors.  The tensors must outlive the calls."""
    arr = (gg_sage_layer_t * len(layers))()
    for j, (ws, wn, b, relu) in enumerate(layers):
        if ws.dtype != wn.dtype or ws.shape != wn.shape or ws.dim() != 2:
            raise GGError(f"layer {j}: w_self and w_neigh must be matching 2-d tensors")
        if not (ws.is_contiguous() and wn.is_contiguous()):
            raise GGError(f"layer {j}: weights must be contiguous")
        arr[j].d_in, arr[j].d_out, arr[j].relu = int(ws.shape[0]), int(ws.shape[1]), int(bool(relu))
        arr[j].w_self, arr[j].w_neigh = ws.data_ptr(), wn.data_ptr()
        arr[j].bias = b.data_ptr() if b is not None else None
    return arr


def gg_ws_sage(num_nodes, W, rows_cap, layers_arr):
    return int(lib.gg_ws_sage(num_nodes, W, rows_cap, len(layers_arr), layers_arr))


def gg_sage_forward(wsample, num_nodes, W, fanout, x, x_dtype, x_stride, rows_cap, layers_arr, out,
                    out_rows_cap, status, ws, stream=None):
    fan = np.ascontiguousarray(fanout, dtype=np.int32)
    return check(lib.gg_sage_forward(C.byref(wsample), num_nodes, W, len(fan), fan.ctypes.data,
                                     _ptr(x),
                                     x_dtype, x_stride, rows_cap, layers_arr, _ptr(out),
                                     out_rows_cap, _ptr(status), _ptr(ws), ws.numel(),
                                     _stream(stream)), "gg_sage_forward")


def gg_read_status(status, stream=None):
    """Waits for `stream` and returns the GG_DEV_* bits of the status word."""
    out = C.c_int32(0)
    check(lib.gg_read_status(_ptr(status), C.byref(out), _stream(stream)), "gg_read_status")
    return int(out.value)


def gg_status_string(code):
    return lib.gg_status_string(code).decode()


def gg_last_error():
    return lib.gg_last_error().decode()


def gg_version():
    return int(lib.gg_version())


def stage_stats_from_bytes(buf, P):
    st = gg_stage_stats_t.from_buffer_copy(bytes(buf))
    return _stats_dict(st, P)


def gather_stats_from_bytes(buf, P):
    st = gg_gather_stats_t.from_buffer_copy(bytes(buf))
    return _stats_dict(st, P)


def _stats_dict(st, P):
    d = {}
    for name, _ in st._fields_:
        v = getattr(st, name)
        d[name] = [int(x) for x in v][:P] if hasattr(v, "__len__") else int(v)
    return d
