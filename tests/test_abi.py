"""The C ABI without a GPU: libgg loads, exports every function include/gg.h
declares, the ctypes structures match the header's layout, and host-side
argument checks reject bad calls before anything is enqueued."""
import ctypes as C
import os
import re
import subprocess
import tempfile

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gg.h")


@pytest.fixture(scope="module")
def gg():
    lib = os.path.join(ROOT, "paper_2606_02916_amd", "libgg.so")
    if not os.path.exists(lib):
        from paper_2606_02916_amd import build
        build.build()
    from paper_2606_02916_amd import gg as mod
    return mod


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gg_[a-z_]+)\s*\(", text)))


def test_every_declared_function_is_exported_and_bound(gg):
    names = declared_functions()
    assert len(names) >= 14
    out = subprocess.run(["nm", "-D", "--defined-only", gg.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (gg_\w+)", out))
    for n in names:
        assert n in exported, n
        assert n in gg.SIGNATURES, n
    assert set(gg.SIGNATURES) == set(names)


LAYOUT_PROBE = r"""
#include <stddef.h>
#include <stdio.h>
#include "gg.h"
#define F(T, f) printf(#T " " #f " %zu\n", offsetof(T, f));
#define S(T) printf(#T " sizeof %zu\n", sizeof(T));
int main() {
  S(gg_csr_t) F(gg_csr_t, num_edges) F(gg_csr_t, row_ptr) F(gg_csr_t, row_ptr_bits) F(gg_csr_t, col_idx)
  S(gg_part_t) F(gg_part_t, local_owner) F(gg_part_t, num_nodes) F(gg_part_t, range_start)
  S(gg_feat_t) F(gg_feat_t, shard) F(gg_feat_t, row_stride) F(gg_feat_t, shard_rows)
  S(gg_wsample_t) F(gg_wsample_t, frontier_cap) F(gg_wsample_t, nbr_ids) F(gg_wsample_t, nbr_off)
  F(gg_wsample_t, frontier_bits) F(gg_wsample_t, need)
  S(gg_stage_stats_t) F(gg_stage_stats_t, invalidated) F(gg_stage_stats_t, retained) F(gg_stage_stats_t, requests)
  F(gg_stage_stats_t, rows) F(gg_stage_stats_t, bytes) F(gg_stage_stats_t, delta_rows)
  S(gg_gather_stats_t) F(gg_gather_stats_t, misses) F(gg_gather_stats_t, miss_requests)
  F(gg_gather_stats_t, miss_rows)
  S(gg_sim_coeffs_t) F(gg_sim_coeffs_t, eps_row) F(gg_sim_coeffs_t, lam_init)
  F(gg_sim_coeffs_t, lam_row) F(gg_sim_coeffs_t, bw_bytes_per_s) F(gg_sim_coeffs_t, row_bytes)
  F(gg_sim_coeffs_t, p_idle)
  S(gg_sim_acc_t) F(gg_sim_acc_t, rebuild_events) F(gg_sim_acc_t, miss_rows)
  F(gg_sim_acc_t, hits) F(gg_sim_acc_t, e_rebuild) F(gg_sim_acc_t, t_stall) F(gg_sim_acc_t, e_phy)
  S(gg_sage_layer_t) F(gg_sage_layer_t, relu) F(gg_sage_layer_t, w_self)
  F(gg_sage_layer_t, w_neigh) F(gg_sage_layer_t, bias)
  S(gg_tuning_t) F(gg_tuning_t, gather_blocks) F(gg_tuning_t, gather_loads)
  F(gg_tuning_t, stage_blocks) F(gg_tuning_t, stage_host_blocks) F(gg_tuning_t, emit_blocks)
  F(gg_tuning_t, hot_max_chunks) F(gg_tuning_t, bytemap_max_mb) F(gg_tuning_t, sample_order) F(gg_tuning_t, sample_tile_runs)
  F(gg_tuning_t, mark_slices_max) F(gg_tuning_t, mark_slice_chunks)
  F(gg_tuning_t, mark_block) F(gg_tuning_t, mark_min_slots)
  F(gg_tuning_t, mark_min_batches)
  return 0;
}
"""


def test_struct_layouts_match_the_header(gg):
    d = tempfile.mkdtemp(prefix="ggabi_")
    src = os.path.join(d, "probe.cpp")
    with open(src, "w") as f:
        f.write(LAYOUT_PROBE)
    exe = os.path.join(d, "probe")
    subprocess.run(["g++", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    "-I" + os.path.join(ROOT, "include"), src, "-o", exe], check=True)
    lines = subprocess.run([exe], capture_output=True, text=True, check=True).stdout.split("\n")
    for line in filter(None, lines):
        tname, field, val = line.split()
        T = getattr(gg, tname)
        if field == "sizeof":
            assert C.sizeof(T) == int(val), line
        else:
            assert getattr(T, field).offset == int(val), line


def test_host_helpers(gg):
    assert gg.gg_version() == 1
    assert gg.gg_status_string(gg.GG_ERR_ARG) == "invalid argument"
    for n in (1, 31, 32, 33, 65536, 65537, 10**7):
        w = gg.gg_bits_words(n)
        assert w % 2048 == 0 and w * 32 >= n and (w - 2048) * 32 < max(n, 1)
    # worst-case capacities: sum over levels of min(N, B * prod(k_i + 1))
    fc, nc = gg.gg_sample_caps(2_450_000, 16, 1024, [15, 10, 5])
    lev = [1024, 1024 * 16, 1024 * 16 * 11, min(2_450_000, 1024 * 16 * 11 * 6)]
    assert fc == 16 * sum(lev)
    assert nc == 16 * (lev[0] * 15 + lev[1] * 10 + lev[2] * 5)
    fc, nc = gg.gg_sample_caps(1000, 2, 600, [3])
    assert fc == 2 * (600 + 1000) and nc == 2 * 600 * 3
    for f in (gg.gg_ws_sample, gg.gg_ws_hotset):
        assert f(10_000, 4) > 0 and f(10_000, 4) % 256 == 0
    assert gg.gg_ws_bucket(0, 4) > 0 and gg.gg_ws_gather(0, 1, 4) > 0 and gg.gg_ws_stage(0, 4) > 0
    # tuning that changes workspace layouts changes the sizes; bad tuning sizes nothing
    N, W = 2_450_000, 16
    t = gg.make_tuning
    nomap = gg.gg_ws_sample(N, W, t(bytemap_max_mb=-1))
    assert gg.gg_ws_sample(N, W, t(bytemap_max_mb=1)) == nomap
    assert gg.gg_ws_sample(N, W) < gg.gg_ws_sample(N, W, t(sample_order=1))
    # 2.45M nodes: 38 chunks of 65,536 ids, 5 slices of 8 chunks per batch;
    # marks through LDS leave the byte map out: at any batch count with
    # mark_min_batches = -1; by default only from 8 batches on, so a
    # 16-batch workspace holds the 7-batch map a shorter window may take
    assert gg.gg_ws_sample(N, W, t(mark_slices_max=5, mark_min_batches=-1)) == nomap
    per_batch_map = gg.gg_bits_words(N) * 32
    assert gg.gg_ws_sample(N, W) >= 7 * per_batch_map
    assert gg.gg_ws_sample(N, W) < nomap + 8 * per_batch_map
    assert gg.gg_ws_sample(N, W, t(mark_slices_max=4)) == \
        gg.gg_ws_sample(N, W, t(mark_slices_max=-1)) >= nomap + 16 * per_batch_map
    assert gg.gg_ws_sample(N, W, t(mark_min_batches=17)) == \
        gg.gg_ws_sample(N, W, t(mark_slices_max=-1))
    assert gg.gg_ws_hotset(N, W, gg.make_tuning(hot_max_chunks=4)) < gg.gg_ws_hotset(N, W)
    assert gg.gg_ws_gather(10**6, 1, 4, gg.make_tuning(gather_blocks=64)) < \
        gg.gg_ws_gather(10**6, 1, 4)
    assert gg.gg_ws_gather(10**6, 1, 4, gg.make_tuning(gather_loads=3)) == 0
    assert gg.make_tuning() is None
    with pytest.raises(gg.GGError):
        gg.make_tuning(tile=3)
    # a workspace sized for W batches (nseg segments) serves every shorter
    # call: a short last window may take the byte map that W batches do not
    # (2.45M nodes: 2.49 MB of map per batch; 64 MB holds 25 batches, so
    # W = 32 runs without it and a 16-batch window with it), and fewer
    # segments may launch more gather blocks in all (1024 = 1 x 1024, but
    # 3 x 341)
    for t in (None, gg.make_tuning(bytemap_max_mb=64, mark_slices_max=-1),
              gg.make_tuning(bytemap_max_mb=8, mark_slices_max=-1),
              gg.make_tuning(bytemap_max_mb=64, sample_order=1, mark_slices_max=-1),
              gg.make_tuning(bytemap_max_mb=64, mark_slices_max=4)):
        for N in (60_001, 2_450_000):
            for W in (1, 3, 16, 32, 64):
                big = gg.gg_ws_sample(N, W, t)
                assert all(gg.gg_ws_sample(N, w, t) <= big for w in range(1, W + 1)), (N, W)
                big = gg.gg_ws_hotset(N, W, t)
                assert all(gg.gg_ws_hotset(N, w, t) <= big for w in range(1, W + 1)), (N, W)
    assert gg.gg_ws_sample(2_450_000, 32, gg.make_tuning(bytemap_max_mb=64,
                                                         mark_slices_max=-1)) >= 2_450_000 * 16
    for t in (None, gg.make_tuning(gather_blocks=1000), gg.make_tuning(gather_blocks=96)):
        for n_cap in (1, 5000, 10**6, 4 * 10**7):
            for nseg in (1, 3, 7, 16, 64):
                big = gg.gg_ws_gather(n_cap, nseg, 4, t)
                assert all(gg.gg_ws_gather(n, s, 4, t) <= big
                           for s in range(1, nseg + 1) for n in (1, n_cap // 3, n_cap)), \
                    (n_cap, nseg)
    for cap in (0, 1, 1000, 10**6):
        for f in (lambda c: gg.gg_ws_bucket(c, 4), lambda c: gg.gg_ws_stage(c, 4),
                  lambda c: gg.gg_ws_stage_inplace(c, 2 * c, 4)):
            assert all(f(c) <= f(cap) for c in (0, cap // 2, cap))
    # the status read checks its pointers before any HIP call
    with pytest.raises(gg.GGError, match="null"):
        gg.gg_read_status(None, stream=0)


class _FakeTensor:
    """Stands in for a device tensor in calls that must be rejected before
    any device work: only its address and size are read."""

    def __init__(self, addr, n=1):
        self.addr, self.n = addr, n

    def data_ptr(self):
        return self.addr

    def numel(self):
        return self.n

    def element_size(self):
        return 8


def test_bad_arguments_are_rejected_on_the_host(gg):
    t = _FakeTensor(1 << 20, 1 << 20)
    csr = gg.make_csr(_FakeTensor(4096, 101), _FakeTensor(8192, 500), num_nodes=100)
    ws = gg.make_wsample(t, t, t, t, t, t)
    for W, fan, off in [(0, [2], [0]), (65, [2], [0] * 66), (2, [0], [0, 1, 2]),
                        (2, [33], [0, 1, 2]), (2, [2], [0, 3, 2]), (2, [2], [1, 2, 3])]:
        with pytest.raises(gg.GGError) as e:
            gg.gg_sample_window(csr, t, np.array(off), W, fan, len(fan), 0, 0, 0, ws, t, t,
                                stream=0)
        assert "invalid argument" in str(e.value)
    part = gg.make_part(0, gg.PART_MOD, 0, 100)
    with pytest.raises(gg.GGError):
        gg.gg_build_hotset(t, 4, part, -1, t, None, 10, t, t, t, stream=0)
    part = gg.make_part(4, gg.PART_MOD, 0, 100)
    for n_hot, frac in [(5, (1, 10)), (-1, (11, 10)), (-1, (-1, 10)), (-1, (1, 1 << 32))]:
        with pytest.raises(gg.GGError):                                  # bad relative budgets
            gg.gg_build_hotset(t, 4, part, n_hot, t, None, 10, t, t, t, stream=0, hot_frac=frac)
    part = gg.make_part(4, gg.PART_RANGE, 0, 100, [0, 10, 20, 30, 99])  # does not end at N
    with pytest.raises(gg.GGError):
        gg.gg_bucket_by_owner(t, t, 10, part, t, t, t, t, stream=0)
    part = gg.make_part(4, gg.PART_RANGE, 0, 100, [0, 10, 20, 30, 100])
    with pytest.raises(gg.GGError):                                      # unknown flag bit
        gg.gg_bucket_by_owner(t, t, 10, part, t, t, t, t, stream=0, flags=2)
    part = gg.make_part(4, gg.PART_MOD, 4, 100)                          # local owner >= P
    feat = gg.make_feat(256, [t] * 4, [256] * 4, [25] * 4)
    with pytest.raises(gg.GGError):
        gg.gg_stage_bulk(t, t, 10, part, feat, t, 256, 10, t, None, None, None, None, t, t, t, stream=0)
    part = gg.make_part(4, gg.PART_MOD, 0, 100)
    feat = gg.make_feat(256, [t] * 4, [256] * 4, [25] * 4)
    u = _FakeTensor(1 << 22, 1 << 20)
    big = _FakeTensor(1 << 23, 1 << 30)
    for prev, occ_prev, occ, what in [(t, t, u, "remap"),          # previous remap = this one
                                      (u, None, t, "both"),        # occupancy without remap
                                      (u, t, t, "occupancy")]:     # occupancy buffers shared
        with pytest.raises(gg.GGError):
            gg.gg_stage_inplace(t, t, 10, part, feat, t, 256, 10, t, None, None, prev, occ_prev,
                                occ, t, t, big, stream=0)
        assert what in gg.gg_last_error()
    with pytest.raises(gg.GGError):                                      # workspace too small
        gg.gg_stage_inplace(t, t, 10, part, feat, t, 256, 10, t, None, None, None, None, u, t, t,
                            _FakeTensor(1 << 24, 16), stream=0)
    assert "workspace" in gg.gg_last_error()
    feat = gg.make_feat(250, [t] * 4, [256] * 4, [25] * 4)              # row_bytes % 4 != 0
    with pytest.raises(gg.GGError):
        gg.gg_gather_batch(t, t.data_ptr(), 1, 10, part, feat, t, 256, 10, t, t, 256,
                           t.data_ptr(), t, t, stream=0)
    feat = gg.make_feat(256, [t] * 4, [256] * 4, [25] * 4)
    with pytest.raises(gg.GGError):                                      # nseg outside 1..64
        gg.gg_gather_batch(t, t.data_ptr(), 0, 10, part, feat, t, 256, 10, t, t, 256,
                           t.data_ptr(), t, t, stream=0)
    assert "nseg" in gg.gg_last_error()
    with pytest.raises(gg.GGError):                                      # unknown gather flag
        gg.gg_gather_batch(t, t.data_ptr(), 1, 10, part, feat, t, 256, 10, t, t, 256,
                           t.data_ptr(), t, t, stream=0, flags=2)
    assert "flags" in gg.gg_last_error()
    for field, bad in [("tile_rows", 65), ("tile_rows", -1), ("gather_blocks", 4),
                       ("gather_loads", 3), ("stage_blocks", -2), ("stage_host_blocks", -2),
                       ("emit_blocks", 513), ("hot_max_chunks", 4097), ("bytemap_max_mb", -2),
                       ("sample_tile_runs", 3), ("sample_tile_runs", 128),
                       ("sample_tile_runs", -1), ("sample_order", 3), ("sample_order", -1),
                       ("mark_slices_max", -2), ("mark_slices_max", 4097),
                       ("mark_slice_chunks", -1), ("mark_slice_chunks", 9),
                       ("mark_block", 128), ("mark_block", 512),
                       ("mark_min_slots", -2), ("mark_min_batches", -2),
                       ("mark_min_batches", 65)]:
        tune = gg.make_tuning(**{field: bad})
        with pytest.raises(gg.GGError):                                  # tuning out of range
            gg.gg_gather_batch(t, t.data_ptr(), 1, 10, part, feat, t, 256, 10, t, t, 256,
                               t.data_ptr(), t, t, stream=0, tuning=tune)
        assert field in gg.gg_last_error()
        with pytest.raises(gg.GGError):
            gg.gg_stage_inplace(t, t, 10, part, feat, t, 256, 10, t, None, None, None, None, u,
                                t, t, big, stream=0, tuning=tune)
        assert field in gg.gg_last_error()
    # the no-allocation gather rejects a call whose scratch exceeds its array,
    # before any device work
    part64 = gg.make_part(64, gg.PART_MOD, 0, 100)
    feat64 = gg.make_feat(256, [t] * 64, [256] * 64, [2] * 64)
    with pytest.raises(gg.GGError) as e:
        gg.gg_gather_batch_noalloc(t, t.data_ptr(), 64, 10**9, part64, feat64, t, 256, 10, t, t,
                                   256, t.data_ptr(), t, stream=0,
                                   tuning=gg.make_tuning(gather_blocks=65536))
    assert "capacity" in str(e.value) and "scratch" in gg.gg_last_error()
    c = gg.make_sim_coeffs(4, 1.0, 0.01, 1e-3, 1e-5, 0.0, 256, 30.0)    # no bandwidth ceiling
    with pytest.raises(gg.GGError):
        gg.gg_sim_accumulate(t, t.data_ptr(), 4, part, c, t, stream=0)
    c = gg.make_sim_coeffs(4, 1.0, 0.01, 1e-3, 1e-5, 1e9, 256, 30.0)
    with pytest.raises(gg.GGError):                                      # more batches than W max
        gg.gg_sim_accumulate(t, t.data_ptr(), 65, part, c, t, stream=0)
    # GraphSAGE consumer: inconsistent layer shapes and bad dtypes
    smp = gg.make_wsample(t, t, t, t, t, t)
    w = _FakeTensor(1 << 21, 64 * 16)
    for dtype, stride, dims in [(2, 256, [(64, 16), (16, 8)]),         # unknown dtype
                                (gg.GG_F32, 128, [(64, 16), (16, 8)]),  # row wider than stride
                                (gg.GG_F32, 256, [(64, 16), (15, 8)]),  # d_in != previous d_out
                                (gg.GG_F32, 256, [(64, 16), (16, 129)])]:  # d_out > 128
        arr = (gg.gg_sage_layer_t * 2)()
        for j, (di, do) in enumerate(dims):
            arr[j].d_in, arr[j].d_out, arr[j].relu = di, do, 1
            arr[j].w_self = arr[j].w_neigh = w.data_ptr()
        with pytest.raises(gg.GGError):
            gg.gg_sage_forward(smp, 1000, 4, [3, 2], t, dtype, stride, 100, arr, t, 100, t, t,
                               stream=0)


def test_lookahead_byte_map_choice_follows_last_hop_density(gg):
    """The look-ahead driver keeps the sampler's byte map for a dense last
    hop (at least as many draws per batch as nodes, by the frontier bound)
    and caps it otherwise: the bound is min(N, B * prod_{i<L-1}(k_i + 1))
    draws of k_{L-1} each.  It samples the last hop in node tiles when at
    least two batches share a frontier node, by the same bound."""
    from paper_2606_02916_amd.window import last_hop_density, last_hop_sharing
    assert last_hop_density(2_450_000, [15, 10, 5], 1024) == 1024 * 16 * 11 * 5 / 2_450_000
    assert last_hop_density(2_450_000, [15, 10, 5], 4096) == 4096 * 16 * 11 * 5 / 2_450_000
    assert last_hop_density(1000, [15, 10, 5], 512) == 1000 * 5 / 1000    # capped at N
    assert last_hop_density(233_000, [25, 10], 1024) == 1024 * 26 * 10 / 233_000
    assert last_hop_density(100, [7], 3) == 3 * 7 / 100                     # one hop: seeds
    # frontier bound per level as gg_sample_caps sums it (one batch)
    fc, nc = gg.gg_sample_caps(2_450_000, 1, 4096, [15, 10, 5])
    lev2 = min(2_450_000, 4096 * 16 * 11)
    assert nc == 4096 * 15 + 4096 * 16 * 10 + lev2 * 5
    assert last_hop_density(2_450_000, [15, 10, 5], 4096) == lev2 * 5 / 2_450_000
    # batches sharing a last-hop node, by the bound: W * min(N, ...) / N
    assert last_hop_sharing(2_450_000, [15, 10, 5], 4096, 16) == 16 * lev2 / 2_450_000 > 2
    assert last_hop_sharing(2_450_000, [15, 10, 5], 1024, 16) == \
        16 * 1024 * 16 * 11 / 2_450_000 < 2
    assert last_hop_sharing(233_000, [25, 10], 1024, 8) == 8 * 1024 * 26 / 233_000 < 2
    assert last_hop_sharing(1000, [15, 10, 5], 512, 4) == 4.0                # capped at N


@pytest.mark.parametrize("order", ["package first", "torch first"])
def test_one_hip_runtime_whatever_the_import_order(gg, order):
    """libgg is handed torch's streams, so it must bind to the HIP runtime
    torch loads: imported before torch, it would bring in the system
    runtime through its own search path, and torch a second one."""
    first = ("from paper_2606_02916_amd import gg; import torch" if order == "package first"
             else "import torch; from paper_2606_02916_amd import gg")
    code = (f"{first}\n"
            "maps = sorted({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l})\n"
            "print(len(maps), maps)\n")
    out = subprocess.run(["python3", "-c", code], cwd=ROOT, capture_output=True, text=True,
                         timeout=300)
    assert out.returncode == 0, out.stderr[-2000:]
    assert out.stdout.split()[0] == "1", out.stdout
