"""Shared set-up for the GPU parity tests: the same seeded inputs go to the
HIP path (through the C ABI) and to the CPU oracle; results are compared
byte for byte."""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import ggref
from paper_2606_02916_amd import FetchPipeline


def log(msg):
    print(msg, flush=True)


class World:
    """One workload instance on the GPU and its oracle counterpart."""

    def __init__(self, inst, W=None, n_hot=-1, local_owner=None, fanout=None, batch=None,
                 device="cuda:0", shards=None, row_bytes=None, stride=None, cache_stride=None,
                 tensors=None, delta=False, hot_frac=None, inplace=False):
        wl = inst.wl
        self.inst = inst
        self.wl = wl
        self.shards = inst.shards if shards is None else shards
        self.row_bytes = wl.row_bytes if row_bytes is None else row_bytes
        self.stride = wl.row_stride if stride is None else stride
        self.W = W or wl.W
        self.n_hot = n_hot
        self.local = wl.local_owner if local_owner is None else local_owner
        self.fanout = tuple(fanout or wl.fanout)
        self.batch = batch or wl.batch_size
        self.dev = torch.device(device)
        self.P = wl.num_parts
        self.rs = inst.range_start
        if tensors is not None:        # (row_ptr_d, col_idx_d, shards_d) already placed
            self.row_ptr_d, self.col_idx_d, self.shards_d = tensors
        else:
            self.row_ptr_d = torch.from_numpy(inst.row_ptr).to(self.dev)
            self.col_idx_d = torch.from_numpy(inst.col_idx).to(self.dev)
            self.shards_d = [torch.from_numpy(s).to(self.dev) for s in self.shards]
        rows = [s.shape[0] for s in self.shards]
        self.pipe = FetchPipeline(self.row_ptr_d, self.col_idx_d, self.P, wl.part_kind, self.local,
                                  self.rs, self.shards_d, rows, self.row_bytes, self.stride,
                                  self.W, self.fanout, self.batch, n_hot=n_hot, device=self.dev,
                                  cache_stride=cache_stride, delta=delta, hot_frac=hot_frac,
                                  inplace=inplace)
        self.part_ref = ggref.make_part(self.P, wl.part_kind, self.local, wl.num_nodes, self.rs)
        self.feat_ref = ggref.make_feat(self.row_bytes, self.shards, [self.stride] * self.P)
        self.cstride = self.pipe.cache_stride
        self.delta = delta or inplace
        self.inplace = inplace
        self.hot_frac = hot_frac
        self.cache_refs = [np.zeros((self.pipe.cache_rows, self.cstride), dtype=np.uint8)
                           for _ in range(2 if delta and not inplace else 1)]
        # the in-place driver alternates two remaps, each cleared of the
        # window it held two windows back
        self.slot_refs = [np.full(wl.num_nodes, -1, dtype=np.int32)
                          for _ in range(2 if inplace else 1)]
        self.held = [None, None]
        self.prev_ref = None

    @property
    def slot_ref(self):
        return self.slot_refs[self.pipe.k % len(self.slot_refs)]

    def window_inputs(self, k, W=None):
        W = W or self.W
        b0, b1 = synth.window_batches(self.inst.batch_off, W, k)
        boff = self.inst.batch_off
        so = boff[b0:b1 + 1] - boff[b0]
        seeds = self.inst.seeds[boff[b0]:boff[b1]]
        return seeds, so, b0

    def run_and_compare(self, k, epoch=0, rng_seed=0, check_outputs=True, seeds=None, so=None,
                        b0=None):
        """Runs window k on both sides and asserts every intermediate equal."""
        if seeds is None:
            seeds, so, b0 = self.window_inputs(k)
        pipe, rb, st = self.pipe, self.row_bytes, self.stride
        L = len(self.fanout)
        seeds_d = torch.from_numpy(np.ascontiguousarray(seeds, dtype=np.int32)).to(self.dev)
        cur = pipe.slot_index()
        Wk = pipe.sample(seeds_d, so, b0, epoch, rng_seed)
        pipe.hotset(Wk, cur)
        pipe.bucket(cur)
        pipe.stage(cur)
        torch.cuda.synchronize()
        assert pipe.read_status() == 0, pipe.read_status()
        # sampling
        fids, foff, nids, noff = ggref.sample_window(self.inst.row_ptr, self.inst.col_idx, seeds,
                                                     so, self.fanout, rng_seed, epoch, b0)
        g_fids, g_foff, g_nids, g_noff = pipe.sample_outputs(Wk)
        assert np.array_equal(g_foff, foff)
        assert np.array_equal(g_fids, fids)
        assert np.array_equal(g_noff, noff)
        assert np.array_equal(g_nids, nids)
        # the bit sets hold exactly N_b
        bits = pipe.frontier_bits.view(torch.int32)[:Wk * pipe.wpb].cpu().numpy().view(np.uint32)
        for b in range(Wk):
            ids = fids[foff[L * Wk + b]:foff[L * Wk + b + 1]]
            row = bits[b * pipe.wpb:(b + 1) * pipe.wpb]
            got = np.nonzero(np.unpackbits(row.view(np.uint8), bitorder="little"))[0]
            assert np.array_equal(got, ids)
        # hot set and buckets
        hot, freq = ggref.build_hotset(fids, foff, Wk, L, self.part_ref, self.n_hot,
                                       hot_frac=self.hot_frac)
        bucket, owner_off = ggref.bucket_by_owner(hot, self.part_ref)
        g_hot, g_freq, g_cnt, g_bucket, g_owner_off = pipe.hot_outputs(cur)
        assert int(g_cnt[0]) == len(hot) == int(g_cnt[1])
        assert np.array_equal(g_hot, hot)
        assert np.array_equal(g_freq, freq)
        assert np.array_equal(g_bucket, bucket)
        assert np.array_equal(g_owner_off, owner_off)
        # stage (delta mode: retained rows come from the previous cache;
        # in place: they stay in their slots)
        kk, nc = pipe.k, len(self.cache_refs)
        cache_ref = self.cache_refs[kk % nc]
        H = len(hot)
        if self.inplace:
            X = kk % 2
            sst = ggref.stage_inplace(bucket, owner_off, self.part_ref, self.feat_ref, cache_ref,
                                      self.cstride, self.slot_refs[X],
                                      self.slot_refs[1 - X] if kk > 0 else None,
                                      clear_ids=self.held[X])
            self.held[X] = bucket.copy()
            slots = self.slot_ref[bucket]
            assert np.all(slots >= 0)
            g_rows = pipe.staged_cache()[torch.from_numpy(slots.astype(np.int64)).to(self.dev)]
            assert np.array_equal(g_rows.cpu().numpy()[:, :rb], cache_ref[slots, :rb])
        else:
            src = self.cache_refs[(kk - 1) % nc] if (self.delta and kk > 0) else None
            sst = ggref.stage_bulk(bucket, owner_off, self.part_ref, self.feat_ref, cache_ref,
                                   self.cstride, self.slot_ref, self.prev_ref, src_cache=src,
                                   src_slot_of=self.slot_ref if src is not None else None)
            g_cache = pipe.staged_cache()[:H].cpu().numpy()
            assert np.array_equal(g_cache[:, :rb], cache_ref[:H, :rb])
        self.prev_ref = bucket.copy()
        assert pipe.stage_stats_dict() == sst
        assert np.array_equal(pipe.slot_of.cpu().numpy(), self.slot_ref)
        # gathers, one batch at a time, then the whole window in one launch
        refs, gstats = [], []
        for b in range(Wk):
            out = torch.empty((pipe.out_cap, st), dtype=torch.uint8,
                              device=self.dev)
            pipe.gather(Wk, b, out)
            torch.cuda.synchronize()
            assert pipe.read_status() == 0
            s = L * Wk + b
            ids = fids[foff[s]:foff[s + 1]]
            ref = np.zeros((len(ids), st), dtype=np.uint8)
            gs = ggref.gather_batch(ids, self.part_ref, self.feat_ref, cache_ref,
                                    self.cstride, self.slot_ref, ref, st)
            assert pipe.gather_stats_dict(b) == gs
            gstats.append(gs)
            if check_outputs:
                got = out[:len(ids)].cpu().numpy()
                assert np.array_equal(got[:, :rb], ref[:, :rb]), f"batch {b}"
                refs.append(ref)
            del out
        pipe.gather_stats.zero_()
        win = pipe.gather_window(Wk)
        torch.cuda.synchronize()
        assert pipe.read_status() == 0
        base = foff[L * Wk]
        for b in range(Wk):
            assert pipe.gather_stats_dict(b) == gstats[b]
            if check_outputs:
                lo, hi = foff[L * Wk + b] - base, foff[L * Wk + b + 1] - base
                got = win[lo:hi].cpu().numpy()
                assert np.array_equal(got[:, :rb], refs[b][:, :rb]), f"window batch {b}"
        pipe.k += 1
        return dict(Wk=Wk, fids=fids, foff=foff, nids=nids, noff=noff, hot=hot, stage=sst,
                    outs=refs if check_outputs else None)
