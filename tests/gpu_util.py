"""Shared set-up for the GPU parity tests: the same seeded inputs go to the
HIP path (through the C ABI) and to the CPU oracle; results are compared
byte for byte."""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import ggref
from paper_2606_02916_amd import FetchPipeline, gg


def log(msg):
    print(msg, flush=True)


class World:
    """One workload instance on the GPU and its oracle counterpart."""

    def __init__(self, inst, W=None, n_hot=-1, local_owner=None, fanout=None, batch=None,
                 device="cuda:0", shards=None, row_bytes=None, stride=None, cache_stride=None,
                 tensors=None, delta=False, hot_frac=None, inplace=False, cache_rows=None,
                 tuning=None):
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
                                  inplace=inplace, cache_rows=cache_rows, tuning=tuning)
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
        stage_status = pipe.read_status()
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
        check_bits(bits, pipe.wpb, Wk, lambda b: fids[foff[L * Wk + b]:foff[L * Wk + b + 1]])
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
        short = False
        if self.inplace:
            X = kk % 2
            sst, short = ggref.stage_inplace(bucket, owner_off, self.part_ref, self.feat_ref,
                                             cache_ref, self.cstride, self.slot_refs[X],
                                             self.slot_refs[1 - X] if kk > 0 else None,
                                             clear_ids=self.held[X], allow_short=True)
            self.held[X] = bucket.copy()
            slots = self.slot_ref[bucket]
            slots = slots[slots >= 0]
            assert short or len(slots) == len(bucket)
            g_rows = pipe.staged_cache()[torch.from_numpy(slots.astype(np.int64)).to(self.dev)]
            assert np.array_equal(g_rows.cpu().numpy()[:, :rb], cache_ref[slots, :rb])
        else:
            src = self.cache_refs[(kk - 1) % nc] if (self.delta and kk > 0) else None
            sst = ggref.stage_bulk(bucket, owner_off, self.part_ref, self.feat_ref, cache_ref,
                                   self.cstride, self.slot_ref, self.prev_ref, src_cache=src,
                                   src_slot_of=self.slot_ref if src is not None else None)
            g_cache = pipe.staged_cache()[:H].cpu().numpy()
            assert np.array_equal(g_cache[:, :rb], cache_ref[:H, :rb])
        # a persistent cache too small for two windows flags the shortfall
        assert stage_status == (gg.DEV_CAPACITY if short else 0), (stage_status, short)
        if short:
            pipe.status.zero_()
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
        # the whole window in one launch, as the sequential driver gathers it
        # and with the look-ahead's flag (other tiles, fewer loads in flight);
        # the output is overwritten with a pattern first
        base = foff[L * Wk]
        for flags in (0, gg.GG_GATHER_SHARED):
            pipe.gather_stats.zero_()
            pipe.win_out.fill_(0xA5)
            win = pipe.gather_window(Wk, flags=flags)
            torch.cuda.synchronize()
            assert pipe.read_status() == 0
            for b in range(Wk):
                assert pipe.gather_stats_dict(b) == gstats[b]
                if check_outputs:
                    lo, hi = foff[L * Wk + b] - base, foff[L * Wk + b + 1] - base
                    got = win[lo:hi].cpu().numpy()
                    assert np.array_equal(got[:, :rb], refs[b][:, :rb]), \
                        f"window batch {b}, flags {flags}"
        pipe.k += 1
        return dict(Wk=Wk, fids=fids, foff=foff, nids=nids, noff=noff, hot=hot, stage=sst,
                    outs=refs if check_outputs else None, short=short)


def check_bits(words, wpb, Wk, ids_of_batch):
    """The W bit sets hold exactly N_b: every id's bit is set and each set
    has as many bits as N_b has ids."""
    for b in range(Wk):
        row = words[b * wpb:(b + 1) * wpb]
        ids = ids_of_batch(b)
        assert int(np.bitwise_count(row).sum()) == len(ids), f"bit set of batch {b}"
        if len(ids):
            assert np.all((row[ids >> 5] >> (ids & 31).astype(np.uint32)) & 1), \
                f"bit set of batch {b}"


class LookaheadOracle:
    """The oracle's run of consecutive windows as the look-ahead driver
    computes them (delta staging into one persistent cache), checked against
    a finished window's buffer set element by element: every batch's
    frontiers and neighbour slots, the bit sets, hot set, frequencies,
    counts, buckets and owner offsets, the staging statistics, the whole
    remap, every staged row at its slot, the gather statistics and every
    gathered row."""

    def __init__(self, inst, look, n_hot=-1, shards=None, hot_frac=None):
        wl = inst.wl
        self.inst, self.look, self.n_hot, self.hot_frac = inst, look, n_hot, hot_frac
        self.shards = inst.shards if shards is None else shards
        self.P, self.L = wl.num_parts, len(look.fanout)
        self.part = ggref.make_part(self.P, wl.part_kind, wl.local_owner, wl.num_nodes,
                                    inst.range_start)
        self.feat = ggref.make_feat(look.row_bytes, self.shards, [look.stride] * self.P)
        self.cache = np.zeros((look.cache_rows, look.cache_stride), dtype=np.uint8)
        # one remap per buffer set of the driver, each cleared of the window
        # that last used the set
        self.remaps = [np.full(wl.num_nodes, -1, dtype=np.int32) for _ in range(look.nsets)]
        self.held = [None] * look.nsets
        self.k = 0

    def check(self, k, Wk, bufs, seeds, so, b0, rng_seed=0, epoch=0):
        """Window k (the next one in order) after its gather finished."""
        assert k == self.k
        look, L, rb = self.look, self.L, self.look.row_bytes
        torch.cuda.synchronize()
        fids, foff, nids, noff = ggref.sample_window(self.inst.row_ptr, self.inst.col_idx, seeds,
                                                     so, look.fanout, rng_seed, epoch, b0)
        g_foff = bufs.frontier_off[:(L + 1) * Wk + 1].cpu().numpy()
        g_noff = bufs.nbr_off[:L * Wk + 1].cpu().numpy()
        assert np.array_equal(g_foff, foff), f"window {k} frontier offsets"
        assert np.array_equal(g_noff, noff), f"window {k} neighbour offsets"
        assert np.array_equal(bufs.frontier_ids[:int(foff[-1])].cpu().numpy(), fids), \
            f"window {k} frontiers"
        assert np.array_equal(bufs.nbr_ids[:int(noff[-1])].cpu().numpy(), nids), \
            f"window {k} neighbour slots"
        wpb = look.geo.wpb
        words = bufs.frontier_bits.view(torch.int32)[:Wk * wpb].cpu().numpy().view(np.uint32)
        check_bits(words, wpb, Wk, lambda b: fids[foff[L * Wk + b]:foff[L * Wk + b + 1]])
        hot, freq = ggref.build_hotset(fids, foff, Wk, L, self.part, self.n_hot,
                                       hot_frac=self.hot_frac)
        bucket, owner_off = ggref.bucket_by_owner(hot, self.part)
        T = k % look.NSLOT
        cnt = look.hot_count[T].cpu().numpy()
        assert int(cnt[0]) == len(hot) == int(cnt[1]), f"window {k} hot count"
        assert np.array_equal(bufs.hot_ids[:len(hot)].cpu().numpy(), hot), f"window {k} hot set"
        assert np.array_equal(bufs.hot_freq[:len(hot)].cpu().numpy(), freq), f"window {k} freq"
        assert np.array_equal(look.bucket_ids[T][:len(hot)].cpu().numpy(), bucket), \
            f"window {k} buckets"
        assert np.array_equal(bufs.owner_off.cpu().numpy(), owner_off), f"window {k} owner_off"
        X, ns = k % look.nsets, look.nsets
        sst, short = ggref.stage_inplace(bucket, owner_off, self.part, self.feat, self.cache,
                                         look.cache_stride, self.remaps[X],
                                         self.remaps[(k - 1) % ns] if k > 0 else None,
                                         clear_ids=self.held[X], allow_short=True)
        assert not short
        self.held[X] = bucket.copy()
        assert bufs.stage_stats_dict() == sst, f"window {k} staging statistics"
        remap = self.remaps[X]
        assert np.array_equal(bufs.slot_of.cpu().numpy(), remap), f"window {k} remap"
        slots = remap[bucket].astype(np.int64)
        got = look.cache[torch.from_numpy(slots).to(look.device)][:, :rb].cpu().numpy()
        assert np.array_equal(got, self.cache[slots, :rb]), f"window {k} staged rows"
        base = int(foff[L * Wk])
        win = bufs.win_out[:int(foff[-1]) - base, :rb].cpu().numpy()
        for b in range(Wk):
            s = L * Wk + b
            ids = fids[foff[s]:foff[s + 1]]
            ref = np.zeros((len(ids), look.stride), dtype=np.uint8)
            gs = ggref.gather_batch(ids, self.part, self.feat, self.cache, look.cache_stride,
                                    remap, ref, look.stride)
            assert bufs.gather_stats_dict(b) == gs, f"window {k} batch {b} gather statistics"
            lo, hi = foff[s] - base, foff[s + 1] - base
            assert np.array_equal(win[lo:hi], ref[:, :rb]), f"window {k} batch {b} rows"
        self.k += 1
        return dict(Wk=Wk, hot=hot, stage=sst, fids=fids, foff=foff)
