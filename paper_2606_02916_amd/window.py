"""Window driver: device buffers (torch allocations) and the call sequence
of one window through libgg.  Orchestration only; every step runs in the
library's kernels, on one stream, with no host synchronisation inside a
window.

Algorithm 1 of the paper (GreenGNN, arXiv 2606.02916) per window k:
sample the W batches, build H_k, group it by owner, stage the cache with
one bulk copy per owner (clearing window k-1's remap entries), then gather
every batch's input rows through the remap with the miss path.
"""
from __future__ import annotations

import numpy as np
import torch

from . import gg


class FetchPipeline:
    def __init__(self, row_ptr, col_idx, num_parts, part_kind, local_owner, range_start, shards,
                 shard_rows, row_bytes, stride, W, fanout, max_batch, n_hot=-1, device=None,
                 out_buffers=2, cache_stride=None):
        self.device = torch.device(device if device is not None else "cuda")
        self.N = int(row_ptr.numel() - 1)
        self.W = int(W)
        self.fanout = [int(k) for k in fanout]
        self.L = len(self.fanout)
        self.P = int(num_parts)
        self.row_bytes = int(row_bytes)
        self.stride = int(stride)
        # Cache rows are packed at the feature stride: neighbouring slots
        # share HBM sectors, which a sparse ascending gather reuses.
        self.cache_stride = int(cache_stride) if cache_stride else self.stride
        self.n_hot = int(n_hot)
        self.row_ptr, self.col_idx = row_ptr, col_idx
        self.shards = shards
        self.csr = gg.make_csr(row_ptr, col_idx)
        self.part = gg.make_part(self.P, part_kind, local_owner, self.N, range_start)
        self.feat = gg.make_feat(self.row_bytes, shards, [self.stride] * self.P, shard_rows)
        dev = self.device
        fcap, ncap = gg.gg_sample_caps(self.N, self.W, max_batch, self.fanout)
        self.frontier_ids = torch.empty(max(fcap, 1), dtype=torch.int32, device=dev)
        self.frontier_off = torch.zeros((self.L + 1) * self.W + 1, dtype=torch.int64, device=dev)
        self.nbr_ids = torch.empty(max(ncap, 1), dtype=torch.int32, device=dev)
        self.nbr_off = torch.zeros(self.L * self.W + 1, dtype=torch.int64, device=dev)
        self.wpb = gg.gg_bits_words(self.N)
        self.frontier_bits = torch.empty(self.W * self.wpb, dtype=torch.int32, device=dev)
        self.need = torch.zeros(2, dtype=torch.int64, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.wsample = gg.make_wsample(self.frontier_ids, self.frontier_off, self.nbr_ids,
                                       self.nbr_off, self.frontier_bits, self.need)
        # Per-batch bound of |N_b| and of the window's remote nodes.
        lev = min(max_batch, self.N)
        for k in self.fanout:
            lev = min(self.N, lev * (k + 1))
        self.out_cap = max(lev, 1)
        remote = self.N - (int(shard_rows[local_owner]) if local_owner >= 0 else 0)
        self.hot_cap = max(1, min(remote, self.W * self.out_cap))
        self.hot_ids = torch.empty(self.hot_cap, dtype=torch.int32, device=dev)
        self.hot_freq = torch.empty(self.hot_cap, dtype=torch.int32, device=dev)
        self.hot_count = [torch.zeros(2, dtype=torch.int64, device=dev) for _ in range(2)]
        self.bucket_ids = [torch.empty(self.hot_cap, dtype=torch.int32, device=dev)
                           for _ in range(2)]
        self.owner_off = torch.zeros(self.P + 1, dtype=torch.int64, device=dev)
        self.cache = torch.empty((self.hot_cap, self.cache_stride), dtype=torch.uint8, device=dev)
        self.slot_of = torch.full((self.N,), -1, dtype=torch.int32, device=dev)
        self.win_cap = self.W * self.out_cap
        ws_bytes = max(gg.gg_ws_sample(self.N, self.W), gg.gg_ws_hotset(self.N, self.W),
                       gg.gg_ws_bucket(self.hot_cap, self.P), gg.gg_ws_stage(self.hot_cap, self.P),
                       gg.gg_ws_gather(self.out_cap, 1, self.P),
                       gg.gg_ws_gather(self.win_cap, self.W, self.P))
        self.ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        self.stage_stats = torch.zeros(gg.STAGE_STATS_BYTES, dtype=torch.uint8, device=dev)
        self.gather_stats = torch.zeros((self.W, gg.GATHER_STATS_BYTES), dtype=torch.uint8,
                                        device=dev)
        self.outs = [torch.empty((self.out_cap, self.stride), dtype=torch.uint8, device=dev)
                     for _ in range(out_buffers)]
        self._win_out = None
        self.k = 0

    @property
    def win_out(self):
        """Output of a whole-window gather: the W batches' rows back to back."""
        if self._win_out is None:
            self._win_out = torch.empty((self.win_cap, self.stride), dtype=torch.uint8,
                                        device=self.device)
        return self._win_out

    def reset_cache(self):
        self.slot_of.fill_(-1)
        self.k = 0

    # -- the five calls of one window ------------------------------------
    def sample(self, seeds, seed_off, batch0, epoch=0, rng_seed=0):
        Wk = len(seed_off) - 1
        gg.gg_sample_window(self.csr, seeds, seed_off, Wk, self.fanout, self.L, rng_seed, epoch,
                            batch0, self.wsample, self.status, self.ws)
        return Wk

    def hotset(self, Wk, cur):
        gg.gg_build_hotset(self.frontier_bits, Wk, self.part, self.n_hot, self.hot_ids,
                           self.hot_freq, self.hot_cap, self.hot_count[cur], self.status, self.ws)

    def bucket(self, cur):
        gg.gg_bucket_by_owner(self.hot_ids, self.hot_count[cur], self.hot_cap, self.part,
                              self.bucket_ids[cur], self.owner_off, self.status, self.ws)

    def stage(self, cur):
        prev = 1 - cur
        have_prev = self.k > 0
        gg.gg_stage_bulk(self.bucket_ids[cur], self.owner_off, self.hot_cap, self.part, self.feat,
                         self.cache, self.cache_stride, self.hot_cap, self.slot_of,
                         self.bucket_ids[prev] if have_prev else None,
                         self.hot_count[prev] if have_prev else None, self.stage_stats,
                         self.status, self.ws)

    def gather(self, Wk, b, out):
        """Batch b of the window into out (one launch)."""
        bounds = self.frontier_off.data_ptr() + 8 * (self.L * Wk + b)
        stats = self.gather_stats.data_ptr() + b * gg.GATHER_STATS_BYTES
        gg.gg_gather_batch(self.frontier_ids, bounds, 1, out.shape[0], self.part, self.feat,
                           self.cache, self.cache_stride, self.hot_cap, self.slot_of, out,
                           self.stride, stats, self.status, self.ws)

    def gather_window(self, Wk, out=None):
        """All Wk batches of the window in one launch; batch b's rows start at
        row frontier_off[L*Wk + b] - frontier_off[L*Wk] of out."""
        out = self.win_out if out is None else out
        bounds = self.frontier_off.data_ptr() + 8 * (self.L * Wk)
        gg.gg_gather_batch(self.frontier_ids, bounds, Wk, out.shape[0], self.part, self.feat,
                           self.cache, self.cache_stride, self.hot_cap, self.slot_of, out,
                           self.stride, self.gather_stats.data_ptr(), self.status, self.ws)
        return out

    def window(self, seeds, seed_off, batch0, epoch=0, rng_seed=0, outs=None, events=None,
               gather_events=None, per_batch=False):
        """Enqueues one window.  By default the W gathers run as one launch
        into win_out; with per_batch=True every batch is its own launch into
        outs[b] (default: the driver's ping-pong buffers).  events: optional
        list of 6 torch events recorded between the calls; gather_events:
        optional list of (start, end) event pairs, one per gather launch."""
        cur = self.k & 1
        ev = events if events is not None else [None] * 6
        _rec(ev[0])
        Wk = self.sample(seeds, seed_off, batch0, epoch, rng_seed)
        _rec(ev[1])
        self.hotset(Wk, cur)
        _rec(ev[2])
        self.bucket(cur)
        _rec(ev[3])
        self.stage(cur)
        _rec(ev[4])
        if per_batch:
            for b in range(Wk):
                out = outs[b] if outs is not None else self.outs[b % len(self.outs)]
                if gather_events is not None:
                    gather_events[b][0].record()
                self.gather(Wk, b, out)
                if gather_events is not None:
                    gather_events[b][1].record()
        else:
            if gather_events is not None:
                gather_events[0][0].record()
            self.gather_window(Wk, outs)
            if gather_events is not None:
                gather_events[0][1].record()
        _rec(ev[5])
        self.k += 1
        return Wk

    # -- host copies for checking ------------------------------------------
    def read_status(self):
        return int(self.status.item())

    def sample_outputs(self, Wk):
        foff = self.frontier_off[:(self.L + 1) * Wk + 1].cpu().numpy()
        noff = self.nbr_off[:self.L * Wk + 1].cpu().numpy()
        fids = self.frontier_ids[:int(foff[-1])].cpu().numpy()
        nids = self.nbr_ids[:int(noff[-1])].cpu().numpy()
        return fids, foff, nids, noff

    def hot_outputs(self, cur=None):
        cur = ((self.k - 1) & 1) if cur is None else cur
        cnt = self.hot_count[cur].cpu().numpy()
        n = int(cnt[0])
        return (self.hot_ids[:n].cpu().numpy(), self.hot_freq[:n].cpu().numpy(), cnt,
                self.bucket_ids[cur][:n].cpu().numpy(), self.owner_off.cpu().numpy())

    def stage_stats_dict(self):
        return gg.stage_stats_from_bytes(self.stage_stats.cpu().numpy().tobytes(), self.P)

    def gather_stats_dict(self, b):
        return gg.gather_stats_from_bytes(self.gather_stats[b].cpu().numpy().tobytes(), self.P)


def _rec(e):
    if e is not None:
        e.record()
