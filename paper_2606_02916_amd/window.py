"""Window drivers: device buffers (torch allocations) and the call sequence
of a window through libgg.  Orchestration only; every step runs in the
library's kernels and no host synchronisation happens inside a window.

Algorithm 1 of the paper (GreenGNN, arXiv 2606.02916) per window k: sample
the W batches, build H_k, group it by owner, rebuild the cache with one
bulk request per owner, then gather every batch's input rows through the
ID-to-slot remap with the miss path.

FetchPipeline runs the five calls in order on one stream.  With delta=True
it keeps two caches and requests only the rebuild delta
Delta_{k,m} = (H_k in owner m) minus C_{k-1} from the owners, copying the
rows it retains from the previous cache (Sec. IV-A, Eq. (1)); with
inplace=True it keeps one persistent cache in which those rows stay where
they are.  LookaheadPipeline is the paper's pipelined runtime (Algorithm 1,
Sec. IV-C) on a persistent cache: window k+1 is sampled, bucketed and
staged while window k is gathered.
"""
from __future__ import annotations

import torch

from . import gg


# Largest sampler byte map (MB) the look-ahead driver lets a sparse last hop
# use: above it the map's scattered writes, clearing and folding cost more
# HBM traffic than atomic marks into the bit sets.
LOOKAHEAD_BYTEMAP_MAX_MB = 8


def _last_frontier_bound(num_nodes, fanout, max_batch):
    """min(N, B * prod_{i<L-1}(k_i + 1)): the bound on a batch's entries at
    the last hop."""
    f = min(num_nodes, max_batch)
    for k in fanout[:-1]:
        f = min(num_nodes, f * (k + 1))
    return f


def last_hop_density(num_nodes, fanout, max_batch):
    """Bound on the last hop's draws per batch over the node count:
    min(N, B * prod_{i<L-1}(k_i + 1)) * k_{L-1} / N."""
    return _last_frontier_bound(num_nodes, fanout, max_batch) * fanout[-1] / max(num_nodes, 1)


def last_hop_sharing(num_nodes, fanout, max_batch, W):
    """Bound on the number of a window's batches whose last-hop frontier
    holds a given node: W * min(N, B * prod_{i<L-1}(k_i + 1)) / N."""
    return W * _last_frontier_bound(num_nodes, fanout, max_batch) / max(num_nodes, 1)


# The look-ahead driver's streams, created once per device and shared by
# every look-ahead pipeline on it.  HIP spreads a process's streams over a
# few hardware queues (four by default) in an order the caller does not
# control, and two of a pipeline's streams on one queue run its chains one
# after the other: building six pipelines in turn on the 2.45M-node graph
# (batch 4096, W = 4), the fourth and fifth ran at 0.418 and 0.342 ms per
# window against 0.296-0.302 for the others, and at 0.296-0.300 all six
# when they reused the first one's streams.  Pipelines driven from one
# thread at a time lose nothing by sharing them.
_STREAMS = {}


def _driver_streams(dev):
    idx = torch.device(dev).index
    if idx is None:
        idx = torch.cuda.current_device()
    if idx not in _STREAMS:
        _STREAMS[idx] = tuple(torch.cuda.Stream(device=idx) for _ in range(3))
    return _STREAMS[idx]


def _bucket_flags(part):
    """The hot set comes out ascending, which under a range book is owner
    order: bucketing is then one copy pass."""
    return gg.GG_BUCKET_OWNER_ORDERED if part.kind == gg.PART_RANGE else 0


class _Geometry:
    """Sizes shared by all buffer sets of a pipeline."""

    def __init__(self, N, W, fanout, max_batch, P, local_owner, shard_rows, stride, cache_stride,
                 tuning=None):
        self.N, self.W, self.P = N, W, P
        self.fanout = [int(k) for k in fanout]
        self.L = len(self.fanout)
        self.stride = stride
        self.cache_stride = cache_stride
        self.fcap, self.ncap = gg.gg_sample_caps(N, W, max_batch, self.fanout)
        self.wpb = gg.gg_bits_words(N)
        lev = min(max_batch, N)
        for k in self.fanout:
            lev = min(N, lev * (k + 1))
        self.out_cap = max(lev, 1)                      # rows of one N_b
        remote = N - (int(shard_rows[local_owner]) if local_owner >= 0 else 0)
        self.hot_cap = max(1, min(remote, W * self.out_cap))
        # a persistent cache holds two consecutive windows' hot sets
        self.inplace_rows = max(1, min(remote, 2 * W * self.out_cap))
        self.win_cap = W * self.out_cap                 # rows of a whole window
        self.seed_cap = W * max(min(max_batch, N), 1)   # F_0 rows of a whole window
        self.ws_bytes = max(gg.gg_ws_sample(N, W, tuning), gg.gg_ws_hotset(N, W, tuning),
                            gg.gg_ws_bucket(self.hot_cap, P), gg.gg_ws_stage(self.hot_cap, P),
                            gg.gg_ws_gather(self.out_cap, 1, P, tuning),
                            gg.gg_ws_gather(self.win_cap, W, P, tuning))
        # hot set and bucketing, while the sampler's workspace still serves
        # the last level's compaction on another stream
        self.ws2_bytes = max(gg.gg_ws_hotset(N, W, tuning), gg.gg_ws_bucket(self.hot_cap, P))


class _Buffers:
    """Everything one window writes: sampling outputs, hot set, cache and
    remap, workspace, statistics and (lazily) the window's gathered rows.
    With own_cache=False the cache is the pipeline's persistent one and the
    set holds an occupancy bitmap of it instead."""

    def __init__(self, g: _Geometry, dev, own_cache=True, split=False):
        self.g, self.dev = g, dev
        self.frontier_ids = torch.empty(max(g.fcap, 1), dtype=torch.int32, device=dev)
        self.frontier_off = torch.zeros((g.L + 1) * g.W + 1, dtype=torch.int64, device=dev)
        self.nbr_ids = torch.empty(max(g.ncap, 1), dtype=torch.int32, device=dev)
        self.nbr_off = torch.zeros(g.L * g.W + 1, dtype=torch.int64, device=dev)
        self.frontier_bits = torch.empty(g.W * g.wpb, dtype=torch.int32, device=dev)
        self.need = torch.zeros(2, dtype=torch.int64, device=dev)
        self.wsample = gg.make_wsample(self.frontier_ids, self.frontier_off, self.nbr_ids,
                                       self.nbr_off, self.frontier_bits, self.need)
        self.hot_ids = torch.empty(g.hot_cap, dtype=torch.int32, device=dev)
        self.hot_freq = torch.empty(g.hot_cap, dtype=torch.int32, device=dev)
        self.owner_off = torch.zeros(g.P + 1, dtype=torch.int64, device=dev)
        self.cache = (torch.empty((g.hot_cap, g.cache_stride), dtype=torch.uint8, device=dev)
                      if own_cache else None)
        self.occ = (None if own_cache else
                    torch.zeros(gg.occ_bytes(g.inplace_rows), dtype=torch.uint8, device=dev))
        self.slot_of = torch.full((g.N,), -1, dtype=torch.int32, device=dev)
        self.ws = torch.empty(g.ws_bytes, dtype=torch.uint8, device=dev)
        self.ws2 = torch.empty(g.ws2_bytes, dtype=torch.uint8, device=dev) if split else self.ws
        self.stage_stats = torch.zeros(gg.STAGE_STATS_BYTES, dtype=torch.uint8, device=dev)
        self.gather_stats = torch.zeros((g.W, gg.GATHER_STATS_BYTES), dtype=torch.uint8,
                                        device=dev)
        self._win_out = None

    def stage_stats_dict(self):
        return gg.stage_stats_from_bytes(self.stage_stats.cpu().numpy().tobytes(), self.g.P)

    def gather_stats_dict(self, b):
        return gg.gather_stats_from_bytes(self.gather_stats[b].cpu().numpy().tobytes(), self.g.P)

    @property
    def win_out(self):
        if self._win_out is None:
            self._win_out = torch.empty((self.g.win_cap, self.g.stride), dtype=torch.uint8,
                                        device=self.dev)
        return self._win_out


class FetchPipeline:
    def __init__(self, row_ptr, col_idx, num_parts, part_kind, local_owner, range_start, shards,
                 shard_rows, row_bytes, stride, W, fanout, max_batch, n_hot=-1, device=None,
                 out_buffers=2, cache_stride=None, delta=False, hot_frac=None, inplace=False,
                 cache_rows=None, tuning=None):
        """delta: rebuild the cache from the previous window's, requesting only
        the rebuild delta; the cache then alternates between two buffers and
        the rows still wanted are copied across.  inplace (implies delta):
        one persistent cache in which those rows stay put (gg_stage_inplace);
        the remap then alternates between two buffers.  cache_rows (in place
        only): slots of the persistent cache, by default enough for two
        windows' hot sets; fewer leave rows to the miss path.  tuning: a
        gg_tuning_t (gg.make_tuning) passed to every call, or None."""
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
        self.hot_frac = hot_frac
        self.inplace = bool(inplace)
        self.delta = bool(delta) or self.inplace
        self.row_ptr, self.col_idx = row_ptr, col_idx
        self.shards = shards
        self.csr = gg.make_csr(row_ptr, col_idx)
        self.part = gg.make_part(self.P, part_kind, local_owner, self.N, range_start)
        self.feat = gg.make_feat(self.row_bytes, shards, [self.stride] * self.P, shard_rows)
        # Alone on the chip the sampler's mark blocks may take whole CUs:
        # 1,024 lanes (the library's 256 leave room beside a running gather)
        # took the 2.45M-node window from 0.509 to 0.492 ms.  A caller's
        # tuning replaces this one as a whole.
        if tuning is None:
            tuning = gg.make_tuning(mark_block=1024)
        self.tuning = tuning
        self.geo = _Geometry(self.N, self.W, self.fanout, max_batch, self.P, local_owner,
                             shard_rows, self.stride, self.cache_stride, tuning)
        g, dev = self.geo, self.device
        self.out_cap, self.hot_cap, self.win_cap, self.wpb = g.out_cap, g.hot_cap, g.win_cap, g.wpb
        self.buf = _Buffers(g, dev, own_cache=not self.inplace)
        b = self.buf
        for name in ("frontier_ids", "frontier_off", "nbr_ids", "nbr_off", "frontier_bits", "need",
                     "wsample", "hot_ids", "hot_freq", "owner_off", "ws",
                     "stage_stats", "gather_stats"):
            setattr(self, name, getattr(b, name))
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        # Hot-set counts and bucket lists of the last nslot windows: the
        # in-place remap of window k last held window k - 2, whose list
        # clears it.
        self.nslot = 3 if self.inplace else 2
        self.hot_count = [torch.zeros(2, dtype=torch.int64, device=dev)
                          for _ in range(self.nslot)]
        self.bucket_ids = [torch.empty(g.hot_cap, dtype=torch.int32, device=dev)
                           for _ in range(self.nslot)]
        if self.inplace:
            rows = g.inplace_rows if cache_rows is None else int(cache_rows)
            self.cache_rows = rows
            self.caches = [torch.empty((max(rows, 1), self.cache_stride), dtype=torch.uint8,
                                       device=dev)]
            self.slot_ofs = [b.slot_of, torch.full_like(b.slot_of, -1)]
            self.occs = [torch.zeros(gg.occ_bytes(rows), dtype=torch.uint8, device=dev)
                         for _ in range(2)]
            self.stage_ws = torch.empty(gg.gg_ws_stage_inplace(g.hot_cap, rows, self.P),
                                        dtype=torch.uint8, device=dev)
        else:
            # With delta staging the cache alternates between two buffers.
            self.cache_rows = g.hot_cap
            self.caches = [b.cache] + ([torch.empty_like(b.cache)] if self.delta else [])
            self.slot_ofs = [b.slot_of]
        self.outs = [torch.empty((g.out_cap, self.stride), dtype=torch.uint8, device=dev)
                     for _ in range(out_buffers)]
        self.k = 0

    @property
    def cache(self):
        """The cache of the most recently staged window."""
        return self.caches[(self.k - 1) % len(self.caches)] if self.k else self.caches[0]

    @property
    def slot_of(self):
        """The remap of window k (= self.k, advanced after the gathers)."""
        return self.slot_ofs[self.k % len(self.slot_ofs)]

    @property
    def win_out(self):
        """Output of a whole-window gather: the W batches' rows back to back."""
        return self.buf.win_out

    def reset_cache(self):
        for r in self.slot_ofs:
            r.fill_(-1)
        self.k = 0

    # -- the five calls of one window ------------------------------------
    def sample(self, seeds, seed_off, batch0, epoch=0, rng_seed=0):
        Wk = len(seed_off) - 1
        gg.gg_sample_window(self.csr, seeds, seed_off, Wk, self.fanout, self.L, rng_seed, epoch,
                            batch0, self.wsample, self.status, self.ws, tuning=self.tuning)
        return Wk

    def hotset(self, Wk, cur):
        gg.gg_build_hotset(self.frontier_bits, Wk, self.part, self.n_hot, self.hot_ids,
                           self.hot_freq, self.hot_cap, self.hot_count[cur], self.status, self.ws,
                           hot_frac=self.hot_frac, tuning=self.tuning)

    def bucket(self, cur):
        gg.gg_bucket_by_owner(self.hot_ids, self.hot_count[cur], self.hot_cap, self.part,
                              self.bucket_ids[cur], self.owner_off, self.status, self.ws,
                              flags=_bucket_flags(self.part))

    def slot_index(self):
        """Hot-set and bucket slot of window k (= self.k)."""
        return self.k % self.nslot

    def stage(self, cur):
        """Rebuilds the cache for window k (= self.k, advanced by the caller)."""
        if self.inplace:
            k = self.k
            X = k % 2
            old = (k - 2) % self.nslot          # the window this remap held
            gg.gg_stage_inplace(self.bucket_ids[cur], self.owner_off, self.hot_cap, self.part,
                                self.feat, self.caches[0], self.cache_stride, self.cache_rows,
                                self.slot_ofs[X], self.bucket_ids[old] if k >= 2 else None,
                                self.hot_count[old] if k >= 2 else None,
                                self.slot_ofs[1 - X] if k >= 1 else None,
                                self.occs[1 - X] if k >= 1 else None, self.occs[X],
                                self.stage_stats, self.status, self.stage_ws, tuning=self.tuning)
            return
        prev = (cur - 1) % self.nslot
        have_prev = self.k > 0
        nc = len(self.caches)
        cache = self.caches[self.k % nc]
        src = self.caches[(self.k - 1) % nc] if (self.delta and have_prev) else None
        gg.gg_stage_bulk(self.bucket_ids[cur], self.owner_off, self.hot_cap, self.part, self.feat,
                         cache, self.cache_stride, self.hot_cap, self.slot_of,
                         self.bucket_ids[prev] if have_prev else None,
                         self.hot_count[prev] if have_prev else None,
                         src, self.slot_of if src is not None else None, self.stage_stats,
                         self.status, self.ws, tuning=self.tuning)

    def staged_cache(self):
        """The cache stage() just filled (valid until the window advances)."""
        return self.caches[self.k % len(self.caches)]

    def gather(self, Wk, b, out):
        """Batch b of the window into out (one launch)."""
        bounds = self.frontier_off.data_ptr() + 8 * (self.L * Wk + b)
        stats = self.gather_stats.data_ptr() + b * gg.GATHER_STATS_BYTES
        gg.gg_gather_batch(self.frontier_ids, bounds, 1, out.shape[0], self.part, self.feat,
                           self.staged_cache(), self.cache_stride, self.cache_rows, self.slot_of,
                           out, self.stride, stats, self.status, self.ws, tuning=self.tuning)

    def gather_window(self, Wk, out=None, flags=0):
        """All Wk batches of the window in one launch; batch b's rows start at
        row frontier_off[L*Wk + b] - frontier_off[L*Wk] of out.  flags:
        gg_gather_batch's (GG_GATHER_SHARED: the look-ahead's tiles and
        loads in flight)."""
        out = self.win_out if out is None else out
        bounds = self.frontier_off.data_ptr() + 8 * (self.L * Wk)
        gg.gg_gather_batch(self.frontier_ids, bounds, Wk, out.shape[0], self.part, self.feat,
                           self.staged_cache(), self.cache_stride, self.cache_rows, self.slot_of,
                           out, self.stride, self.gather_stats.data_ptr(), self.status, self.ws,
                           flags=flags, tuning=self.tuning)
        return out

    def capture_window(self, seeds, seed_off, batch0, epoch=0, rng_seed=0):
        """Captures one whole window into a HIP graph on the current stream:
        the remap reset (a fill kernel), then sampling, hot set, buckets,
        staging and the whole-window gather into win_out.  Every replay
        recomputes the window from `seeds` (refill it in place between
        replays to change the seeds; its length and seed_off stay as
        captured) into the same buffers, so a replay costs its kernels and
        not their launches.  Full restage only: a replay starts from an empty
        cache.  Returns (graph, number of batches)."""
        if self.delta:
            raise ValueError("graph capture replays full restages only")
        self.win_out                       # allocated before the capture
        cur = torch.cuda.current_stream(self.device)
        side = torch.cuda.Stream(device=self.device)
        side.wait_stream(cur)
        with torch.cuda.stream(side):      # one eager pass first
            self.reset_cache()
            self.window(seeds, seed_off, batch0, epoch, rng_seed)
        cur.wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            self.reset_cache()
            Wk = self.window(seeds, seed_off, batch0, epoch, rng_seed)
        return graph, Wk

    def sim_accumulate(self, Wk, coeffs, acc):
        """Adds the window just gathered to the simulator totals `acc` (a
        device buffer of SIM_ACC_BYTES, zeroed before the first window)."""
        gg.gg_sim_accumulate(self.stage_stats, self.gather_stats.data_ptr(), Wk, self.part,
                             coeffs, acc)

    def window(self, seeds, seed_off, batch0, epoch=0, rng_seed=0, outs=None, events=None,
               gather_events=None, per_batch=False, sim=None, consumer=None,
               consumer_events=None):
        """Enqueues one window.  By default the W gathers run as one launch
        into win_out; with per_batch=True every batch is its own launch into
        outs[b] (default: the driver's ping-pong buffers).  events: optional
        list of 6 torch events recorded between the calls; gather_events:
        optional list of (start, end) event pairs, one per gather launch;
        sim: optional (coeffs, acc) to add the window to simulator totals;
        consumer: optional SageConsumer run on the window's rows (whole-window
        gather only), bracketed by the optional event pair consumer_events."""
        cur = self.slot_index()
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
        if sim is not None:
            self.sim_accumulate(Wk, *sim)
        if consumer is not None:
            if per_batch:
                raise ValueError("the consumer reads a whole-window gather")
            _rec(consumer_events[0] if consumer_events else None)
            consumer.forward(self.buf, Wk, outs if outs is not None else self.win_out,
                             self.stride, self.status)
            _rec(consumer_events[1] if consumer_events else None)
        self.k += 1
        return Wk

    # -- host copies for checking ------------------------------------------
    def read_status(self):
        return gg.gg_read_status(self.status)

    def sample_outputs(self, Wk):
        foff = self.frontier_off[:(self.L + 1) * Wk + 1].cpu().numpy()
        noff = self.nbr_off[:self.L * Wk + 1].cpu().numpy()
        fids = self.frontier_ids[:int(foff[-1])].cpu().numpy()
        nids = self.nbr_ids[:int(noff[-1])].cpu().numpy()
        return fids, foff, nids, noff

    def hot_outputs(self, cur=None):
        cur = ((self.k - 1) % self.nslot) if cur is None else cur
        cnt = self.hot_count[cur].cpu().numpy()
        n = int(cnt[0])
        return (self.hot_ids[:n].cpu().numpy(), self.hot_freq[:n].cpu().numpy(), cnt,
                self.bucket_ids[cur][:n].cpu().numpy(), self.owner_off.cpu().numpy())

    def stage_stats_dict(self):
        return gg.stage_stats_from_bytes(self.stage_stats.cpu().numpy().tobytes(), self.P)

    def gather_stats_dict(self, b):
        return gg.gather_stats_from_bytes(self.gather_stats[b].cpu().numpy().tobytes(), self.P)


class LookaheadPipeline:
    """Pipelined runtime: window k+1 is built (sampled, its hot set formed
    and bucketed by owner) and its cache staged while window k is gathered,
    so a window costs about the longer of the two chains instead of their
    sum.

    Staging follows the build on the build stream and the fetch stream only
    gathers: staging window k+1 (which writes its own buffer set and reads
    window k's cache) runs beside window k's gather.  Where staging would
    hold up the next build (stage_apart: by default when shards live in
    pinned host memory, where staging is bound by PCIe, and when the build
    is the longer chain), it runs on the fetch stream instead and the gather
    gets a stream of its own, running beside the next window's staging.

    The cache is one persistent buffer (gg_stage_inplace): a row window k
    shares with window k-1 stays in its slot, and only the delta is
    fetched, into slots window k-1 does not occupy.  `nsets` buffer sets
    (remap, occupancy map, sampling outputs) rotate over the windows (window
    k uses set k mod nsets); the default is three with shards in device
    memory and two otherwise.  Building window k waits for the gather of
    window k - nsets, the last reader of its set; with more sets the build
    may run further ahead.  Staging window k waits for the gather of window
    k - 2, whose slots it may reuse.  Bucket lists and hot-set counts rotate
    over 2 * nsets slots: staging window k reads slot k and clears its remap
    with the slot of window k - nsets while windows up to k + nsets - 1 are
    being built.  Every other reuse is ordered through these waits or stream
    order."""

    def __init__(self, row_ptr, col_idx, num_parts, part_kind, local_owner, range_start, shards,
                 shard_rows, row_bytes, stride, W, fanout, max_batch, n_hot=-1, device=None,
                 cache_stride=None, nsets=None, hot_frac=None, tuning=None, split_last=None,
                 stage_apart=None):
        self.device = torch.device(device if device is not None else "cuda")
        self.N = int(row_ptr.numel() - 1)
        self.W = int(W)
        self.fanout = [int(k) for k in fanout]
        self.L = len(self.fanout)
        self.P = int(num_parts)
        self.row_bytes, self.stride = int(row_bytes), int(stride)
        self.cache_stride = int(cache_stride) if cache_stride else self.stride
        self.n_hot = int(n_hot)
        self.hot_frac = hot_frac
        self.csr = gg.make_csr(row_ptr, col_idx)
        self.part = gg.make_part(self.P, part_kind, local_owner, self.N, range_start)
        self.feat = gg.make_feat(self.row_bytes, shards, [self.stride] * self.P, shard_rows)
        self.shards = shards
        # Beside the gather, traffic decides.  The last hop samples in node
        # tiles, so that the batches share the CSR lines they fetch, when it
        # is a third hop or later (its frontiers are large) or the window's
        # batches share its frontier (a node in at least two of them, by the
        # bound): on the 2.45M-node graph at batch 4096 (4.7 batches) 0.703
        # -> 0.674 ms per window, at batch 1024 (1.2; staging on a stream of
        # its own) 0.367 -> 0.351 (the last hop's CSR fetches fall from 264
        # to about 170 MB); on the 233K-node graph (two hops, 0.9 batches)
        # batch order is faster, 0.335 -> 0.330.  Where the sampler marks
        # with atomics (sets too large for
        # LDS slices), a sparse last hop (fewer draws per batch than nodes,
        # by the bound) marks with atomics unless its byte map stays small
        # enough to live in the caches: the map's fold pass costs more than
        # the atomics it saves (batch 1024, density 0.37: 0.444 -> 0.431
        # ms); a dense one keeps the map (batch 4096, density 1.47: W = 16
        # from 0.86 to 0.77 ms).  The sequential driver, alone on the chip,
        # keeps the library's defaults.  A caller's tuning replaces this one
        # as a whole.
        shared = last_hop_sharing(self.N, self.fanout, max_batch, self.W) >= 2.0
        if tuning is None:
            dense = last_hop_density(self.N, self.fanout, max_batch) >= 1.0
            tiles = self.L >= 3 or shared
            tuning = gg.make_tuning(
                sample_order=gg.GG_SAMPLE_TILES_LAST if tiles else gg.GG_SAMPLE_BATCH_ORDER,
                **({} if dense else {"bytemap_max_mb": LOOKAHEAD_BYTEMAP_MAX_MB}))
        self.tuning = tuning
        self.geo = g = _Geometry(self.N, self.W, self.fanout, max_batch, self.P, local_owner,
                                 shard_rows, self.stride, self.cache_stride, tuning)
        dev = self.device
        on_host = any(t is not None and not t.is_cuda for t in shards)
        if nsets is None:
            nsets = 2 if on_host else 3
        if int(nsets) < 2:
            raise ValueError("the look-ahead pipeline needs at least two buffer sets")
        self.nsets = int(nsets)
        self.NSLOT = 2 * self.nsets
        # The hot set, buckets and staging read only the bit sets; the last
        # level's lists are first read by the gather.  With split_last that
        # compaction moves from the build stream to the gather stream, ahead
        # of the gather (or to the staging stream, when the hot set follows
        # the sampling there): it shortens the build chain, which pays where
        # the build is the longer chain.
        # The build grows with the sampling depth (a hop and a compaction
        # per level) and the gather does not, so by default the split is
        # taken from three hops on: on the 2.45M-node graph (three hops) the
        # window went from 0.430 to 0.419 ms; on the 233K-node graph (two
        # hops, gather-bound) it went from 0.335 to 0.350 ms, and to
        # 0.337-0.343 with the compaction on a fourth stream.
        self.split_last = (self.L >= 3) if split_last is None else bool(split_last)
        self.sets = [_Buffers(g, dev, own_cache=False, split=self.split_last)
                     for _ in range(self.nsets)]
        # One persistent cache (gg_stage_inplace): rows a window shares with
        # the previous one stay in their slot; each set keeps its remap and
        # occupancy map.
        self.cache_rows = g.inplace_rows
        self.cache = torch.empty((g.inplace_rows, self.cache_stride), dtype=torch.uint8,
                                 device=dev)
        self.stage_ws = torch.empty(gg.gg_ws_stage_inplace(g.hot_cap, g.inplace_rows, self.P),
                                    dtype=torch.uint8, device=dev)
        self.gather_ws = torch.empty(g.ws_bytes, dtype=torch.uint8, device=dev)
        self.bucket_ids = [torch.empty(g.hot_cap, dtype=torch.int32, device=dev)
                           for _ in range(self.NSLOT)]
        self.hot_count = [torch.zeros(2, dtype=torch.int64, device=dev)
                          for _ in range(self.NSLOT)]
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.build_stream, self.fetch_stream, third = _driver_streams(dev)
        # Staging gets a stream of its own when it would otherwise hold up the
        # next build: with shards in host memory (PCIe-bound), and where the
        # build is the longer chain, i.e. three or more hops whose last
        # frontier the batches barely share (2.45M-node graph, batch 1024:
        # 0.394 -> 0.374 ms per window).  Where the gather is the longer
        # chain, staging beside it only slows it (233K-node graph, two hops:
        # 0.330 -> 0.342; batch 4096: 0.677 -> 0.715).
        if stage_apart is None:
            stage_apart = on_host or (self.L >= 3 and not shared)
        self.stage_apart = bool(stage_apart)
        # With staging on a stream of its own and shards in device memory,
        # the hot set and the buckets (which read only the bit sets and write
        # the window's own buffers) follow the sampling on that stream too,
        # so that the next window's sampling starts at once; with shards in
        # host memory that stream is bound by PCIe and keeps only staging.
        self.hotset_on_stage = self.stage_apart and not on_host
        if self.stage_apart:
            self.stage_stream = self.fetch_stream
            self.gather_stream = third
        else:
            self.stage_stream = self.build_stream
            self.gather_stream = self.fetch_stream
        self.built = [torch.cuda.Event() for _ in range(self.nsets)]
        self.sampled = [torch.cuda.Event() for _ in range(self.nsets)]
        self.staged = [torch.cuda.Event() for _ in range(self.nsets)]
        self._released = [torch.cuda.Event() for _ in range(self.nsets)]
        self.gathered = list(self._released)
        self.k = 0

    def window(self, seeds, seed_off, batch0, epoch=0, rng_seed=0, out=None, events=None,
               gather_events=None, sim=None, consumer=None, consumer_events=None,
               after_caller=True):
        """Enqueues window k; returns (number of batches, buffer set).  The
        window's rows land in the set's win_out (or `out`) on the gather
        stream; wait on gathered_event(k) before reading them.  Inputs
        uploaded on the caller's stream are visible to the build stream
        (after_caller=False skips that wait, for inputs the caller has
        already synchronised: it saves the host a stream wait per window,
        which took windows of one batch of 4,096 seeds from 0.167 to 0.138
        ms; the wait also shapes how the chains interleave, and without it
        16 such batches with staging on the build stream took 0.743 ms
        instead of 0.690).
        events: optional 5 torch events recorded around the window's calls:
        before and after sampling (build stream), after the hot set and after
        the buckets (build stream, or the staging stream when
        hotset_on_stage) and after staging (staging stream).
        gather_events: optional (start, end) pair recorded around the gather
        on the gather stream; start may be None, which keeps one marker out
        of that stream's queue (the gather then starts at the later of
        events[4] and the previous window's gather end).  Without sim and
        consumer, `end` also serves as the buffer set's release, which the
        build of window k + nsets waits for: record it nowhere else before
        that build is enqueued.  sim: optional (coeffs, acc) to add the
        window to simulator totals; consumer: optional SageConsumer run on
        the gather stream after the gather (so it overlaps the next window's
        build), bracketed by the optional event pair consumer_events."""
        k, g = self.k, self.geo
        X, T = k % self.nsets, k % self.NSLOT
        cur, prev = self.sets[X], self.sets[(k - 1) % self.nsets]
        Wk = len(seed_off) - 1
        bs, ss, gs = self.build_stream, self.stage_stream, self.gather_stream
        ev = events if events is not None else [None] * 5
        if after_caller:
            bs.wait_stream(torch.cuda.current_stream(self.device))
        if k >= self.nsets:
            bs.wait_event(self.gathered[X])      # window k - nsets read this set
        s = bs.cuda_stream
        _rec(ev[0], bs)
        sargs = (self.csr, seeds, seed_off, Wk, self.fanout, self.L, rng_seed, epoch, batch0,
                 cur.wsample)
        if self.split_last:
            gg.gg_sample_window_part(*sargs, gg.GG_SAMPLE_PART_BITS, self.status, cur.ws,
                                     stream=s, tuning=self.tuning)
            self.sampled[X].record(bs)
            # the last level's lists before the gather: on the staging stream
            # when the hot set follows the sampling there (the gather waits
            # for its staging anyway), else on the gather stream
            ls = ss if self.hotset_on_stage else gs
            ls.wait_event(self.sampled[X])
            gg.gg_sample_window_part(*sargs, gg.GG_SAMPLE_PART_LAST, self.status, cur.ws,
                                     stream=ls.cuda_stream, tuning=self.tuning)
        else:
            gg.gg_sample_window(*sargs, self.status, cur.ws, stream=s, tuning=self.tuning)
        _rec(ev[1], bs)
        hs = bs
        if self.hotset_on_stage:
            # the sampling's end: the split's marker (already waited for),
            # a caller's event at that point, or the set's own
            if not self.split_last:
                sampled = ev[1] if ev[1] is not None else self.built[X]
                if sampled is self.built[X]:
                    sampled.record(bs)
                ss.wait_event(sampled)
            hs = ss
        gg.gg_build_hotset(cur.frontier_bits, Wk, self.part, self.n_hot, cur.hot_ids,
                           cur.hot_freq, g.hot_cap, self.hot_count[T], self.status, cur.ws2,
                           stream=hs.cuda_stream, hot_frac=self.hot_frac, tuning=self.tuning)
        _rec(ev[2], hs)
        gg.gg_bucket_by_owner(cur.hot_ids, self.hot_count[T], g.hot_cap, self.part,
                              self.bucket_ids[T], cur.owner_off, self.status, cur.ws2,
                              stream=hs.cuda_stream, flags=_bucket_flags(self.part))
        _rec(ev[3], hs)
        if ss is not hs:
            # a caller's event recorded at the same point serves as the
            # marker to wait on (one marker fewer in the queue)
            built = ev[3] if ev[3] is not None else self.built[X]
            if built is self.built[X]:
                built.record(bs)
            ss.wait_event(built)
        if k >= 2 and self.nsets > 2:
            # staging may reuse the slots of window k-2's rows (with two sets
            # the build already waited for that gather)
            ss.wait_event(self.gathered[(k - 2) % self.nsets])
        C = (k - self.nsets) % self.NSLOT
        clear_ids = self.bucket_ids[C] if k >= self.nsets else None
        clear_cnt = self.hot_count[C] if k >= self.nsets else None
        stage_args = (self.bucket_ids[T], cur.owner_off, g.hot_cap, self.part, self.feat,
                      self.cache, self.cache_stride, self.cache_rows, cur.slot_of, clear_ids,
                      clear_cnt, prev.slot_of if k >= 1 else None, prev.occ if k >= 1 else None,
                      cur.occ, cur.stage_stats, self.status, self.stage_ws)
        self._last_stage = stage_args
        gg.gg_stage_inplace(*stage_args, stream=ss.cuda_stream, tuning=self.tuning)
        _rec(ev[4], ss)
        if gs is not ss:
            staged = ev[4] if ev[4] is not None else self.staged[X]
            if staged is self.staged[X]:
                staged.record(ss)
            gs.wait_event(staged)
        start, end = gather_events if gather_events is not None else (None, None)
        _rec(start, gs)
        o = cur.win_out if out is None else out
        bounds = cur.frontier_off.data_ptr() + 8 * (self.L * Wk)
        gg.gg_gather_batch(cur.frontier_ids, bounds, Wk, o.shape[0], self.part, self.feat,
                           self.cache, self.cache_stride, self.cache_rows, cur.slot_of, o,
                           self.stride, cur.gather_stats.data_ptr(), self.status, self.gather_ws,
                           stream=gs.cuda_stream, flags=gg.GG_GATHER_SHARED, tuning=self.tuning)
        _rec(end, gs)
        if sim is not None:           # simulator totals, in window order on the gather stream
            gg.gg_sim_accumulate(cur.stage_stats, cur.gather_stats.data_ptr(), Wk, self.part,
                                 sim[0], sim[1], stream=gs.cuda_stream)
        if consumer is not None:      # reads the set's sampling outputs and rows
            _rec(consumer_events[0] if consumer_events else None, gs)
            consumer.forward(cur, Wk, o, self.stride, self.status, stream=gs.cuda_stream)
            _rec(consumer_events[1] if consumer_events else None, gs)
        if end is not None and sim is None and consumer is None:
            # the gather's end marks the set free: every marker in the
            # gather stream's queue delays the next gather by a few us
            self.gathered[X] = end
        else:
            self.gathered[X] = self._released[X]
            self.gathered[X].record(gs)
        self.k += 1
        return Wk, cur

    def regather(self, bufs, Wk, out=None, stream=None):
        """Launches the gather of a finished window again (same inputs, same
        output, same flags) on `stream` (default: the caller's current
        stream), e.g. to time it with the chip to itself.  The window must be
        complete, and no window after the next one staged (that staging may
        reuse the window's slots)."""
        o = bufs.win_out if out is None else out
        bounds = bufs.frontier_off.data_ptr() + 8 * (self.L * Wk)
        gg.gg_gather_batch(bufs.frontier_ids, bounds, Wk, o.shape[0], self.part, self.feat,
                           self.cache, self.cache_stride, self.cache_rows, bufs.slot_of, o,
                           self.stride, bufs.gather_stats.data_ptr(), self.status,
                           self.gather_ws, stream=stream, flags=gg.GG_GATHER_SHARED,
                           tuning=self.tuning)
        return o

    def restage(self, stream=None):
        """Launches the staging call of the last window again, with the same
        arguments, on `stream` (default: the caller's current stream), e.g.
        to time it with the chip to itself.  The window must be complete and
        no later window enqueued; the call then writes the same slots, remap
        and statistics again (its inputs, the previous window's remap and
        occupancy, are unchanged)."""
        gg.gg_stage_inplace(*self._last_stage, stream=stream, tuning=self.tuning)

    def gathered_event(self, k):
        return self.gathered[k % self.nsets]

    def synchronize(self):
        for s in (self.build_stream, self.fetch_stream, self.gather_stream):
            s.synchronize()

    def read_status(self):
        self.synchronize()
        return gg.gg_read_status(self.status)


def _rec(e, stream=None):
    if e is not None:
        e.record(stream)
