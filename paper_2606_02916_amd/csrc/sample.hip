// gg_sample_window: neighbour sampling of the W batches of one window.
//
// Every batch keeps a bit set over all node ids (N bits, in HBM).  The set
// starts as the batch's seeds; hop l samples the neighbours of every node of
// the current frontier F_l and ORs them in, so the set becomes F_{l+1} =
// F_l plus the sampled neighbours.  After each hop the sets are compacted
// into ascending id lists in two launches: a per-chunk popcount (with
// per-batch totals), then an emit pass in which every block finds its own
// place from those counts.  Deduplication therefore costs streaming passes
// over N/8 bytes per batch and hop instead of a sort of the sampled ids.
// Where a batch's set splits into few LDS-sized slices, a hop's draws are
// ORed in by a pass of their own through LDS (k_mark_slices), which also
// makes the counts; elsewhere the sampler ORs them in with atomics.
#include <limits.h>
#include <stdlib.h>

#include "gg_host.hpp"

namespace gg {
namespace {

struct SeedOff {
  int64_t off[GG_MAX_W + 1];  // entries past W hold INT64_MAX
};

struct LevelArgs {
  int32_t lv, L, W, k;
  int32_t nch;
  int32_t cnt_only;   // offsets from the chunk counts alone (no group totals)
  int64_t fcap, ncap;
  // Node-tile table of the level for the next hop's sampler (tile_runs = 0:
  // none): tstart[b * ntiles + t] = list position of batch b's first entry
  // in tile t, a tile being tile_runs runs of 256 nodes.
  int64_t* tstart;
  int64_t ntiles;
  int32_t tile_runs;
  int32_t pad_;
};

// Raw (unclamped) running ends of the window's frontier and neighbour
// lists, one slot per level, so a level reads its predecessor's while it
// writes its own.
struct LevelState {
  int64_t fend[GG_MAX_LAYERS + 1];   // frontier entries up to and including level l
  int64_t nend[GG_MAX_LAYERS + 1];   // neighbour slots up to and including level l
  int64_t nbase[GG_MAX_LAYERS + 1];  // first neighbour slot of level l
};

struct SampleArgs {
  int64_t N;
  int64_t wpb;
  int64_t fcap, ncap;
  int64_t batch0;
  int32_t W, l, k;
  uint32_t key0, key1, epoch;
  uint8_t* bytemap;   // non-null: marks go to one byte per node (bytes per batch: 32 * wpb)
  int32_t nomark;     // marks are left to k_mark_slices
};

// The last hop marks its draws with byte stores into a byte map instead of
// atomic ORs into the bit sets when the map (one byte per node and batch)
// is at most this large: a random byte store costs about a third of a
// random atomic, and folding the map into the bit sets is one streaming
// pass.  Above it (the 111M-node graph) the pass would cost more than the
// atomics it saves.  The limit is the tuning's bytemap_max_mb (default
// kByteMapMaxBytes); the workspace layout depends on it.
inline bool use_bytemap(int64_t num_nodes, int32_t W, const Tune& tune) {
  return tune.bytemap_max_bytes >= 0 &&
         (int64_t)W * gg_bits_words(num_nodes) * 32 <= tune.bytemap_max_bytes;
}

// Marks through LDS: block (s, b) of k_mark_slices holds slice s of batch
// b's set (the tuning's mark_slice_chunks chunks of 8 KB) and reads every
// slot the hop wrote for batch b, so each slot is read once per slice:
// worth it while a batch's set has few slices (at most the tuning's
// mark_slices_max).  A random OR then costs an LDS atomic instead of one
// performed at memory (about 32 bytes of memory-side traffic each, and the
// rate that bounded the sampler's last hop).  By default a block is one
// wave per SIMD (256 lanes), so that it finds room beside a running gather
// (four waves per SIMD of 74 VGPRs leave no SIMD room for a block of four
// waves each: a 1,024-lane block waited 170 us for the gather to drain);
// its lanes keep 8 loads of 16 bytes in flight instead.  Registers decide
// the size of a round: the 2.45M-node window took 0.341 ms per step with
// 32 KB rounds (68 VGPRs, mostly the slice load's), 0.346 with 64 KB (100
// VGPRs) and 0.423 with 96 KB (145 VGPRs): a block beside the gather and
// the staging stream's kernels must find its registers free.
constexpr int kMarkRoundBytes = 32768;   // slot bytes a block has in flight per round

inline int64_t mark_slices(int64_t num_nodes, const Tune& tune) {
  return cdiv(gg_bits_words(num_nodes) / kChunkWords, (int64_t)tune.mark_slice_chunks);
}

inline bool use_slices(int64_t num_nodes, const Tune& tune) {
  return tune.mark_slices_max > 0 && mark_slices(num_nodes, tune) <= tune.mark_slices_max;
}

// A mark pass runs slices x W blocks, each reading its batch's whole slot
// list, so its time hardly falls with fewer batches, where atomic marks and
// the byte map, spread over the chip, take time in proportion to the
// batches.  At about 8 G slots/s per block against 26 G atomics/s and 80 G
// byte stores/s for the chip, the pass pays from about 4 batches against
// atomics and 8 against the byte map (batch 4096 on the 2.45M-node graph:
// W = 1 0.247 ms per window through LDS, 0.190 with the map; W = 4 0.332
// against 0.300; W = 16 0.679 against 0.816).  The tuning's
// mark_min_batches fixes the minimum instead.
constexpr int kMarkMinBatchesAtomic = 4;
constexpr int kMarkMinBatchesMap = 8;

inline int32_t min_batches(bool map_instead, const Tune& tune) {
  if (tune.mark_min_batches != 0) return tune.mark_min_batches < 0 ? 1 : tune.mark_min_batches;
  return map_instead ? kMarkMinBatchesMap : kMarkMinBatchesAtomic;
}

// The last hop of a W-batch call marks through LDS slices (else into the
// byte map, if it fits, or with atomics).
inline bool last_hop_slices(int64_t num_nodes, int32_t W, const Tune& tune) {
  return use_slices(num_nodes, tune) && W >= min_batches(use_bytemap(num_nodes, W, tune), tune);
}

// Largest b in [0, 64) with off[b] <= x, for a table padded with INT64_MAX.
__device__ __forceinline__ int find_batch(const int64_t* off, int64_t x) {
  int idx = 0;
#pragma unroll
  for (int step = 32; step >= 1; step >>= 1)
    if (off[idx + step] <= x) idx += step;
  return idx;
}

// Zeroes the window's bit sets (n4 16-byte words), the byte map (m4
// 16-byte words, if any) and the per-level partial totals (nbtot).
__global__ void __launch_bounds__(kBlock) k_zero_words(uint32_t* p, int64_t n4, uint8_t* map,
                                                       int64_t m4, int32_t* btot, int32_t nbtot) {
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < nbtot;
       t += (int64_t)gridDim.x * blockDim.x)
    btot[t] = 0;
  const u32x4 z = {0u, 0u, 0u, 0u};
  u32x4* q = (u32x4*)p;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4;
       i += (int64_t)gridDim.x * blockDim.x)
    q[i] = z;
  u32x4* r = (u32x4*)map;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m4;
       i += (int64_t)gridDim.x * blockDim.x)
    r[i] = z;
}

// Bits of four bytes that are each 0 or 1: byte i gives bit i.
__device__ __forceinline__ uint32_t pack4(uint32_t v) {
  return (v & 1u) | ((v >> 7) & 2u) | ((v >> 14) & 4u) | ((v >> 21) & 8u);
}

__device__ __forceinline__ uint32_t pack16(u32x4 v) {
  return pack4(v.x) | (pack4(v.y) << 4) | (pack4(v.z) << 8) | (pack4(v.w) << 12);
}

__global__ void __launch_bounds__(kBlock) k_mark_seeds(const int32_t* seeds, SeedOff so, int32_t W,
                                                       uint32_t* bits, int64_t wpb, int64_t N,
                                                       int32_t* status) {
  const int64_t total = so.off[W];
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int b = find_batch(so.off, i);
    const int32_t u = seeds[i];
    if (u < 0 || (int64_t)u >= N) {
      set_status(status, GG_DEV_BAD_ID);
      continue;
    }
    atomicOr(bits + (int64_t)b * wpb + (u >> 5), 1u << (u & 31));
  }
}

// Level 0 in one launch: block (c, b) assembles chunk c (kChunkWords
// words) of batch b's bit set in LDS from the batch's seeds and stores it
// whole, so the bit sets need no clearing pass and the seeds no global
// atomics.  It also clears its part of the byte map (if any) and, spread
// over the grid, the group totals.  Every block reads its batch's seeds, so
// batches of at most kSeedBitsMaxBatch seeds take this path.
constexpr int64_t kSeedBitsMaxBatch = 16384;
// Most chunks (W times the chunks of one bit set) for which a level-0 emit
// block sums every chunk count before its own: 608 for 16 batches over
// 2.45M nodes; 27K for the 111M-node graph keeps the counting pass.
constexpr int64_t kCntOnlyMaxChunks = 4096;

__global__ void __launch_bounds__(kBlock) k_seed_bits(const int32_t* seeds, SeedOff so,
                                                      uint32_t* bits, int64_t wpb, int64_t N,
                                                      uint8_t* map, int32_t* btot, int32_t nbtot,
                                                      int32_t* cnt, int32_t* status) {
  __shared__ uint32_t w[kChunkWords];
  __shared__ int32_t s_pop[kBlock / kWave];
  const int c = blockIdx.x, b = blockIdx.y;
  const int64_t flat = ((int64_t)b * gridDim.x + c) * blockDim.x + threadIdx.x;
  const int64_t nthreads = (int64_t)gridDim.x * gridDim.y * blockDim.x;
  for (int64_t t = flat; t < nbtot; t += nthreads) btot[t] = 0;
  for (int i = threadIdx.x; i < kChunkWords; i += blockDim.x) w[i] = 0u;
  __syncthreads();
  const int64_t lo = (int64_t)c * kChunkWords * 32, hi = lo + (int64_t)kChunkWords * 32;
  int32_t st = 0;
  for (int64_t i = so.off[b] + threadIdx.x; i < so.off[b + 1]; i += blockDim.x) {
    const int32_t u = seeds[i];
    if (u < 0 || (int64_t)u >= N) {
      if (c == 0) st |= GG_DEV_BAD_ID;
    } else if ((int64_t)u >= lo && (int64_t)u < hi) {
      atomicOr(&w[(u - lo) >> 5], 1u << (u & 31));
    }
  }
  __syncthreads();
  u32x4* dst = (u32x4*)(bits + (int64_t)b * wpb + (int64_t)c * kChunkWords);
  int32_t pop = 0;
  for (int i = threadIdx.x; i < kChunkWords / 4; i += blockDim.x) {
    const u32x4 v = {w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]};
    dst[i] = v;
    pop += __popc(v.x) + __popc(v.y) + __popc(v.z) + __popc(v.w);
  }
  if (cnt) {   // the chunk's count, so that level 0 needs no counting pass
    pop = wave_sum(pop);
    if (lane_id() == 0) s_pop[threadIdx.x / kWave] = pop;
    __syncthreads();
    if (threadIdx.x == 0) {
      int32_t n = 0;
      for (int q = 0; q < kBlock / kWave; ++q) n += s_pop[q];
      cnt[(int64_t)b * gridDim.x + c] = n;
    }
  }
  if (map) {
    u32x4* m = (u32x4*)(map + ((int64_t)b * wpb + (int64_t)c * kChunkWords) * 32);
    const u32x4 z = {0u, 0u, 0u, 0u};
    for (int i = threadIdx.x; i < kChunkWords * 2; i += blockDim.x) m[i] = z;
  }
  if (st) set_status(status, st);
}

// Popcount of one chunk (kChunkWords words) of one batch's bit set.  The
// chunk's count goes to cnt and is added to its group's partial total (a
// group is kGroupChunks consecutive chunks of one batch), spread over
// kTotLanes words so that at most eight blocks add to one word (one total
// per batch had 212 blocks contending for a word on the 111M-node graph).
// An emit block then finds its place from the group totals of the batches
// before its own, those of its batch before its group, and the counts of
// its group's chunks before it: a few KB that stay in the caches.  With a
// byte map (after a hop that marked bytes) the chunk's bytes are first
// folded into its bit-set words.
constexpr int kTotLanes = 8;
constexpr int kGroupChunks = 64;

struct Totals {
  int32_t* gtot;   // [W][ngroups][kTotLanes]
  int32_t ngroups;
};

__global__ void __launch_bounds__(kBlock) k_bits_count(uint32_t* bits, int64_t wpb,
                                                       const uint8_t* map, int32_t* cnt,
                                                       Totals tt) {
  __shared__ int32_t lds[kBlock / kWave];
  const int c = blockIdx.x, b = blockIdx.y, nch = gridDim.x;
  const int64_t w0 = (int64_t)c * kChunkWords + threadIdx.x * kWordsPerThread;
  u32x4* p = (u32x4*)(bits + (int64_t)b * wpb + w0);
  u32x4 x = p[0], y = p[1];
  if (map) {
    const u32x4* q = (const u32x4*)(map + ((int64_t)b * wpb + w0) * 32);
    u32x4 m[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) m[j] = q[j];
    x.x |= pack16(m[0]) | (pack16(m[1]) << 16);
    x.y |= pack16(m[2]) | (pack16(m[3]) << 16);
    x.z |= pack16(m[4]) | (pack16(m[5]) << 16);
    x.w |= pack16(m[6]) | (pack16(m[7]) << 16);
    y.x |= pack16(m[8]) | (pack16(m[9]) << 16);
    y.y |= pack16(m[10]) | (pack16(m[11]) << 16);
    y.z |= pack16(m[12]) | (pack16(m[13]) << 16);
    y.w |= pack16(m[14]) | (pack16(m[15]) << 16);
    p[0] = x;
    p[1] = y;
  }
  int s = __popc(x.x) + __popc(x.y) + __popc(x.z) + __popc(x.w) + __popc(y.x) + __popc(y.y) +
          __popc(y.z) + __popc(y.w);
  s = wave_sum(s);
  if (lane_id() == 0) lds[threadIdx.x / kWave] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const int32_t n = lds[0] + lds[1] + lds[2] + lds[3];
    cnt[(int64_t)b * nch + c] = n;
    if (n)
      atomicAdd(tt.gtot + ((int64_t)b * tt.ngroups + c / kGroupChunks) * kTotLanes +
                    (c & (kTotLanes - 1)),
                n);
  }
}

struct MarkArgs {
  int64_t N, wpb, ncap;
  int32_t W, l, k, nch;
  int32_t vec;      // the slots are 16-byte aligned
  int32_t schunks;  // chunks per slice (the block's dynamic LDS: schunks * 8 KB)
  int32_t nslices;  // slices per batch
  int32_t pad_;
};

// Workgroups go to the chip's 8 XCDs (each with its own L2) round robin by
// block index.  The grid is numbered so that every slice of a batch lands
// on one XCD: the batch's slot list then comes from memory once and the
// other slices' blocks read it from that L2.  Block i: XCD i mod 8, batch
// (i / 8 / nslices) * 8 + i mod 8, slice (i / 8) mod nslices; a block past
// the last batch has no work.
constexpr int kXcds = 8;

// One round of a mark block's slot loads: lane t reads the 16-byte groups
// at p + u * 4 * kMarkBlock (p at the lane's first group), all in flight at
// once, then marks their slots.  The lane's groups end at `mine` slots past
// p (a round's last lane may have fewer); a load past that end reads the
// lane's last group again (in bounds, no branch) and its slots are not
// marked, nor are the first `head` slots, which precede the batch's list.
template <int kMarkBlock, typename F>
__device__ __forceinline__ void mark_round(const int32_t* p, int32_t mine, int32_t head,
                                           F& mark) {
  constexpr int kMarkLoads = kMarkRoundBytes / 16 / kMarkBlock;
  constexpr int kStep = 4 * kMarkBlock;
  u32x4 t[kMarkLoads];
#pragma unroll
  for (int u = 0; u < kMarkLoads; ++u)
    t[u] = *(const u32x4*)(p + (u * kStep < mine ? u * kStep : mine - 4));
#pragma unroll
  for (int u = 0; u < kMarkLoads; ++u) {
    const bool ok = u * kStep < mine;
    mark((int32_t)t[u].x, ok && u * kStep + 0 >= head);
    mark((int32_t)t[u].y, ok && u * kStep + 1 >= head);
    mark((int32_t)t[u].z, ok && u * kStep + 2 >= head);
    mark((int32_t)t[u].w, ok && u * kStep + 3 >= head);
  }
}

// The marks of hop l, with level l+1's counts (as k_bits_count makes them):
// block (s, b) loads slice s of batch b's set (F_l's bits) into LDS, ORs in
// every id in batch b's slots of hop l that falls in the slice, writes the
// slice back and counts its chunks.  Only the slots of complete entries are
// read: an entry that would pass the slot capacity wrote none of its slots,
// and the end of the last complete one bounds what was written.
template <int kMarkBlock>
__device__ __forceinline__ void mark_slices_body(uint32_t* bits, const int32_t* nbr,
                                                 const int64_t* nbr_off, const LevelState* ls,
                                                 int32_t* cnt, Totals tt, MarkArgs a) {
  extern __shared__ uint32_t sl[];
  const int xcd = blockIdx.x % kXcds, j = blockIdx.x / kXcds;
  const int s = j % a.nslices, b = j / a.nslices * kXcds + xcd;
  if (b >= a.W) return;
  const int c0 = s * a.schunks;
  const int nc = min(a.schunks, a.nch - c0);
  const int nw = nc * kChunkWords;
  uint32_t* brow = bits + (int64_t)b * a.wpb + (int64_t)c0 * kChunkWords;
  int64_t lo = nbr_off[(int64_t)a.l * a.W + b], hi = nbr_off[(int64_t)a.l * a.W + b + 1];
  const int64_t nbase = ls->nbase[a.l];
  {
    // the slice (at most 8 chunks) in one round of loads: beside a gather
    // that saturates HBM a round trip takes several microseconds
    constexpr int kSliceLoads = 8 * kChunkWords / 4 / kMarkBlock;
    u32x4 t[kSliceLoads];
#pragma unroll
    for (int u = 0; u < kSliceLoads; ++u) {
      const int i = u * kMarkBlock + threadIdx.x;
      if (i < nw / 4) t[u] = ((const u32x4*)brow)[i];
    }
#pragma unroll
    for (int u = 0; u < kSliceLoads; ++u) {
      const int i = u * kMarkBlock + threadIdx.x;
      if (i < nw / 4) ((u32x4*)sl)[i] = t[u];
    }
  }
  if (nbase < a.ncap) {
    const int64_t lim = nbase + (a.ncap - nbase) / a.k * a.k;
    hi = hi < lim ? hi : lim;
  }
  __syncthreads();
  const uint32_t node_lo = (uint32_t)c0 * (uint32_t)(kChunkWords * 32);
  const uint32_t span = (uint32_t)nw * 32u;
  // Branch-free: every lane ORs, a value outside the slice (or not a slot
  // of the batch) ORs 0 into a word of its own past the slice.  A branch per
  // value would cost more than the extra LDS operations: a wave has few
  // neighbours on its SIMD to hide the branch latency behind.
  const uint32_t dummy = (uint32_t)nw + (uint32_t)lane_id();
  auto mark = [&](int32_t v, bool ok) {
    const uint32_t x = (uint32_t)v - node_lo;   // wraps above span for v < node_lo
    const bool in = ok && x < span && (uint32_t)v < (uint32_t)a.N;
    atomicOr(&sl[in ? x >> 5 : dummy], in ? 1u << (x & 31) : 0u);
  };

  // Rounds of up to kMarkRoundBytes of slots in whole 16-byte groups, from
  // the boundary at or below lo to the one at or below hi, all of a round's
  // loads in flight at once (a loop of one load per lane and step would pay
  // a memory round trip per step); then the at most three slots after the
  // last group.
  constexpr int kRound = kMarkRoundBytes / 4;   // slots
  if (a.vec) {
    const int64_t a0 = lo & ~(int64_t)3, hv = hi & ~(int64_t)3;
    // slots of this lane's first group before lo (lo - a0 < 4): 0..3
    const int64_t h = lo - a0 - 4 * (int64_t)threadIdx.x;
    int32_t head = h > 0 ? (int32_t)h : 0;
    for (int64_t base = a0; base < hv; base += kRound, head = 0) {
      const int64_t rem = hv - base;
      const int32_t r = rem < kRound ? (int32_t)rem : kRound;   // a multiple of 4
      const int32_t mine = r - 4 * (int32_t)threadIdx.x;       // <= 0: no group this round
      if (mine > 0) mark_round<kMarkBlock>(nbr + base + 4 * threadIdx.x, mine, head, mark);
    }
    const int64_t q = (hv > lo ? hv : lo) + threadIdx.x;
    if (q < hi) mark(nbr[q], true);
  } else {
    for (int64_t q = lo + threadIdx.x; q < hi; q += kMarkBlock) mark(nbr[q], true);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nw / 4; i += kMarkBlock) ((u32x4*)brow)[i] = ((const u32x4*)sl)[i];
  const int lane = lane_id();
  for (int cc = threadIdx.x / kWave; cc < nc; cc += kMarkBlock / kWave) {
    const u32x4* cw = (const u32x4*)(sl + cc * kChunkWords);
    int n = 0;
    for (int j = lane; j < kChunkWords / 4; j += kWave) {
      const u32x4 w = cw[j];
      n += __popc(w.x) + __popc(w.y) + __popc(w.z) + __popc(w.w);
    }
    n = wave_sum(n);
    if (lane == 0) {
      const int c = c0 + cc;
      cnt[(int64_t)b * a.nch + c] = n;
      if (n)
        atomicAdd(tt.gtot + ((int64_t)b * tt.ngroups + c / kGroupChunks) * kTotLanes +
                      (c & (kTotLanes - 1)),
                  n);
    }
  }
}

#define GG_MARK_ARGS                                                                        \
  uint32_t *bits, const int32_t *nbr, const int64_t *nbr_off, const LevelState *ls, int32_t *cnt, \
      Totals tt, MarkArgs a
__global__ void __launch_bounds__(256) k_mark_slices_256(GG_MARK_ARGS) {
  mark_slices_body<256>(bits, nbr, nbr_off, ls, cnt, tt, a);
}
__global__ void __launch_bounds__(1024) k_mark_slices_1024(GG_MARK_ARGS) {
  mark_slices_body<1024>(bits, nbr, nbr_off, ls, cnt, tt, a);
}
#undef GG_MARK_ARGS

// Sums of three values over the block.
__device__ __forceinline__ void block_sum3(int64_t (&v)[3], int64_t (*lds)[3]) {
  const int w = threadIdx.x / kWave;
#pragma unroll
  for (int j = 0; j < 3; ++j) v[j] = wave_sum(v[j]);
  if (lane_id() == 0)
#pragma unroll
    for (int j = 0; j < 3; ++j) lds[w][j] = v[j];
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    int64_t t = 0;
    for (int q = 0; q < kBlock / kWave; ++q) t += lds[q][j];
    v[j] = t;
  }
  __syncthreads();
}

// Writes the ids of one chunk of one batch's bit set, ascending, at its
// place in the level's list.  The place comes from the counts of the
// previous launch: the totals of the batches before b plus the counts of
// the chunks before c, summed by the block itself (no separate scan
// launch).  Block (0, b) writes batch b's frontier and neighbour offsets;
// block (0, 0) also the level's ends and capacity checks.
__global__ void __launch_bounds__(kBlock) k_bits_emit(const uint32_t* bits, int64_t wpb,
                                                      const int32_t* cnt, Totals tt,
                                                      int32_t* ids, int64_t* frontier_off,
                                                      int64_t* nbr_off, LevelState* ls,
                                                      int64_t* need, int32_t* status,
                                                      LevelArgs a) {
  __shared__ int64_t lds3[kBlock / kWave][3];
  __shared__ int32_t lds[kBlock / kWave];
  __shared__ int64_t s_off;
  const int c = blockIdx.x, b = blockIdx.y, nch = gridDim.x;
  const int64_t w0 = (int64_t)c * kChunkWords + threadIdx.x * kWordsPerThread;
  const u32x4* p = (const u32x4*)(bits + (int64_t)b * wpb + w0);
  const u32x4 x = p[0], y = p[1];      // in flight while the offsets are summed
  const int64_t raw_base = a.lv == 0 ? 0 : ls->fend[a.lv - 1];
  const int64_t raw_nbase = a.lv == 0 ? 0 : ls->nend[a.lv - 1];
  int64_t v[3] = {0, 0, 0};  // batches before b, all batches (block (0, 0)), chunks of b before c
  if (a.cnt_only) {
    // a window of few chunks: every block sums the chunk counts before it
    const int64_t mine = (int64_t)b * nch;
    const int64_t upto = (b == 0 && c == 0) ? (int64_t)a.W * nch : mine + c;
    for (int64_t t = threadIdx.x; t < upto; t += kBlock) {
      const int64_t x = cnt[t];
      v[1] += x;
      if (t < mine) v[0] += x;
      else if (t < mine + c) v[2] += x;
    }
  } else {
    const int64_t per_batch = (int64_t)tt.ngroups * kTotLanes;
    const int64_t upto = (b == 0 && c == 0) ? a.W * per_batch : b * per_batch;
    for (int64_t t = threadIdx.x; t < upto; t += kBlock) {
      const int64_t x = tt.gtot[t];
      v[1] += x;
      if (t < b * per_batch) v[0] += x;
    }
    const int g = c / kGroupChunks;
    const int32_t* gb = tt.gtot + b * per_batch;
    for (int t = threadIdx.x; t < g * kTotLanes; t += kBlock) v[2] += gb[t];
    for (int t = g * kGroupChunks + threadIdx.x; t < c; t += kBlock)
      v[2] += cnt[(int64_t)b * nch + t];
  }
  block_sum3(v, lds3);
  const int64_t cb = raw_base < a.fcap ? raw_base : a.fcap;
  if (threadIdx.x == 0) {
    s_off = raw_base + v[0] + v[2];
    if (c == 0) {
      int64_t fo = raw_base + v[0];
      fo = fo < a.fcap ? fo : a.fcap;
      frontier_off[(int64_t)a.lv * a.W + b] = fo;
      if (a.lv < a.L) {
        const int64_t nv = raw_nbase + (fo - cb) * a.k;
        nbr_off[(int64_t)a.lv * a.W + b] = nv < a.ncap ? nv : a.ncap;
      }
      if (b == 0) {
        const int64_t raw_end = raw_base + v[1];
        const int64_t ce = raw_end < a.fcap ? raw_end : a.fcap;
        frontier_off[(int64_t)(a.lv + 1) * a.W] = ce;
        ls->fend[a.lv] = raw_end;
        need[0] = raw_end;
        int32_t st = raw_end > a.fcap ? GG_DEV_CAPACITY : 0;
        if (a.lv < a.L) {
          const int64_t nend = raw_nbase + (ce - cb) * a.k;
          nbr_off[(int64_t)(a.lv + 1) * a.W] = nend < a.ncap ? nend : a.ncap;
          ls->nbase[a.lv] = raw_nbase;
          ls->nend[a.lv] = nend;
          need[1] = nend;
          if (nend > a.ncap) st |= GG_DEV_CAPACITY;
        }
        if (st) set_status(status, st);
      }
    }
  }
  __syncthreads();
  const uint32_t w[8] = {x.x, x.y, x.z, x.w, y.x, y.y, y.z, y.w};
  int n = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) n += __popc(w[j]);
  int32_t tot;
  int64_t pos = s_off + block_excl_scan<kBlock>(n, lds, &tot);
  if (a.tile_runs) {
    // this thread's run of 8 words starts a tile every tile_runs runs
    const int64_t run = (int64_t)c * kBlock + threadIdx.x;
    if (run % a.tile_runs == 0) a.tstart[(int64_t)b * a.ntiles + run / a.tile_runs] = pos;
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    for (uint32_t m = w[j]; m; m &= m - 1u) {
      if (pos < a.fcap) ids[pos] = (int32_t)((w0 + j) * 32 + (__ffs(m) - 1));
      ++pos;
    }
  }
}

template <int KMAX>
__device__ __forceinline__ void floyd_positions(uint32_t u, uint32_t bglob, const SampleArgs& a,
                                                uint32_t d, uint32_t* pos) {
  const uint32_t k = (uint32_t)a.k;
  uint4 blk = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    if ((uint32_t)i < k) {
      if ((i & 3) == 0)
        blk = philox4x32_10(make_uint4(u, bglob, a.epoch, ((uint32_t)a.l << 16) | (uint32_t)(i >> 2)),
                            a.key0, a.key1);
      const uint32_t r = (i & 3) == 0 ? blk.x : (i & 3) == 1 ? blk.y : (i & 3) == 2 ? blk.z : blk.w;
      const uint32_t j = d - k + (uint32_t)i;
      const uint32_t t = (uint32_t)(((uint64_t)r * ((uint64_t)j + 1u)) >> 32);
      bool dup = false;
#pragma unroll
      for (int q = 0; q < i; ++q) dup |= (pos[q] == t);
      pos[i] = dup ? j : t;
    } else {
      pos[i] = 0xFFFFFFFFu;
    }
  }
  // Bitonic sorting network, ascending.
#pragma unroll
  for (int size = 2; size <= KMAX; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
#pragma unroll
      for (int i = 0; i < KMAX; ++i) {
        const int j = i ^ stride;
        if (j > i) {
          const bool up = (i & size) == 0;
          const uint32_t x = pos[i], y = pos[j];
          const bool sw = up ? (x > y) : (x < y);
          pos[i] = sw ? y : x;
          pos[j] = sw ? x : y;
        }
      }
    }
  }
}

// Samples frontier entry gi of level l (batch b): writes its k neighbour
// slots and, unless a.nomark, sets the sampled neighbours' bits in batch
// b's set.  All neighbour loads are issued before any store or atomic.  An
// entry whose slots would pass the capacity writes neither slots nor bits,
// so the ids in the written slots are exactly the marks.
template <typename RowT, int KMAX>
__device__ __forceinline__ void sample_one(const RowT* row_ptr, const int32_t* col_idx,
                                           const int32_t* fids, int64_t gi, int b, int64_t begin,
                                           int64_t nbase, int32_t* nbr, uint32_t* bits,
                                           const SampleArgs& a, int32_t& st) {
  const int32_t k = a.k;
  const int32_t u = fids[gi];
  const int64_t obase = nbase + (gi - begin) * k;
  if (obase + k > a.ncap) {
    st |= GG_DEV_CAPACITY;
    return;
  }
  int32_t* out = nbr + obase;
  uint32_t* brow = bits + (int64_t)b * a.wpb;
  const int64_t beg = (int64_t)row_ptr[u];
  const int64_t d = (int64_t)row_ptr[u + 1] - beg;
  uint32_t pos[KMAX];
  int32_t cnt;
  if (d <= k) {
#pragma unroll
    for (int i = 0; i < KMAX; ++i) pos[i] = (uint32_t)i;
    cnt = (int32_t)d;
  } else if (d > 0xFFFFFFFFLL) {
    st |= GG_DEV_BAD_DEGREE;
    cnt = 0;
  } else {
    floyd_positions<KMAX>((uint32_t)u, (uint32_t)(a.batch0 + b), a, (uint32_t)d, pos);
    cnt = k;
  }
  int32_t v[KMAX];
#pragma unroll
  for (int i = 0; i < KMAX; ++i) v[i] = (i < cnt) ? col_idx[beg + pos[i]] : -1;
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    if (i < k && i < cnt && (v[i] < 0 || (int64_t)v[i] >= a.N)) {
      st |= GG_DEV_BAD_ID;
      v[i] = -1;
    }
  }
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    if (i < k) {
      const int32_t x = v[i];
      if (x >= 0 && !a.nomark) {
        if (a.bytemap)
          a.bytemap[(int64_t)b * a.wpb * 32 + x] = 1;
        else
          atomicOr(brow + (x >> 5), 1u << (x & 31));
      }
      out[i] = (i < cnt) ? x : -1;
    }
  }
}

// One lane per frontier node of level l (all batches of the window).
template <typename RowT, int KMAX>
__global__ void __launch_bounds__(kBlock) k_sample(const RowT* row_ptr, const int32_t* col_idx,
                                                   const int32_t* fids, const int64_t* frontier_off,
                                                   const LevelState* ls, int32_t* nbr, uint32_t* bits,
                                                   int32_t* status, SampleArgs a) {
  __shared__ int64_t so[GG_MAX_W + 1];
  __shared__ int64_t s_nbase;
  for (int t = threadIdx.x; t <= GG_MAX_W; t += blockDim.x)
    so[t] = t <= a.W ? frontier_off[(int64_t)a.l * a.W + t] : INT64_MAX;
  if (threadIdx.x == 0) s_nbase = ls->nbase[a.l];
  __syncthreads();
  const int64_t begin = so[0], end = so[a.W];
  const int64_t nbase = s_nbase;
  int32_t st = 0;
  for (int64_t gi = begin + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; gi < end;
       gi += (int64_t)gridDim.x * blockDim.x)
    sample_one<RowT, KMAX>(row_ptr, col_idx, fids, gi, find_batch(so, gi), begin, nbase, nbr, bits,
                           a, st);
  if (st) set_status(status, st);
}

// Node-tile order: a wavefront takes one tile of consecutive node ids
// (tile_runs runs of 256) and samples the entries of that tile in every
// batch of the window, batch by batch.  A node that several batches reach
// is then sampled by the same wavefront, whose CSR lines (row_ptr and the
// node's neighbour row) the caches serve after the first batch fetches
// them; in batch order the batches' copies of a node land on different
// CUs and XCDs, and every batch fetches the lines again.  Each entry is
// sampled exactly once, by the same code, so results do not depend on the
// order.  Lane b (b < W) finds batch b's entries of the tile from the
// level's tile table; pair j of the tile belongs to the first batch whose
// running count exceeds j, found by a binary search over the lanes.  A
// wavefront's tile is g consecutive tiles of the table (ntab of them), g a
// power of two chosen from the level's entry count so that a tile holds
// about a wavefront of entries (at most gmax); with fixed = 1, g = 1.
// Too few entries per wavefront would launch many thinly filled waves,
// which beside another kernel's resident blocks wait for CU slots in
// several rounds.
template <typename RowT, int KMAX>
__global__ void __launch_bounds__(kBlock) k_sample_tiles(const RowT* row_ptr,
                                                         const int32_t* col_idx,
                                                         const int32_t* fids,
                                                         const int64_t* frontier_off,
                                                         const LevelState* ls,
                                                         const int64_t* tstart, int64_t ntab,
                                                         int32_t gmax, int32_t* nbr,
                                                         uint32_t* bits, int32_t* status,
                                                         SampleArgs a) {
  __shared__ int64_t so[GG_MAX_W + 1];
  __shared__ int64_t s_nbase;
  for (int t = threadIdx.x; t <= GG_MAX_W; t += blockDim.x)
    so[t] = t <= a.W ? frontier_off[(int64_t)a.l * a.W + t] : INT64_MAX;
  if (threadIdx.x == 0) s_nbase = ls->nbase[a.l];
  __syncthreads();
  const int64_t begin = so[0];
  const int64_t nbase = s_nbase;
  const int lane = lane_id();
  // table tiles per wavefront tile: about kWave entries each on average
  const int64_t entries = so[a.W] - begin;
  int64_t g = 1;
  while (g < gmax && (g * 2) * entries <= ntab * kWave) g *= 2;
  const int64_t ntiles = (ntab + g - 1) / g;
  int32_t st = 0;
  for (int64_t t = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; t < ntiles;
       t += (int64_t)gridDim.x * (kBlock / kWave)) {
    // batch `lane`'s entries of tile t, clamped to its (clamped) segment
    int64_t lo = 0, n = 0;
    if (lane < a.W) {
      const int64_t* tb = tstart + (int64_t)lane * ntab;
      const int64_t s0 = so[lane], s1 = so[lane + 1];
      lo = tb[t * g];
      int64_t hi = (t + 1) * g < ntab ? tb[(t + 1) * g] : s1;
      lo = lo < s0 ? s0 : (lo > s1 ? s1 : lo);
      hi = hi > s1 ? s1 : (hi < lo ? lo : hi);
      n = hi - lo;
    }
    const int64_t inc = wave_incl_scan(n);
    const int64_t total = __shfl(inc, a.W - 1, kWave);
    for (int64_t j0 = 0; j0 < total; j0 += kWave) {
      const int64_t j = j0 + lane;
      // b = number of batches whose running count is at most j
      int b = 0;
#pragma unroll
      for (int step = kWave / 2; step >= 1; step >>= 1) {
        const int probe = b + step - 1;
        const int64_t v = __shfl(inc, probe < a.W ? probe : a.W - 1, kWave);
        if (probe < a.W && v <= j) b += step;
      }
      const int bb = b < a.W ? b : a.W - 1;
      const int64_t before = __shfl(inc - n, bb, kWave);
      const int64_t gi = __shfl(lo, bb, kWave) + (j - before);
      if (j < total)
        sample_one<RowT, KMAX>(row_ptr, col_idx, fids, gi, bb, begin, nbase, nbr, bits, a, st);
    }
  }
  if (st) set_status(status, st);
}

struct SampleWs {
  int32_t* cnt;       // per (batch, chunk) counts of the current level
  int32_t* tot;       // per level: group totals; zeroed by k_seed_bits (or k_zero_words)
  int32_t ngroups;    // groups of kGroupChunks chunks per batch
  int64_t tot_level;  // entries of tot per level
  LevelState* lvl;
  uint8_t* map;       // the last hop's byte map (32 * wpb bytes per batch), or null
  int64_t* tstart;    // node-tile table of one level: W * (wpb / 8) entries at most
};

size_t sample_ws_layout(int64_t num_nodes, int32_t W, const Tune& tune, char* base,
                        SampleWs* out) {
  const int64_t nch = gg_bits_words(num_nodes) / kChunkWords;
  Carve cv{base, 0, ~(size_t)0};
  SampleWs s;
  s.cnt = cv.take<int32_t>((size_t)(W * nch));
  s.ngroups = (int32_t)std::max<int64_t>(1, cdiv(nch, kGroupChunks));
  s.tot_level = (int64_t)W * kTotLanes * s.ngroups;
  s.tot = cv.take<int32_t>((size_t)(GG_MAX_LAYERS + 1) * s.tot_level);
  s.lvl = cv.take<LevelState>(1);
  s.map = use_bytemap(num_nodes, W, tune) && !last_hop_slices(num_nodes, W, tune)
              ? cv.take<uint8_t>((size_t)W * (size_t)gg_bits_words(num_nodes) * 32)
              : nullptr;
  s.tstart = tune.sample_order != GG_SAMPLE_BATCH_ORDER
                 ? cv.take<int64_t>((size_t)W * (size_t)(gg_bits_words(num_nodes) / kWordsPerThread))
                 : nullptr;
  if (out) *out = s;
  return align_up(cv.used, 256);
}

// Runs of 256 nodes per tile of the table a level's emit writes for the
// next hop's sampler (level lv of at most `bound` entries over nruns runs),
// or 0 for batch order.  Node tiles cover the last hop only, or every hop
// (the tuning's sample_order).  Sized per hop, a table tile is a power of
// two (at most 64) that holds at most a wavefront of entries by the bound,
// and the sampler joins table tiles by the level's actual count (deeper
// levels reach far fewer entries than their bound, as batches overlap);
// the tuning's sample_tile_runs fixes the size instead.  Measured beside
// the look-ahead's gather on the 2.45M-node graph, last-hop tiles cut that
// hop's fetched bytes by a third; tiles at the first two hops, whose
// frontiers the batches share little, made the window slower.
int32_t tile_runs_for(const Tune& tune, int lv, int L, int64_t nruns, int64_t bound) {
  if (tune.sample_order == GG_SAMPLE_BATCH_ORDER) return 0;
  if (tune.sample_order == GG_SAMPLE_TILES_LAST && lv != L - 1) return 0;
  if (tune.sample_tile_runs > 0) return tune.sample_tile_runs;
  int64_t g = 1;
  while (g < 64 && (g * 2) * std::max<int64_t>(bound, 1) <= nruns * kWave) g *= 2;
  return (int32_t)g;
}

template <typename RowT>
int launch_sample(const gg_csr_t* csr, const gg_wsample_t* out, const SampleWs& ws, int32_t* status,
                  const SampleArgs& a, int64_t bound, int64_t ntab, int32_t gmax,
                  hipStream_t stream) {
  const RowT* rp = (const RowT*)csr->row_ptr;
  if (ntab > 0) {
    // one wavefront per node tile, four per block; the tiles are joined
    // table tiles, so there are at most ntab
    const int grid = (int)std::min<int64_t>(cdiv(ntab, kBlock / kWave), 8192);
    if (a.k <= 8)
      hipLaunchKernelGGL((k_sample_tiles<RowT, 8>), dim3(grid), dim3(kBlock), 0, stream, rp,
                         csr->col_idx, out->frontier_ids, out->frontier_off, ws.lvl, ws.tstart,
                         ntab, gmax, out->nbr_ids, out->frontier_bits, status, a);
    else if (a.k <= 16)
      hipLaunchKernelGGL((k_sample_tiles<RowT, 16>), dim3(grid), dim3(kBlock), 0, stream, rp,
                         csr->col_idx, out->frontier_ids, out->frontier_off, ws.lvl, ws.tstart,
                         ntab, gmax, out->nbr_ids, out->frontier_bits, status, a);
    else
      hipLaunchKernelGGL((k_sample_tiles<RowT, 32>), dim3(grid), dim3(kBlock), 0, stream, rp,
                         csr->col_idx, out->frontier_ids, out->frontier_off, ws.lvl, ws.tstart,
                         ntab, gmax, out->nbr_ids, out->frontier_bits, status, a);
    GG_LAUNCH_CHECK("k_sample_tiles");
    return GG_OK;
  }
  const int grid = (int)std::min<int64_t>(std::max<int64_t>(cdiv(bound, kBlock), 1), 8192);
  if (a.k <= 8)
    hipLaunchKernelGGL((k_sample<RowT, 8>), dim3(grid), dim3(kBlock), 0, stream, rp, csr->col_idx,
                       out->frontier_ids, out->frontier_off, ws.lvl, out->nbr_ids,
                       out->frontier_bits, status, a);
  else if (a.k <= 16)
    hipLaunchKernelGGL((k_sample<RowT, 16>), dim3(grid), dim3(kBlock), 0, stream, rp,
                       csr->col_idx, out->frontier_ids, out->frontier_off, ws.lvl, out->nbr_ids,
                       out->frontier_bits, status, a);
  else
    hipLaunchKernelGGL((k_sample<RowT, 32>), dim3(grid), dim3(kBlock), 0, stream, rp,
                       csr->col_idx, out->frontier_ids, out->frontier_off, ws.lvl, out->nbr_ids,
                       out->frontier_bits, status, a);
  GG_LAUNCH_CHECK("k_sample");
  return GG_OK;
}

}  // namespace
}  // namespace gg

using namespace gg;

extern "C" size_t gg_ws_sample(int64_t num_nodes, int32_t W, const gg_tuning_t* tuning) {
  Tune tune;
  if (resolve_tuning(tuning, &tune) != GG_OK) return 0;
  // A call with fewer batches may take the byte map where W batches do not
  // (the map grows with the batches, and LDS marks need enough of them),
  // so the size is the largest over every call of at most W batches.
  size_t need = sample_ws_layout(num_nodes, W, tune, nullptr, nullptr);
  for (int32_t w = 1; w < std::min<int32_t>(W, GG_MAX_W); ++w)
    need = std::max(need, sample_ws_layout(num_nodes, w, tune, nullptr, nullptr));
  return need;
}

namespace gg {
namespace {

// The sampling of one window, or a part of it: GG_SAMPLE_PART_BITS is everything
// up to the last level's compaction (with a byte map, its fold into the bit
// sets included), GG_SAMPLE_PART_LAST that compaction (the count, unless the
// fold already made it, and the emit of F_L).
int sample_window_impl(const gg_csr_t* csr, const int32_t* seeds_d, const int64_t* seed_off_h,
                       int32_t W, const int32_t* fanout_h, int32_t L, uint64_t rng_seed,
                       int32_t epoch, int64_t batch0, const gg_wsample_t* out,
                       const gg_tuning_t* tuning, int32_t* status_d, void* ws, size_t ws_bytes,
                       int32_t part, hipStream_t stream) {
  GG_REQUIRE(csr && out && seed_off_h && fanout_h && status_d, "NULL argument");
  const bool do_bits = (part & GG_SAMPLE_PART_BITS) != 0, do_last = (part & GG_SAMPLE_PART_LAST) != 0;
  Tune tune;
  if (resolve_tuning(tuning, &tune) != GG_OK) return GG_ERR_ARG;
  GG_REQUIRE(W >= 1 && W <= GG_MAX_W, "W = %d outside 1..%d", W, GG_MAX_W);
  GG_REQUIRE(L >= 1 && L <= GG_MAX_LAYERS, "L = %d outside 1..%d", L, GG_MAX_LAYERS);
  GG_REQUIRE(csr->num_nodes >= 1 && csr->num_nodes < (1LL << 31), "num_nodes %lld unsupported",
             (long long)csr->num_nodes);
  GG_REQUIRE(csr->row_ptr_bits == 32 || csr->row_ptr_bits == 64, "row_ptr_bits must be 32 or 64");
  GG_REQUIRE(csr->row_ptr && (csr->num_edges == 0 || csr->col_idx), "CSR arrays are NULL");
  GG_REQUIRE(csr->row_ptr_bits == 64 || csr->num_edges < (1LL << 31),
             "int32 row_ptr with %lld edges", (long long)csr->num_edges);
  for (int l = 0; l < L; ++l)
    GG_REQUIRE(fanout_h[l] >= 1 && fanout_h[l] <= GG_MAX_FANOUT, "fanout[%d] = %d outside 1..%d",
               l, fanout_h[l], GG_MAX_FANOUT);
  GG_REQUIRE(seed_off_h[0] == 0, "seed_off[0] must be 0");
  for (int b = 0; b < W; ++b)
    GG_REQUIRE(seed_off_h[b + 1] >= seed_off_h[b], "seed_off not ascending");
  GG_REQUIRE(seed_off_h[W] == 0 || seeds_d, "seeds are NULL");
  GG_REQUIRE(out->frontier_ids && out->frontier_off && out->nbr_ids && out->nbr_off &&
                 out->frontier_bits && out->need,
             "NULL output buffer");
  GG_REQUIRE(out->frontier_cap >= 0 && out->nbr_cap >= 0, "negative capacity");
  GG_REQUIRE(aligned16(out->frontier_bits), "frontier_bits must be 16-byte aligned");
  const int64_t N = csr->num_nodes;
  SampleWs sw;
  const size_t need_ws = sample_ws_layout(N, W, tune, (char*)ws, &sw);
  GG_REQUIRE(ws && ws_bytes >= need_ws, "workspace of %zu bytes < %zu", ws_bytes, need_ws);

  const int64_t wpb = gg_bits_words(N);
  const int32_t nch = (int32_t)(wpb / kChunkWords);
  const bool slices = use_slices(N, tune);
  const bool last_slices = last_hop_slices(N, W, tune);

  SeedOff so;
  for (int b = 0; b <= GG_MAX_W; ++b) so.off[b] = b <= W ? seed_off_h[b] : INT64_MAX;
  int64_t max_batch = 0;
  for (int b = 0; b < W; ++b)
    max_batch = std::max<int64_t>(max_batch, seed_off_h[b + 1] - seed_off_h[b]);
  // With few chunks in the window, level 0's counts come from k_seed_bits
  // and its emit sums them directly: one launch fewer.  Beside a running
  // gather even a small launch costs 7-12 us.
  const bool seed_counts = max_batch <= kSeedBitsMaxBatch && (int64_t)W * nch <= kCntOnlyMaxChunks;
  if (!do_bits) {
    // the last level only: its count unless the fold already made it, and
    // its emit
  } else if (max_batch <= kSeedBitsMaxBatch) {
    hipLaunchKernelGGL(k_seed_bits, dim3((unsigned)nch, (unsigned)W), dim3(kBlock), 0, stream,
                       seeds_d, so, out->frontier_bits, wpb, N, sw.map, sw.tot,
                       (int32_t)((L + 1) * sw.tot_level), seed_counts ? sw.cnt : nullptr,
                       status_d);
    GG_LAUNCH_CHECK("k_seed_bits");
  } else {
    const int64_t map4 = sw.map ? W * wpb * 2 : 0;   // 32 bytes per word, 16 per store
    hipLaunchKernelGGL(k_zero_words,
                       dim3((unsigned)std::min<int64_t>(cdiv(W * wpb / 4, kBlock), 4096)),
                       dim3(kBlock), 0, stream, out->frontier_bits, W * wpb / 4, sw.map, map4,
                       sw.tot, (int32_t)((L + 1) * sw.tot_level));
    GG_LAUNCH_CHECK("k_zero_words");
    hipLaunchKernelGGL(k_mark_seeds,
                       dim3((unsigned)std::min<int64_t>(cdiv(seed_off_h[W], kBlock), 4096)),
                       dim3(kBlock), 0, stream, seeds_d, so, W, out->frontier_bits, wpb, N,
                       status_d);
    GG_LAUNCH_CHECK("k_mark_seeds");
  }
  // Host bound on each level's entries, for the sampler's grid.
  int64_t bound[GG_MAX_LAYERS + 1] = {0};
  for (int b = 0; b < W; ++b) {
    int64_t lev = std::min<int64_t>(seed_off_h[b + 1] - seed_off_h[b], N);
    for (int l = 0; l <= L; ++l) {
      bound[l] += lev;
      if (l < L) lev = std::min<int64_t>(lev * (fanout_h[l] + 1), N);
    }
  }
  // Hop lv - 1 (making level lv) marks through LDS slices when the graph's
  // sets split into few slices and, before the last hop, when its bound on
  // slots per batch reaches the tuning's minimum.
  int64_t bbound[GG_MAX_LAYERS + 1];   // entries of the largest batch, by level
  {
    int64_t lev = std::min<int64_t>(max_batch, N);
    for (int l = 0; l <= L; ++l) {
      bbound[l] = lev;
      if (l < L) lev = std::min<int64_t>(lev * (fanout_h[l] + 1), N);
    }
  }
  auto lds_marks = [&](int lv) {
    if (lv == L) return last_slices;
    return slices && W >= min_batches(false, tune) &&
           bbound[lv - 1] * fanout_h[lv - 1] >= tune.mark_min_slots;
  };
  const int64_t nruns = wpb / kWordsPerThread;
  int64_t ntab_prev = 0;     // tiles of the previous level's table (0: none)
  int32_t gmax_prev = 1;     // table tiles a sampler tile may join
  for (int lv = 0; lv <= L; ++lv) {
    const bool last = lv == L;
    if (!last && !do_bits) continue;
    if (lv > 0 && do_bits) {
      SampleArgs a;
      a.N = N;
      a.wpb = wpb;
      a.fcap = out->frontier_cap;
      a.ncap = out->nbr_cap;
      a.batch0 = batch0;
      a.W = W;
      a.l = lv - 1;
      a.k = fanout_h[lv - 1];
      a.key0 = (uint32_t)rng_seed;
      a.key1 = (uint32_t)(rng_seed >> 32);
      a.epoch = (uint32_t)epoch;
      a.bytemap = lv == L ? sw.map : nullptr;
      a.nomark = lds_marks(lv) ? 1 : 0;
      const int64_t bnd = std::min<int64_t>(bound[lv - 1], out->frontier_cap);
      int rc = csr->row_ptr_bits == 64
                   ? launch_sample<int64_t>(csr, out, sw, status_d, a, bnd, ntab_prev, gmax_prev,
                                            stream)
                   : launch_sample<int32_t>(csr, out, sw, status_d, a, bnd, ntab_prev, gmax_prev,
                                            stream);
      if (rc != GG_OK) return rc;
    }
    Totals tt;
    tt.gtot = sw.tot + (int64_t)lv * sw.tot_level;
    tt.ngroups = sw.ngroups;
    const bool cnt_only = lv == 0 && seed_counts;
    // the last level's count folds the byte map, or makes the marks, which
    // the hot set needs, so it belongs to the bits part then; after atomic
    // marks it belongs to the compaction
    const bool count_here = last ? ((sw.map || last_slices) ? do_bits : do_last) : do_bits;
    if (!cnt_only && count_here && lv > 0 && lds_marks(lv)) {
      MarkArgs ma;
      ma.N = N;
      ma.wpb = wpb;
      ma.ncap = out->nbr_cap;
      ma.W = W;
      ma.l = lv - 1;
      ma.k = fanout_h[lv - 1];
      ma.nch = nch;
      ma.vec = aligned16(out->nbr_ids) ? 1 : 0;
      ma.schunks = tune.mark_slice_chunks;
      ma.nslices = (int32_t)mark_slices(N, tune);
      ma.pad_ = 0;
      const dim3 mg((unsigned)(ma.nslices * cdiv(W, kXcds) * kXcds));
      // the slice, and a word per lane of a wavefront for the marks that miss it
      const size_t lds = ((size_t)tune.mark_slice_chunks * kChunkWords + kWave) * 4;
      if (tune.mark_block == 1024)
        hipLaunchKernelGGL(k_mark_slices_1024, mg, dim3(1024), lds, stream, out->frontier_bits,
                           out->nbr_ids, out->nbr_off, sw.lvl, sw.cnt, tt, ma);
      else
        hipLaunchKernelGGL(k_mark_slices_256, mg, dim3(256), lds, stream, out->frontier_bits,
                           out->nbr_ids, out->nbr_off, sw.lvl, sw.cnt, tt, ma);
      GG_LAUNCH_CHECK("k_mark_slices");
    } else if (!cnt_only && count_here) {
      hipLaunchKernelGGL(k_bits_count, dim3(nch, W), dim3(kBlock), 0, stream, out->frontier_bits,
                         wpb, lv == L ? sw.map : nullptr, sw.cnt, tt);
      GG_LAUNCH_CHECK("k_bits_count");
    }
    LevelArgs la;
    la.lv = lv;
    la.L = L;
    la.W = W;
    la.k = lv < L ? fanout_h[lv] : 0;
    la.nch = nch;
    la.cnt_only = cnt_only ? 1 : 0;
    la.fcap = out->frontier_cap;
    la.ncap = out->nbr_cap;
    // the tile table for the next hop's sampler
    la.tile_runs = (lv < L && sw.tstart) ? tile_runs_for(tune, lv, L, nruns, bound[lv]) : 0;
    la.ntiles = la.tile_runs ? nruns / la.tile_runs : 0;
    la.tstart = la.tile_runs ? sw.tstart : nullptr;
    la.pad_ = 0;
    ntab_prev = la.ntiles;
    // a fixed tile size is kept as is; otherwise tiles of up to 64 runs
    gmax_prev = tune.sample_tile_runs > 0 ? 1 : (la.tile_runs ? 64 / la.tile_runs : 1);
    if (last && !do_last) break;
    hipLaunchKernelGGL(k_bits_emit, dim3(nch, W), dim3(kBlock), 0, stream, out->frontier_bits, wpb,
                       sw.cnt, tt, out->frontier_ids, out->frontier_off, out->nbr_off, sw.lvl,
                       out->need, status_d, la);
    GG_LAUNCH_CHECK("k_bits_emit");
  }
  return GG_OK;
}

}  // namespace
}  // namespace gg

extern "C" int gg_sample_window(const gg_csr_t* csr, const int32_t* seeds_d,
                                const int64_t* seed_off_h, int32_t W, const int32_t* fanout_h,
                                int32_t L, uint64_t rng_seed, int32_t epoch, int64_t batch0,
                                const gg_wsample_t* out, const gg_tuning_t* tuning,
                                int32_t* status_d, void* ws, size_t ws_bytes,
                                hipStream_t stream) {
  return sample_window_impl(csr, seeds_d, seed_off_h, W, fanout_h, L, rng_seed, epoch, batch0,
                            out, tuning, status_d, ws, ws_bytes,
                            GG_SAMPLE_PART_BITS | GG_SAMPLE_PART_LAST, stream);
}

extern "C" int gg_sample_window_part(const gg_csr_t* csr, const int32_t* seeds_d,
                                     const int64_t* seed_off_h, int32_t W,
                                     const int32_t* fanout_h, int32_t L, uint64_t rng_seed,
                                     int32_t epoch, int64_t batch0, const gg_wsample_t* out,
                                     int32_t part, const gg_tuning_t* tuning, int32_t* status_d,
                                     void* ws, size_t ws_bytes, hipStream_t stream) {
  GG_REQUIRE(part == GG_SAMPLE_PART_BITS || part == GG_SAMPLE_PART_LAST, "part %d is not GG_SAMPLE_PART_BITS "
             "or GG_SAMPLE_PART_LAST", part);
  return sample_window_impl(csr, seeds_d, seed_off_h, W, fanout_h, L, rng_seed, epoch, batch0,
                            out, tuning, status_d, ws, ws_bytes, part, stream);
}
