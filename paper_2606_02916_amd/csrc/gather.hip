// gg_gather_batch: feature assembly of one or more consecutive batches
// through the ID-to-slot remap, with the on-demand miss path.
//
// Grid (bx, nseg): blocks (., s) serve segment (batch) s, so every block's
// statistics belong to one batch and reduce without atomics.  Each
// wavefront takes a tile of consecutive output rows at a time (up to 64
// rows and 8 KB); every lane of the tile resolves
// its row (local shard, cache slot, or miss) and the wave copies the
// resolved rows with the row copy engine.  Misses are only counted, per
// block and owner.  A second launch serves them: one block per row block
// of the first launch, which returns at once when that block counted no
// miss and otherwise walks the same tiles again and copies the missed rows
// from their owners' shards straight into their output rows.  No queue and
// no counter need clearing between calls.
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "gg_host.hpp"

// Scratch of gg_gather_batch_noalloc (see device_scratch below).
static __device__ __align__(256) int32_t scratch[GG_GATHER_SCRATCH_BYTES / sizeof(int32_t)];

namespace gg {
namespace {

constexpr int kTilesPerBlock = kBlock / kWave;  // 4 waves
// Blocks per launch, shared by the segments (tuning gather_blocks): the
// default 1024 (four per CU) beat 512, 768, 1536 and 2048 on a 1.5M-row
// window, alone (236 us warm, 267 us cold) and beside the next window's
// sampling.

struct GatherArgs {
  int64_t n_cap;        // output rows available
  int64_t cache_stride;
  int64_t cache_rows;
  int64_t out_stride;
  int32_t nseg;
  int32_t nstat;        // 2 + P counters per block
  int32_t tile;         // rows per wave step (copy_tile)
  int32_t pad_;
  CopyGeom geom;
};

// Output rows [lo, hi) of segment s, relative to bounds[0], clamped to n_cap.
__device__ __forceinline__ void seg_range(const int64_t* bounds, int s, const GatherArgs& a,
                                          int64_t* lo, int64_t* hi) {
  const int64_t b0 = bounds[0];
  int64_t l = bounds[s] - b0, h = bounds[s + 1] - b0;
  l = l < 0 ? 0 : (l > a.n_cap ? a.n_cap : l);
  h = h < l ? l : (h > a.n_cap ? a.n_cap : h);
  *lo = l;
  *hi = h;
}

// Row ids and owners of one tile, loaded ahead of its copy.
struct TileIds {
  int32_t u;      // row id, or -1 for a lane past the tile or the segment
  int32_t m;      // owner of u (-1 when u is absent or out of range)
  int32_t s;      // slot of u for a remote owner, loaded one tile ahead
  bool in;        // the lane holds a row of the segment
};

__device__ __forceinline__ bool tile_lane(int64_t t, int64_t ntiles, int64_t lo, int64_t hi,
                                          int32_t tile, int lane) {
  return t < ntiles && lane < tile && lo + t * tile + lane < hi;
}

template <int VB, bool NT, int U>
__global__ void __launch_bounds__(kBlock) k_gather_rows(const int32_t* in_ids, const int64_t* bounds,
                                                        KPart part, KFeat feat, GatherArgs a,
                                                        const char* cache, const int32_t* slot_of,
                                                        char* out, int32_t* blk_stat,
                                                        int32_t* status) {
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  __shared__ int32_t s_cnt[2 + GG_MAX_PARTS];  // local, hits, misses per owner
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  for (int t = threadIdx.x; t < 2 + GG_MAX_PARTS; t += blockDim.x) s_cnt[t] = 0;
  __syncthreads();
  const int seg = blockIdx.y;
  int64_t lo, hi;
  seg_range(bounds, seg, a, &lo, &hi);
  const int64_t begin = bounds[0];
  const int lane = lane_id();
  const int64_t ntiles = (hi - lo + a.tile - 1) / a.tile;
  const int64_t step = (int64_t)gridDim.x * kTilesPerBlock;
  int32_t st = 0;
  int32_t c_local = 0, c_hit = 0;
  // Software pipeline over the wave's tiles: while tile t is copied, the
  // slots of tile t + step and the ids of tile t + 2 step are already in
  // flight, so neither lookup waits in front of a copy.
  auto load_ids = [&](int64_t t) -> TileIds {
    TileIds x{-1, -1, -1, tile_lane(t, ntiles, lo, hi, a.tile, lane)};
    if (x.in) x.u = in_ids[begin + lo + t * a.tile + lane];
    return x;
  };
  auto load_slot = [&](TileIds& x) {
    if (x.in && x.u >= 0 && (int64_t)x.u < part.N) {
      x.m = owner_of(part, s_start, x.u);
      if (x.m != part.local) x.s = slot_of[x.u];
    }
  };
  int64_t t = (int64_t)blockIdx.x * kTilesPerBlock + threadIdx.x / kWave;
  TileIds cur = load_ids(t);
  load_slot(cur);
  TileIds nxt = load_ids(t + step);
  for (; t < ntiles; t += step) {
    load_slot(nxt);
    const TileIds after = load_ids(t + 2 * step);
    const char* src = nullptr;
    bool miss = false, is_local = false, is_hit = false;
    if (cur.in) {
      if (cur.m < 0) {
        st |= GG_DEV_BAD_ID;
      } else if (cur.m == part.local) {
        const int64_t r = row_of(part, s_start, cur.u, cur.m);
        if (r < feat.rows[cur.m]) {
          src = feat.shard[cur.m] + r * feat.stride[cur.m];
          is_local = true;
        } else {
          st |= GG_DEV_BAD_ROW;
        }
      } else if (cur.s >= 0 && (int64_t)cur.s < a.cache_rows) {
        src = cache + (int64_t)cur.s * a.cache_stride;
        is_hit = true;
      } else {
        if (cur.s >= 0) st |= GG_DEV_BAD_ROW;
        miss = true;
      }
    }
    const uint64_t ml = __ballot(is_local), mh = __ballot(is_hit), mm = __ballot(miss);
    c_local += (int32_t)__popcll(ml);
    c_hit += (int32_t)__popcll(mh);
    // Per-owner miss counts: one ballot per owner present.
    for (uint64_t act = mm; act;) {
      const int leader = __ffsll((unsigned long long)act) - 1;
      const int32_t ol = __shfl(cur.m, leader, kWave);
      const uint64_t sel = __ballot(miss && cur.m == ol);
      if (lane == leader) atomicAdd(&s_cnt[2 + ol], (int32_t)__popcll(sel));
      act &= ~sel;
    }
    const int64_t r0 = lo + t * a.tile;
    const int64_t left = hi - r0;
    const int nrows = left < a.tile ? (int)left : a.tile;
    wave_copy_rows<VB, NT, U>(src, out + r0 * a.out_stride, a.out_stride, nrows, a.geom);
    cur = nxt;
    nxt = after;
  }
  if (lane == 0) {
    if (c_local) atomicAdd(&s_cnt[0], c_local);
    if (c_hit) atomicAdd(&s_cnt[1], c_hit);
  }
  if (st) set_status(status, st);
  __syncthreads();
  int32_t* dst = blk_stat + ((int64_t)seg * gridDim.x + blockIdx.x) * a.nstat;
  for (int t = threadIdx.x; t < a.nstat; t += blockDim.x) dst[t] = s_cnt[t];
}

// Blocks 0 .. nseg-1: statistics of batch s.  Block nseg + s * bx + x
// serves the misses of row block (x, s) of k_gather_rows, if it had any.
template <int VB, bool NT>
__global__ void __launch_bounds__(kBlock) k_gather_finish(const int32_t* in_ids, const int64_t* bounds,
                                                          KPart part, KFeat feat, GatherArgs a,
                                                          int32_t bx, const int32_t* blk_stat,
                                                          const int32_t* slot_of, char* out,
                                                          gg_gather_stats_t* stats,
                                                          int32_t* status) {
  const int P = part.P;
  if ((int)blockIdx.x < a.nseg) {
    __shared__ int32_t s_sum[2 + GG_MAX_PARTS];
    const int s = blockIdx.x;
    for (int t = threadIdx.x; t < 2 + GG_MAX_PARTS; t += blockDim.x) s_sum[t] = 0;
    __syncthreads();
    for (int j = 0; j < a.nstat; ++j) {
      int32_t v = 0;
      for (int x = threadIdx.x; x < bx; x += blockDim.x) v += blk_stat[((int64_t)s * bx + x) * a.nstat + j];
      v = wave_sum(v);
      if (lane_id() == 0 && v) atomicAdd(&s_sum[j], v);
    }
    __syncthreads();
    gg_gather_stats_t* o = stats + s;
    if (threadIdx.x < GG_MAX_PARTS) {
      const int m = threadIdx.x;
      const int64_t rows = m < P ? (int64_t)s_sum[2 + m] : 0;
      o->miss_rows[m] = rows;
      o->miss_requests[m] = rows > 0 ? 1 : 0;
    }
    if (threadIdx.x == 0) {
      int64_t misses = 0;
      for (int m = 0; m < P; ++m) misses += s_sum[2 + m];
      int64_t lo, hi;
      seg_range(bounds, s, a, &lo, &hi);
      o->rows = hi - lo;
      o->local = s_sum[0];
      o->hits = s_sum[1];
      o->misses = misses;
      if (bounds[s + 1] - bounds[0] > a.n_cap) set_status(status, GG_DEV_CAPACITY);
    }
    return;
  }
  const int64_t rb = blockIdx.x - a.nseg;    // row block (x, seg) of k_gather_rows
  const int seg = (int)(rb / bx), x = (int)(rb % bx);
  const int32_t* bs = blk_stat + rb * a.nstat;
  int32_t nmiss = 0;
  for (int m = 0; m < P; ++m) nmiss += bs[2 + m];
  if (nmiss == 0) return;
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  __syncthreads();
  int64_t lo, hi;
  seg_range(bounds, seg, a, &lo, &hi);
  const int64_t begin = bounds[0];
  const int lane = lane_id();
  const int64_t ntiles = (hi - lo + a.tile - 1) / a.tile;
  int32_t st = 0;
  // The tiles k_gather_rows gave this row block, in the same order.
  for (int64_t t = (int64_t)x * kTilesPerBlock + threadIdx.x / kWave; t < ntiles;
       t += (int64_t)bx * kTilesPerBlock) {
    const int64_t r0 = lo + t * a.tile;
    const int64_t i = r0 + lane;
    const char* src = nullptr;
    if (lane < a.tile && i < hi) {
      const int32_t u = in_ids[begin + i];
      if (u >= 0 && (int64_t)u < part.N) {
        const int32_t m = owner_of(part, s_start, u);
        if (m != part.local) {
          const int32_t sl = slot_of[u];
          if (!(sl >= 0 && (int64_t)sl < a.cache_rows)) {
            const int64_t r = row_of(part, s_start, u, m);
            if (r < feat.rows[m])
              src = feat.shard[m] + r * feat.stride[m];
            else
              st |= GG_DEV_BAD_ROW;
          }
        }
      }
    }
    if (__ballot(src != nullptr)) {
      const int64_t left = hi - r0;
      wave_copy_rows<VB, NT>(src, out + r0 * a.out_stride, a.out_stride,
                             left < a.tile ? (int)left : a.tile, a.geom);
    }
  }
  if (st) set_status(status, st);
}

struct GatherWs {
  int32_t* blk_stat;   // per row block: local, hits, misses per owner
};

int32_t blocks_per_seg(int64_t n_cap, int32_t nseg, const Tune& tune) {
  int64_t bx = std::max<int64_t>(tune.gather_blocks / nseg, 8);
  bx = std::min<int64_t>(bx, std::max<int64_t>(1, cdiv(n_cap, kBlock)));
  return (int32_t)bx;
}

size_t gather_ws_layout(int64_t n_cap, int32_t nseg, int32_t P, const Tune& tune, char* base,
                        GatherWs* out) {
  const int64_t bx = blocks_per_seg(n_cap, nseg, tune);
  Carve cv{base, 0, ~(size_t)0};
  GatherWs g;
  g.blk_stat = cv.take<int32_t>((size_t)(nseg * bx * (2 + P)));
  if (out) *out = g;
  return align_up(cv.used, 256);
}

template <int VB, bool NT>
void launch_gather(hipStream_t stream, int unroll, int32_t bx, const int32_t* in_ids, const int64_t* bounds,
                   const KPart& kp, const KFeat& kf, const GatherArgs& a, const char* cache,
                   const int32_t* slot_of, char* out, const GatherWs& w, gg_gather_stats_t* stats,
                   int32_t* status) {
  if (VB == 16 && unroll == 8)
    hipLaunchKernelGGL((k_gather_rows<VB, NT, 8>), dim3(bx, a.nseg), dim3(kBlock), 0, stream, in_ids,
                       bounds, kp, kf, a, cache, slot_of, out, w.blk_stat, status);
  else if (VB == 16 && unroll == 4)
    hipLaunchKernelGGL((k_gather_rows<VB, NT, 4>), dim3(bx, a.nseg), dim3(kBlock), 0, stream, in_ids,
                       bounds, kp, kf, a, cache, slot_of, out, w.blk_stat, status);
  else if (VB == 16 && unroll == 2)
    hipLaunchKernelGGL((k_gather_rows<VB, NT, 2>), dim3(bx, a.nseg), dim3(kBlock), 0, stream, in_ids,
                       bounds, kp, kf, a, cache, slot_of, out, w.blk_stat, status);
  else
    hipLaunchKernelGGL((k_gather_rows<VB, NT, VB == 16 ? 4 : 8>), dim3(bx, a.nseg), dim3(kBlock), 0,
                       stream, in_ids, bounds, kp, kf, a, cache, slot_of, out, w.blk_stat, status);
  hipLaunchKernelGGL((k_gather_finish<VB, NT>), dim3(a.nseg + a.nseg * bx), dim3(kBlock), 0, stream,
                     in_ids, bounds, kp, kf, a, bx, w.blk_stat, slot_of, out, stats, status);
}

}  // namespace
}  // namespace gg

using namespace gg;

extern "C" size_t gg_ws_gather(int64_t n_cap, int32_t nseg, int32_t num_parts,
                               const gg_tuning_t* tuning) {
  Tune tune;
  if (resolve_tuning(tuning, &tune) != GG_OK) return 0;
  // Every call with at most nseg segments and n_cap rows fits: the blocks
  // per segment divide the gather's block count, so fewer segments can
  // launch more blocks in all (1024 blocks: 3 x 341, but 1 x 1024).
  size_t need = 0;
  for (int32_t s = 1; s <= std::min(std::max(nseg, 1), GG_MAX_W); ++s)
    need = std::max(need, gather_ws_layout(n_cap, s, num_parts, tune, nullptr, nullptr));
  return need;
}

namespace gg {
namespace {

// The per-block statistics of gg_gather_batch_noalloc: a file-scope device
// array, one copy per GPU, held until the process ends.  Host code never
// hands the array's name to a kernel (in host code it is a stand-in, not a
// device address): it takes the array's address on each device from
// hipGetSymbolAddress, once, with that device current.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int device_scratch(hipStream_t stream, void** out) {
  int dev = 0;
  hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) {
    set_error("gg_gather_batch_noalloc: no device for the stream: %s", hipGetErrorString(e));
    return GG_ERR_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    set_error("gg_gather_batch_noalloc: device %d beyond the %d supported", dev, kMaxDevices);
    return GG_ERR_UNSUPPORTED;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = 0;
    e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    void* p = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p) {
      set_error("gg_gather_batch_noalloc: address of the scratch array on device %d: %s", dev,
                hipGetErrorString(e));
      return GG_ERR_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return GG_OK;
}

// Both gather entry points: ws/ws_bytes is the caller's workspace, or with
// noalloc the device array (ws is then ignored).
int gather_impl(const int32_t* in_ids_d, const int64_t* bounds_d, int32_t nseg, int64_t n_cap,
                const gg_part_t* part, const gg_feat_t* feat, const void* cache_d,
                int64_t cache_stride, int64_t cache_rows, const int32_t* slot_of_d, void* out_d,
                int64_t out_stride, int32_t flags, gg_gather_stats_t* stats_d,
                const gg_tuning_t* tuning, int32_t* status_d, void* ws, size_t ws_bytes,
                bool noalloc, hipStream_t stream) {
  GG_REQUIRE(bounds_d && slot_of_d && stats_d && status_d, "NULL argument");
  Tune tune;
  if (resolve_tuning(tuning, &tune) != GG_OK) return GG_ERR_ARG;
  GG_REQUIRE((flags & ~GG_GATHER_SHARED) == 0, "unknown flags 0x%x", (unsigned)flags);
  GG_REQUIRE(nseg >= 1 && nseg <= GG_MAX_W, "nseg = %d outside 1..%d", nseg, GG_MAX_W);
  GG_REQUIRE(n_cap >= 0 && n_cap < (1LL << 31), "n_cap %lld unsupported", (long long)n_cap);
  GG_REQUIRE(n_cap == 0 || (in_ids_d && out_d), "NULL id or output buffer");
  GG_REQUIRE(cache_rows >= 0 && (cache_rows == 0 || cache_d), "cache is NULL");
  KPart kp;
  int rc = pack_part(part, &kp);
  if (rc != GG_OK) return rc;
  KFeat kf;
  rc = pack_feat(feat, part, &kf);
  if (rc != GG_OK) return rc;
  GG_REQUIRE(out_stride >= kf.row_bytes && out_stride % 4 == 0, "out_stride %lld invalid",
             (long long)out_stride);
  GG_REQUIRE(cache_rows == 0 || (cache_stride >= kf.row_bytes && cache_stride % 4 == 0),
             "cache_stride %lld invalid", (long long)cache_stride);
  GG_REQUIRE(((uintptr_t)out_d & 3u) == 0 && ((uintptr_t)cache_d & 3u) == 0,
             "output and cache must be 4-byte aligned");
  const size_t need_ws = gather_ws_layout(n_cap, nseg, kp.P, tune, nullptr, nullptr);
  if (noalloc) {
    if (need_ws > (size_t)GG_GATHER_SCRATCH_BYTES) {
      set_error("gg_gather_batch_noalloc: %d segments of %d blocks with %d owners need %zu bytes "
                "of scratch; the library's array holds %d",
                nseg, blocks_per_seg(n_cap, nseg, tune), kp.P, need_ws, GG_GATHER_SCRATCH_BYTES);
      return GG_ERR_CAPACITY;
    }
    rc = device_scratch(stream, &ws);
    if (rc != GG_OK) return rc;
    ws_bytes = GG_GATHER_SCRATCH_BYTES;
  }
  GG_REQUIRE(ws && ws_bytes >= need_ws, "workspace of %zu bytes < %zu", ws_bytes, need_ws);
  GatherWs gw;
  gather_ws_layout(n_cap, nseg, kp.P, tune, (char*)ws, &gw);
  bool v16 = aligned16(out_d) && out_stride % 16 == 0 &&
             (cache_rows == 0 || (aligned16(cache_d) && cache_stride % 16 == 0));
  for (int m = 0; m < kf.P; ++m)
    if (kf.rows[m] > 0) v16 = v16 && aligned16(kf.shard[m]) && kf.stride[m] % 16 == 0;
  GatherArgs a;
  a.n_cap = n_cap;
  a.cache_stride = cache_stride;
  a.cache_rows = cache_rows;
  a.out_stride = out_stride;
  a.nseg = nseg;
  a.nstat = 2 + kp.P;
  // Tiles of up to 8 KB.  Against 32 KB tiles the isolated gather took 228
  // instead of 237 us on a 1.5M-row window of 400-byte rows and 246 instead
  // of 261 us on 275K rows of 2,408 bytes: more, smaller tiles leave a
  // shorter tail of waves still copying their last tile.  With four loads
  // in flight (shared) a tile holds as many rows as fit, 20 of 400 bytes
  // (500 chunks: two steps of 256 loads, 98% full), which took the isolated
  // gather from 0.58 to 0.60 of HBM peak on that window and from 0.55 to
  // 0.57 on the wide rows; with eight (alone) it stays a power of two, 16
  // rows and 2, which measured 1-3% faster there than 20 and 3.
  const bool shared = (flags & GG_GATHER_SHARED) != 0;
  a.tile = copy_tile(tune, kf.row_bytes, 8192, !shared);
  a.pad_ = 0;
  a.geom = copy_geom(kf.row_bytes, v16 ? 16 : 4);
  const int32_t bx = blocks_per_seg(n_cap, nseg, tune);
  // Row loads in flight per lane: eight alone; four when sharing the chip
  // (with eight, a concurrent sampler ran ~15% slower and the look-ahead
  // window took 6% longer, for 4% more gather speed).
  const int unroll = tune.gather_loads ? tune.gather_loads
                                       : (shared ? kGatherLoadsShared : kGatherLoadsAlone);
  const char* cache = (const char*)cache_d;
  char* out = (char*)out_d;
  // Output rows are stored non-temporally: the gather never reads them back.
  if (v16)
    launch_gather<16, true>(stream, unroll, bx, in_ids_d, bounds_d, kp, kf, a, cache, slot_of_d,
                            out, gw, stats_d, status_d);
  else
    launch_gather<4, true>(stream, unroll, bx, in_ids_d, bounds_d, kp, kf, a, cache, slot_of_d,
                           out, gw, stats_d, status_d);
  GG_LAUNCH_CHECK("k_gather_rows/k_gather_finish");
  return GG_OK;
}

}  // namespace
}  // namespace gg

extern "C" int gg_gather_batch(const int32_t* in_ids_d, const int64_t* bounds_d, int32_t nseg,
                               int64_t n_cap, const gg_part_t* part, const gg_feat_t* feat,
                               const void* cache_d, int64_t cache_stride, int64_t cache_rows,
                               const int32_t* slot_of_d, void* out_d, int64_t out_stride,
                               int32_t flags, gg_gather_stats_t* stats_d,
                               const gg_tuning_t* tuning, int32_t* status_d, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  return gather_impl(in_ids_d, bounds_d, nseg, n_cap, part, feat, cache_d, cache_stride,
                     cache_rows, slot_of_d, out_d, out_stride, flags, stats_d, tuning, status_d,
                     ws, ws_bytes, false, stream);
}

extern "C" int gg_gather_batch_noalloc(const int32_t* in_ids_d, const int64_t* bounds_d,
                                       int32_t nseg, int64_t n_cap, const gg_part_t* part,
                                       const gg_feat_t* feat, const void* cache_d,
                                       int64_t cache_stride, int64_t cache_rows,
                                       const int32_t* slot_of_d, void* out_d, int64_t out_stride,
                                       int32_t flags, gg_gather_stats_t* stats_d,
                                       const gg_tuning_t* tuning, int32_t* status_d,
                                       hipStream_t stream) {
  return gather_impl(in_ids_d, bounds_d, nseg, n_cap, part, feat, cache_d, cache_stride,
                     cache_rows, slot_of_d, out_d, out_stride, flags, stats_d, tuning, status_d,
                     nullptr, 0, true, stream);
}
