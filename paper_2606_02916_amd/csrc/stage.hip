// gg_stage_bulk: one bulk request per non-empty owner bucket into the
// window cache, plus the ID-to-slot remap.
//
// The bucketed hot set is owner-major, so each owner's rows form one
// contiguous run of cache slots: the bulk request of owner m is the copy of
// slots owner_off[m] .. owner_off[m+1] from shard m.  All owners' requests
// go out in one launch; each wavefront copies 64 consecutive slots with the
// row copy engine and writes slot_of for them.
#include <stdlib.h>
#include <string.h>

#include "gg_host.hpp"

namespace gg {
namespace {

__device__ __forceinline__ int64_t cdiv_dev(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct StageArgs {
  int64_t cap;         // bucket entries usable
  int64_t cache_rows;
  int64_t cache_stride;
  int32_t tile;        // slots per wave step (copy_tile)
  int32_t pad_;
  CopyGeom geom;
};

__device__ __forceinline__ int64_t stage_n(const int64_t* owner_off, int32_t P, const StageArgs& a) {
  int64_t n = owner_off[P];
  n = n < a.cap ? n : a.cap;
  return n < a.cache_rows ? n : a.cache_rows;
}

// Bucket entries an in-place call handles: every entry, since a retained
// row keeps its slot wherever it sits in the list, and a delta row past the
// free slots is left uncached rather than dropped from the count.
__device__ __forceinline__ int64_t inplace_n(const int64_t* owner_off, int32_t P,
                                             const StageArgs& a) {
  const int64_t n = owner_off[P];
  return n < a.cap ? n : a.cap;
}

// Old slots and the rebuild delta: old_slot[s] = the slot the source remap
// (or, without a source cache, the current remap before clearing) gives
// the node of bucket entry s; rows with none are the delta.  Every block
// writes its per-owner delta counts to dcnt[block * P + m].
// When the old slots come from a different remap than the one being
// rebuilt, the same launch also clears the rebuilt remap's entries
// clear[0 .. clear_count[0]) (otherwise k_slot_reset does, afterwards).
__global__ void __launch_bounds__(kBlock) k_stage_delta(const int32_t* bucket, const int64_t* owner_off,
                                                        KPart part, StageArgs a, const int32_t* before,
                                                        int32_t* old_slot, int32_t* dcnt,
                                                        const int32_t* clear,
                                                        const int64_t* clear_count,
                                                        int32_t* slot_of) {
  __shared__ int32_t hist[GG_MAX_PARTS];
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  for (int t = threadIdx.x; t < GG_MAX_PARTS; t += blockDim.x) hist[t] = 0;
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  __syncthreads();
  const int64_t n = stage_n(owner_off, part.P, a);
  for (int64_t base = (int64_t)blockIdx.x * blockDim.x + (threadIdx.x & ~(kWave - 1)); base < n;
       base += (int64_t)gridDim.x * blockDim.x) {
    const int64_t s = base + lane_id();
    bool fresh = false;
    int32_t m = 0;
    if (s < n) {
      const int32_t u = bucket[s];
      int32_t old = -1;
      if (u >= 0 && (int64_t)u < part.N) {
        old = before[u];
        if (old < 0) {
          fresh = true;
          m = owner_of(part, s_start, u);
        }
      }
      old_slot[s] = old;
    }
    wave_hist_add(hist, fresh, m);
  }
  if (clear) {
    const int64_t nc = clear_count[0];
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nc;
         i += (int64_t)gridDim.x * blockDim.x) {
      const int32_t u = clear[i];
      if (u >= 0 && (int64_t)u < part.N) slot_of[u] = -1;
    }
  }
  __syncthreads();
  for (int m = threadIdx.x; m < part.P; m += blockDim.x) dcnt[(int64_t)blockIdx.x * part.P + m] = hist[m];
}

__global__ void __launch_bounds__(kBlock) k_slot_reset(const int32_t* prev, const int64_t* prev_count,
                                                       int64_t N, int32_t* slot_of) {
  const int64_t n = prev_count[0];
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t u = prev[i];
    if (u >= 0 && (int64_t)u < N) slot_of[u] = -1;
  }
}

// Statistics of the call: per-owner requests, rows and bytes and the
// rebuild delta.  Their inputs (owner_off, the delta counts of
// k_stage_delta) are complete before k_stage_rows starts, so its block 0
// computes them.
struct StageStatsArgs {
  const int64_t* prev_count;
  const int32_t* dcnt;
  gg_stage_stats_t* stats;
  // In place only (else NULL): the free slots below the previous extent and
  // the previous occupancy (NULL for a first window).  The delta takes free
  // slots in bucket order, i.e. owner by owner, so owner m's delta rows
  // copied are those of its ranks below the slots available.
  const int64_t* nfree;
  const uint8_t* occ_prev;
  int32_t nblk_delta;
  int32_t has_src;
};

__device__ void stage_stats(const int64_t* owner_off, const KPart& part, const StageArgs& a,
                            int32_t row_bytes, const StageStatsArgs& sa, int32_t* status) {
  const int64_t* prev_count = sa.prev_count;
  const int32_t* dcnt = sa.dcnt;
  const int32_t nblk_delta = sa.nblk_delta, has_src = sa.has_src;
  gg_stage_stats_t* stats = sa.stats;
  __shared__ int32_t s_delta[GG_MAX_PARTS];
  for (int t = threadIdx.x; t < GG_MAX_PARTS; t += blockDim.x) s_delta[t] = 0;
  __syncthreads();
  for (int m = 0; m < part.P; ++m) {
    int32_t v = 0;
    for (int x = threadIdx.x; x < nblk_delta; x += blockDim.x) v += dcnt[(int64_t)x * part.P + m];
    v = wave_sum(v);
    if (lane_id() == 0 && v) atomicAdd(&s_delta[m], v);
  }
  __syncthreads();
  const int64_t n = sa.nfree ? inplace_n(owner_off, part.P, a) : stage_n(owner_off, part.P, a);
  // slots the delta can take (in place): free ones below the previous
  // extent, and every slot from the extent to the end of the cache
  int64_t avail = INT64_MAX;
  if (sa.nfree) {
    int64_t ext = sa.occ_prev ? *(const int64_t*)sa.occ_prev : 0;
    ext = ext < a.cache_rows ? ext : a.cache_rows;
    avail = *sa.nfree + (a.cache_rows - ext);
  }
  __shared__ int64_t s_req[GG_MAX_PARTS], s_rows[GG_MAX_PARTS];
  if (threadIdx.x < GG_MAX_PARTS) {
    const int m = threadIdx.x;
    int64_t rows = 0;
    if (m < part.P) {
      int64_t lo = owner_off[m], hi = owner_off[m + 1];
      lo = lo < n ? lo : n;
      hi = hi < n ? hi : n;
      rows = hi > lo ? hi - lo : 0;
      if (has_src) {                     // only the delta is requested
        int64_t before = 0;              // delta ranks of the owners before m
        for (int q = 0; q < m; ++q) before += s_delta[q];
        const int64_t fit = avail - before;
        rows = fit <= 0 ? 0 : (fit < s_delta[m] ? fit : (int64_t)s_delta[m]);
      }
    }
    stats->rows[m] = rows;
    stats->bytes[m] = rows * row_bytes;
    stats->requests[m] = rows > 0 ? 1 : 0;
    stats->delta_rows[m] = s_delta[m];
    s_req[m] = rows > 0 ? 1 : 0;
    s_rows[m] = rows;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t req = 0, delta = 0;
    for (int m = 0; m < part.P; ++m) {
      req += s_req[m];
      delta += s_delta[m];
    }
    stats->rows_total = n;
    stats->requests_total = req;
    stats->invalidated = prev_count ? prev_count[0] : 0;
    stats->retained = has_src ? n - delta : 0;
    if (owner_off[part.P] > n) set_status(status, GG_DEV_CAPACITY);
  }
}

template <int VB, bool NT>
__global__ void __launch_bounds__(kBlock) k_stage_rows(const int32_t* bucket, const int64_t* owner_off,
                                                       KPart part, KFeat feat, StageArgs a,
                                                       char* cache, int32_t* slot_of,
                                                       const char* src_cache, const int32_t* old_slot,
                                                       StageStatsArgs sa, int32_t* status) {
  if (blockIdx.x == 0) stage_stats(owner_off, part, a, feat.row_bytes, sa, status);
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  __syncthreads();
  const int64_t n = stage_n(owner_off, part.P, a);
  const int64_t ntiles = (n + a.tile - 1) / a.tile;
  const int lane = lane_id();
  int32_t st = 0;
  for (int64_t tile = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; tile < ntiles;
       tile += (int64_t)gridDim.x * (kBlock / kWave)) {
    const int64_t s0 = tile * a.tile;
    const int64_t s = s0 + lane;
    const char* src = nullptr;
    if (lane < a.tile && s < n) {
      const int32_t u = bucket[s];
      if (u < 0 || (int64_t)u >= part.N) {
        st |= GG_DEV_BAD_ID;
      } else {
        const int32_t old = src_cache ? old_slot[s] : -1;
        if (old >= 0 && (int64_t)old < a.cache_rows) {
          src = src_cache + (int64_t)old * a.cache_stride;   // retained: device-local copy
          slot_of[u] = (int32_t)s;
        } else {
          if (old >= 0) st |= GG_DEV_BAD_ROW;
          const int32_t m = owner_of(part, s_start, u);
          const int64_t r = row_of(part, s_start, u, m);
          if (r >= feat.rows[m]) {
            st |= GG_DEV_BAD_ROW;
          } else {
            src = feat.shard[m] + r * feat.stride[m];          // requested from owner m
            slot_of[u] = (int32_t)s;
          }
        }
      }
    }
    const int nrows = (int)((n - s0) < a.tile ? (n - s0) : a.tile);
    wave_copy_rows<VB, NT>(src, cache + s0 * a.cache_stride, a.cache_stride, nrows, a.geom);
  }
  if (st) set_status(status, st);
}

// Cache rows are stored with ordinary stores: the gathers read them next.
template <int VB>
void launch_stage_rows(int grid, hipStream_t stream, const int32_t* bucket,
                       const int64_t* owner_off, const KPart& kp, const KFeat& kf,
                       const StageArgs& a, char* cache, int32_t* slot_of, const char* src_cache,
                       const int32_t* old_slot, const StageStatsArgs& sa, int32_t* status) {
  hipLaunchKernelGGL((k_stage_rows<VB, false>), dim3(grid), dim3(kBlock), 0, stream, bucket,
                     owner_off, kp, kf, a, cache, slot_of, src_cache, old_slot, sa, status);
}

int stage_delta_blocks(int64_t cap) {
  return (int)std::min<int64_t>(std::max<int64_t>(cdiv(cap, kBlock), 1), 1024);
}

// ---------------------------------------------------------------------------
// In-place staging into one persistent cache.  The delta rows of window k
// take, in bucket order, the lowest slots that window k-1 does not occupy;
// rows window k-1 cached keep their slot and are not copied.  Occupancy is
// one byte per slot (plain byte stores, no atomics) after a 16-byte header
// holding the extent: one past the highest slot any window has used.  Free
// slots are taken lowest first, so every slot from the extent on is free and
// only the map below it is scanned.
//   k_inplace_prep  old slot of every bucket entry (-1: delta, -2: bad id),
//                   the delta count of every range of 64 entries and of
//                   every block (block b takes ranges b*R .. b*R+R-1),
//                   the per-owner delta counts and the free slots per chunk
//                   of the previous occupancy; clears the remap's stale
//                   entries and the new occupancy.
//   k_inplace_emit  the prefix of the block counts, and the ascending list
//                   of the first |delta| free slots; the blocks stride over
//                   the chunks below the previous extent and stop at the
//                   first chunk past those slots.
//   k_inplace_rows  remap, occupancy and the delta rows' copies (the
//                   requests); a tile's first delta rank is the prefix of
//                   its range's block plus that block's range counts before
//                   its range.
// ---------------------------------------------------------------------------
constexpr int kRange = kWave;          // bucket entries per delta count (one wave)
constexpr int kOccChunk = kBlock * 32; // slots per free-list block (one 32-slot group a thread)
constexpr int kPrepBlocks = 1024;      // most prep blocks (block counts a rank sums)
// Most free-list blocks (kEmitBlocksMax, or the tuning's emit_blocks).
// Blocks past the previous extent return at once; the cap keeps a large
// cache (4,224 chunks for the 34.6M slots of a Papers100M share) from
// launching thousands of them, and a lower one makes small caches exercise
// blocks that take several chunks.

struct InplaceWs {
  int32_t* old_slot;   // [cap]
  int32_t* dcnt;       // [prep blocks][P]
  int32_t* dr;         // [ranges]
  int32_t* btot;       // [prep blocks]
  int64_t* bpre;       // [prep blocks]
  int32_t* fcnt;       // [occupancy chunks]
  int32_t* freel;      // [cache_rows]
  int64_t* nfree;      // [1]
};

int inplace_prep_blocks(int64_t cap, int64_t cache_rows) {
  const int64_t need = std::max<int64_t>(cdiv(cap, kBlock), cdiv(cache_rows, kOccChunk));
  return (int)std::min<int64_t>(std::max<int64_t>(need, 1), kPrepBlocks);
}

size_t inplace_ws_layout(int64_t cap, int64_t cache_rows, int32_t P, char* base, InplaceWs* out) {
  const int64_t nr = std::max<int64_t>(cdiv(cap, kRange), 1);
  const int64_t nch = std::max<int64_t>(cdiv(cache_rows, kOccChunk), 1);
  const int gp = inplace_prep_blocks(cap, cache_rows);
  Carve cv{base, 0, ~(size_t)0};
  InplaceWs w;
  w.old_slot = cv.take<int32_t>((size_t)std::max<int64_t>(cap, 1));
  w.dcnt = cv.take<int32_t>((size_t)gp * (size_t)P);
  w.dr = cv.take<int32_t>((size_t)nr);
  w.btot = cv.take<int32_t>((size_t)align_up((size_t)gp, 4));   // read four at a time
  w.bpre = cv.take<int64_t>((size_t)gp);
  w.fcnt = cv.take<int32_t>((size_t)nch);
  w.freel = cv.take<int32_t>((size_t)std::max<int64_t>(cache_rows, 1));
  w.nfree = cv.take<int64_t>(1);
  if (out) *out = w;
  return align_up(cv.used, 256);
}

// Free-slot mask of the 32 slots q*32 .. q*32+31 (bit i = slot q*32+i is
// below cache_rows and its occupancy byte is 0).
// The 32 occupancy bytes of slots q*32 .. q*32+31, or zeros past cache_rows.
__device__ __forceinline__ void occ_words(const uint8_t* occ, int64_t q, int64_t cache_rows,
                                          u32x4* a, u32x4* b) {
  const u32x4 z = {0u, 0u, 0u, 0u};
  *a = z;
  *b = z;
  if (cache_rows - q * 32 <= 0) return;
  const u32x4* p = (const u32x4*)(occ + q * 32);
  *a = p[0];
  *b = p[1];
}

// Bit i set where byte i of (a, b) is 0 and i < lim.
__device__ __forceinline__ uint32_t zero_byte_bits(u32x4 a, u32x4 b, int64_t lim) {
  if (lim <= 0) return 0u;
  const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      m |= (((w[i] >> (8 * j)) & 0xFFu) == 0u ? 1u : 0u) << (4 * i + j);
  if (lim < 32) m &= (1u << lim) - 1u;
  return m;
}

__device__ __forceinline__ uint32_t free_mask(const uint8_t* occ, int64_t q, int64_t cache_rows) {
  u32x4 a, b;
  occ_words(occ, q, cache_rows, &a, &b);
  return zero_byte_bits(a, b, cache_rows - q * 32);
}

// Sum of v over a block of kBlock threads (every thread gets it).
__device__ __forceinline__ int64_t block_sum(int64_t v, int64_t* lds) {
  v = wave_sum(v);
  if (lane_id() == 0) lds[threadIdx.x / kWave] = v;
  __syncthreads();
  int64_t t = 0;
#pragma unroll
  for (int q = 0; q < kBlock / kWave; ++q) t += lds[q];
  __syncthreads();
  return t;
}

// Ranges per prep block for n bucket entries and gp prep blocks.
__device__ __forceinline__ int64_t ranges_per_block(int64_t n, int gp) {
  return cdiv_dev(cdiv_dev(n, kRange), gp);
}

constexpr int kOccHeader = 16;          // bytes before an occupancy map: int64 extent

__global__ void __launch_bounds__(kBlock) k_inplace_prep(
    const int32_t* bucket, const int64_t* owner_off, KPart part, StageArgs a, const int32_t* prev,
    int32_t* old_slot, int32_t* dcnt, int32_t* dr, int32_t* btot, const int32_t* clear,
    const int64_t* clear_count, int32_t* slot_of, const uint8_t* occ_prev, int32_t* fcnt,
    uint8_t* occ, int32_t* status) {
  // extent of the previous window's map (0 without one)
  const int64_t ext = occ_prev ? *(const int64_t*)occ_prev : 0;
  const uint8_t* map_prev = occ_prev ? occ_prev + kOccHeader : nullptr;
  uint8_t* map = occ + kOccHeader;
  __shared__ int32_t hist[GG_MAX_PARTS];
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  __shared__ int64_t lds[kBlock / kWave];
  __shared__ int32_t s_fresh;
  for (int t = threadIdx.x; t < GG_MAX_PARTS; t += blockDim.x) hist[t] = 0;
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  if (threadIdx.x == 0) s_fresh = 0;
  __syncthreads();
  const int64_t n = inplace_n(owner_off, part.P, a);
  const int64_t nr = cdiv_dev(n, kRange);
  const int64_t R = ranges_per_block(n, gridDim.x);
  const int64_t rend = (int64_t)(blockIdx.x + 1) * R < nr ? (int64_t)(blockIdx.x + 1) * R : nr;
  const int lane = lane_id();
  int32_t st = 0;
  for (int64_t r = (int64_t)blockIdx.x * R + threadIdx.x / kWave; r < rend; r += kBlock / kWave) {
    const int64_t s = r * kRange + lane;
    bool fresh = false;
    int32_t m = 0;
    if (s < n) {
      const int32_t u = bucket[s];
      int32_t old = -2;
      if (u >= 0 && (int64_t)u < part.N) {
        old = prev ? prev[u] : -1;
        if ((int64_t)old >= a.cache_rows) {
          st |= GG_DEV_BAD_ROW;
          old = -1;
        }
        if (old < 0) {
          old = -1;
          fresh = true;
          m = owner_of(part, s_start, u);
        }
      }
      old_slot[s] = old;
    }
    wave_hist_add(hist, fresh, m);
    const int32_t c = (int32_t)__popcll(__ballot(fresh));
    if (lane == 0) {
      dr[r] = c;
      if (c) atomicAdd(&s_fresh, c);
    }
  }
  if (clear) {
    const int64_t nc = clear_count[0];
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nc;
         i += (int64_t)gridDim.x * blockDim.x) {
      const int32_t u = clear[i];
      if (u >= 0 && (int64_t)u < part.N) slot_of[u] = -1;
    }
  }
  // free slots per chunk below the extent
  const int64_t lim = ext < a.cache_rows ? ext : a.cache_rows;
  const int64_t nch = cdiv_dev(lim, kOccChunk);
  for (int64_t c = blockIdx.x; c < nch; c += gridDim.x) {
    const int64_t g = c * kBlock + threadIdx.x;
    const int64_t f = block_sum(__popc(free_mask(map_prev, g, lim)), lds);
    if (threadIdx.x == 0) fcnt[c] = (int32_t)f;
  }
  // the new map below the extent this window can reach
  int64_t zl = lim + n;
  zl = zl < a.cache_rows ? zl : a.cache_rows;
  const u32x4 z = {0u, 0u, 0u, 0u};
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < cdiv_dev(zl, 32) * 2;
       q += (int64_t)gridDim.x * blockDim.x)
    ((u32x4*)map)[q] = z;
  if (blockIdx.x == 0 && threadIdx.x == 0) *(int64_t*)occ = lim;   // raised by the rows kernel
  if (st) set_status(status, st);
  __syncthreads();
  for (int m = threadIdx.x; m < part.P; m += blockDim.x) dcnt[(int64_t)blockIdx.x * part.P + m] = hist[m];
  if (threadIdx.x == 0) btot[blockIdx.x] = s_fresh;
}

// Block 0 writes the exclusive prefix of the prep blocks' delta counts
// (bpre) and the number of free slots below the previous extent.  Block b
// writes the free slots of occupancy chunk b (below the extent) at their
// place in the ascending free list, as far as the delta needs: staged in
// LDS, then stored contiguously; other blocks return at once.
__global__ void __launch_bounds__(kBlock) k_inplace_emit(const uint8_t* occ_prev,
                                                         const int32_t* fcnt,
                                                         const int32_t* btot, int32_t gp,
                                                         int64_t* bpre, int32_t* freel,
                                                         int64_t* nfree, StageArgs a) {
  __shared__ int64_t lds[kBlock / kWave];
  constexpr int PT = kPrepBlocks / kBlock;     // block counts per thread
  // Two dependent rounds of loads: the extent with the block counts, then
  // the chunk counts with the occupancy bytes of the block's first chunk.
  static_assert(PT == 4, "one 16-byte load of block counts per thread");
  const int b = blockIdx.x;
  const int64_t ext = occ_prev ? *(const int64_t*)occ_prev : 0;
  const int i0 = threadIdx.x * PT;
  u32x4 bv = {0u, 0u, 0u, 0u};
  if (i0 < gp) bv = *(const u32x4*)(btot + i0);   // the workspace pads btot to a multiple of 4
  const int32_t bt[PT] = {(int32_t)bv.x, i0 + 1 < gp ? (int32_t)bv.y : 0,
                          i0 + 2 < gp ? (int32_t)bv.z : 0, i0 + 3 < gp ? (int32_t)bv.w : 0};
  const int64_t v = (int64_t)bt[0] + bt[1] + bt[2] + bt[3];
  const int64_t lim = ext < a.cache_rows ? ext : a.cache_rows;
  const int64_t nch = cdiv_dev(lim, kOccChunk);
  if (b > 0 && b >= nch) return;
  const uint8_t* map_prev = occ_prev + kOccHeader;
  const int64_t q0 = (int64_t)b * kBlock + threadIdx.x;
  u32x4 o0, o1;
  occ_words(map_prev, q0, b < nch ? lim : 0, &o0, &o1);
  int64_t w = 0, all = 0;
  for (int64_t c = threadIdx.x; c < nch; c += blockDim.x) {
    const int64_t x = fcnt[c];
    all += x;
    if (c < b) w += x;
  }
  uint32_t f = zero_byte_bits(o0, o1, lim - q0 * 32);
  int64_t need;
  int64_t run = block_excl_scan<kBlock>(v, lds, &need);
  if (b == 0) {
#pragma unroll
    for (int q = 0; q < PT; ++q) {
      const int i = threadIdx.x * PT + q;
      if (i < gp) bpre[i] = run;
      run += bt[q];
    }
    all = block_sum(all, lds);
    if (threadIdx.x == 0) *nfree = all;
  }
  for (int64_t ch = b; ch < nch; ch += gridDim.x) {
    if (ch != b) {
      w = 0;
      for (int64_t c = threadIdx.x; c < ch; c += blockDim.x) w += fcnt[c];
      f = free_mask(map_prev, ch * kBlock + threadIdx.x, lim);
    }
    const int64_t before = block_sum(w, lds);
    if (before >= need) return;    // the delta's slots lie before this chunk and the later ones
    // Every thread writes its own free slots at its place in the list.  A
    // version that staged the chunk's list in 32 KB of LDS took ~200 us
    // beside the gather of a Papers100M share against 5-14 us alone (a
    // kernel with little LDS, the prep, ran equally fast in both); without
    // the LDS it takes 15-20 us there.
    const int64_t g = ch * kBlock + threadIdx.x;
    int64_t tot;
    int64_t pos = before + block_excl_scan<kBlock>((int64_t)__popc(f), lds, &tot);
    for (; f && pos < need; f &= f - 1u) freel[pos++] = (int32_t)(g * 32 + (__ffs(f) - 1));
  }
}

template <int VB, bool NT>
__global__ void __launch_bounds__(kBlock) k_inplace_rows(
    const int32_t* bucket, const int64_t* owner_off, KPart part, KFeat feat, StageArgs a,
    char* cache, int32_t* slot_of, const int32_t* old_slot, const int32_t* dr,
    const int32_t* btot, const int64_t* bpre, int32_t gp, const int32_t* freel,
    const int64_t* nfree_p, const uint8_t* occ_prev, uint8_t* occ, StageStatsArgs sa,
    int32_t* status) {
  if (blockIdx.x == 0) stage_stats(owner_off, part, a, feat.row_bytes, sa, status);
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  __syncthreads();
  const int64_t n = inplace_n(owner_off, part.P, a);
  const int64_t R = ranges_per_block(n, gp);
  // delta rank j takes free-list entry j below the previous extent, and
  // slot ext + (j - nfree) above it
  const int64_t ext0 = occ_prev ? *(const int64_t*)occ_prev : 0;
  const int64_t ext = ext0 < a.cache_rows ? ext0 : a.cache_rows;
  const int64_t nfree = *nfree_p;
  const int64_t need = bpre[gp - 1] + btot[gp - 1];
  uint8_t* map = occ + kOccHeader;
  const int64_t ntiles = (n + a.tile - 1) / a.tile;
  const int lane = lane_id();
  int32_t st = 0;
  for (int64_t tile = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; tile < ntiles;
       tile += (int64_t)gridDim.x * (kBlock / kWave)) {
    const int64_t s0 = tile * a.tile;
    const int64_t s = s0 + lane;
    const bool live = lane < a.tile && s < n;
    const int32_t old = live ? old_slot[s] : -2;
    const int32_t u = live ? bucket[s] : -1;
    // delta rank of the tile's first entry: the counts of the prep blocks
    // before its range's block, of that block's ranges before its range,
    // and of the range's entries before the tile
    const int64_t rg = s0 / kRange;
    const int64_t pb = rg / R;
    int64_t j = 0;
    for (int64_t q = pb * R + lane; q < rg; q += kWave) j += dr[q];
    const int64_t r0 = rg * kRange;
    if (r0 < s0) {
      const int64_t p = r0 + lane;
      j += (p < s0 && old_slot[p] == -1) ? 1 : 0;
    }
    j = bpre[pb] + wave_sum(j);
    const uint64_t fm = __ballot(old == -1);
    long long src = 0, dst = 0;
    if (live) {
      if (old == -2) {
        st |= GG_DEV_BAD_ID;
      } else if (old >= 0) {
        slot_of[u] = old;                                    // retained in place
        map[old] = 1;
      } else {
        const int64_t jj = j + lanes_below(fm);
        const int64_t slot = jj < nfree ? (int64_t)freel[jj] : ext + (jj - nfree);
        if (jj == need - 1) {
          // The last delta rank raises the extent past every slot the delta
          // took from the extent on; when the cache runs out, those are all
          // the slots up to its end (the ranks beyond stay uncached).
          const int64_t e = slot + 1 < a.cache_rows ? slot + 1 : a.cache_rows;
          if (e > ext) *(int64_t*)occ = e;
        }
        if (slot < 0 || slot >= a.cache_rows) {
          st |= GG_DEV_CAPACITY;
        } else {
          const int32_t m = owner_of(part, s_start, u);
          const int64_t r = row_of(part, s_start, u, m);
          if (r >= feat.rows[m]) {
            st |= GG_DEV_BAD_ROW;
          } else {
            src = (long long)(feat.shard[m] + r * feat.stride[m]);   // requested from owner m
            dst = (long long)(cache + slot * a.cache_stride);
            slot_of[u] = (int32_t)slot;
            map[slot] = 1;
          }
        }
      }
    }
    // the tile's requested rows, packed to the front of the wave
    const uint64_t cm = __ballot(src != 0);
    const int nc = (int)__popcll(cm);
    if (nc) {
      const int from = lane < nc ? nth_set_lane(cm, lane) : 0;
      const long long cs = __shfl(src, from, kWave), cd = __shfl(dst, from, kWave);
      wave_copy_rows_to<VB, NT>(lane < nc ? (const char*)cs : nullptr,
                                lane < nc ? (char*)cd : nullptr, nc, a.geom);
    }
  }
  if (st) set_status(status, st);
}

}  // namespace
}  // namespace gg

using namespace gg;

extern "C" size_t gg_ws_stage(int64_t cap, int32_t num_parts) {
  return align_up((size_t)stage_delta_blocks(cap) * (size_t)num_parts * sizeof(int32_t), 256) +
         align_up((size_t)std::max<int64_t>(cap, 1) * sizeof(int32_t), 256);
}

extern "C" int gg_stage_bulk(const int32_t* bucket_ids_d, const int64_t* owner_off_d, int64_t cap,
                             const gg_part_t* part, const gg_feat_t* feat, void* cache_d,
                             int64_t cache_stride, int64_t cache_rows, int32_t* slot_of_d,
                             const int32_t* clear_ids_d, const int64_t* clear_count_d,
                             const void* src_cache_d, const int32_t* src_slot_of_d,
                             gg_stage_stats_t* stats_d, const gg_tuning_t* tuning,
                             int32_t* status_d, void* ws, size_t ws_bytes, hipStream_t stream) {
  GG_REQUIRE(owner_off_d && slot_of_d && stats_d && status_d, "NULL argument");
  Tune tune;
  if (resolve_tuning(tuning, &tune) != GG_OK) return GG_ERR_ARG;
  GG_REQUIRE(cap >= 0 && cap < (1LL << 31) && cache_rows >= 0, "bad capacity");
  GG_REQUIRE(cap == 0 || bucket_ids_d, "bucket ids are NULL");
  GG_REQUIRE(cache_rows == 0 || cache_d, "cache is NULL");
  GG_REQUIRE((clear_ids_d == nullptr) == (clear_count_d == nullptr),
             "clear_ids and clear_count must both be given or both be NULL");
  GG_REQUIRE(src_cache_d == nullptr || src_slot_of_d != nullptr,
             "a source cache needs its remap src_slot_of");
  GG_REQUIRE(src_cache_d == nullptr || src_cache_d != cache_d,
             "the source cache must be a different buffer from the cache being staged");
  KPart kp;
  int rc = pack_part(part, &kp);
  if (rc != GG_OK) return rc;
  KFeat kf;
  rc = pack_feat(feat, part, &kf);
  if (rc != GG_OK) return rc;
  GG_REQUIRE(cache_stride >= kf.row_bytes && cache_stride % 4 == 0, "cache_stride %lld invalid",
             (long long)cache_stride);
  bool v16 = aligned16(cache_d) && cache_stride % 16 == 0 &&
             (src_cache_d == nullptr || aligned16(src_cache_d));
  for (int m = 0; m < kf.P; ++m)
    if (kf.rows[m] > 0) v16 = v16 && aligned16(kf.shard[m]) && kf.stride[m] % 16 == 0;
  StageArgs a;
  a.cap = cap;
  a.cache_rows = cache_rows;
  a.cache_stride = cache_stride;
  a.tile = copy_tile(tune, kf.row_bytes, 32768);
  a.pad_ = 0;
  a.geom = copy_geom(kf.row_bytes, v16 ? 16 : 4);

  const int gridd = stage_delta_blocks(cap);
  GG_REQUIRE(ws && ws_bytes >= gg_ws_stage(cap, kp.P), "workspace of %zu bytes < %zu", ws_bytes,
             gg_ws_stage(cap, kp.P));
  int32_t* dcnt = (int32_t*)ws;
  int32_t* old_slot =
      (int32_t*)((char*)ws + align_up((size_t)gridd * (size_t)kp.P * sizeof(int32_t), 256));
  const int32_t* before = src_slot_of_d ? src_slot_of_d : slot_of_d;
  // The remap is cleared in the same launch when the old slots are read
  // from another remap; reading and clearing one remap need two launches.
  const bool fuse_clear = clear_ids_d && before != slot_of_d;
  hipLaunchKernelGGL(k_stage_delta, dim3(gridd), dim3(kBlock), 0, stream, bucket_ids_d, owner_off_d,
                     kp, a, before, old_slot, dcnt, fuse_clear ? clear_ids_d : nullptr,
                     clear_count_d, slot_of_d);
  GG_LAUNCH_CHECK("k_stage_delta");
  if (clear_ids_d && !fuse_clear) {
    hipLaunchKernelGGL(k_slot_reset, dim3(2048), dim3(kBlock), 0, stream, clear_ids_d, clear_count_d,
                       kp.N, slot_of_d);
    GG_LAUNCH_CHECK("k_slot_reset");
  }
  const int64_t ntiles = cdiv(std::min(cap, cache_rows), a.tile);
  // Rows read over PCIe need few waves in flight to keep the link busy; a
  // full grid would hold every CU while it waits and starve kernels on
  // other streams (the next window's sampling), so cap it then.
  const int64_t gmax = host_shards(kf) > 0 ? tune.stage_host_blocks : tune.stage_blocks;
  const int grid = (int)std::min<int64_t>(std::max<int64_t>(cdiv(ntiles, kBlock / kWave), 1), gmax);
  StageStatsArgs sa;
  sa.prev_count = clear_count_d;
  sa.dcnt = dcnt;
  sa.stats = stats_d;
  sa.nfree = nullptr;
  sa.occ_prev = nullptr;
  sa.nblk_delta = gridd;
  sa.has_src = src_cache_d ? 1 : 0;
  if (v16)
    launch_stage_rows<16>(grid, stream, bucket_ids_d, owner_off_d, kp, kf, a, (char*)cache_d,
                          slot_of_d, (const char*)src_cache_d, old_slot, sa, status_d);
  else
    launch_stage_rows<4>(grid, stream, bucket_ids_d, owner_off_d, kp, kf, a, (char*)cache_d,
                         slot_of_d, (const char*)src_cache_d, old_slot, sa, status_d);
  GG_LAUNCH_CHECK("k_stage_rows");
  return GG_OK;
}

extern "C" size_t gg_ws_stage_inplace(int64_t cap, int64_t cache_rows, int32_t num_parts) {
  return inplace_ws_layout(std::max<int64_t>(cap, 0), std::max<int64_t>(cache_rows, 0),
                           std::max(num_parts, 1), nullptr, nullptr);
}

extern "C" int gg_stage_inplace(const int32_t* bucket_ids_d, const int64_t* owner_off_d,
                                int64_t cap, const gg_part_t* part, const gg_feat_t* feat,
                                void* cache_d, int64_t cache_stride, int64_t cache_rows,
                                int32_t* slot_of_d, const int32_t* clear_ids_d,
                                const int64_t* clear_count_d, const int32_t* prev_slot_of_d,
                                const uint8_t* occ_prev_d, uint8_t* occ_d,
                                gg_stage_stats_t* stats_d, const gg_tuning_t* tuning,
                                int32_t* status_d, void* ws, size_t ws_bytes,
                                hipStream_t stream) {
  GG_REQUIRE(owner_off_d && slot_of_d && occ_d && stats_d && status_d, "NULL argument");
  Tune tune;
  if (resolve_tuning(tuning, &tune) != GG_OK) return GG_ERR_ARG;
  GG_REQUIRE(cap >= 0 && cap < (1LL << 31), "bad capacity");
  GG_REQUIRE(cache_rows >= 0 && cache_rows < (1LL << 31), "bad cache_rows");
  GG_REQUIRE(cap == 0 || bucket_ids_d, "bucket ids are NULL");
  GG_REQUIRE(cache_rows == 0 || cache_d, "cache is NULL");
  GG_REQUIRE((clear_ids_d == nullptr) == (clear_count_d == nullptr),
             "clear_ids and clear_count must both be given or both be NULL");
  GG_REQUIRE((prev_slot_of_d == nullptr) == (occ_prev_d == nullptr),
             "prev_slot_of and occ_prev must both be given or both be NULL");
  GG_REQUIRE(prev_slot_of_d != slot_of_d, "the previous remap must be another buffer");
  GG_REQUIRE(occ_prev_d != occ_d, "the previous occupancy must be another buffer");
  KPart kp;
  int rc = pack_part(part, &kp);
  if (rc != GG_OK) return rc;
  KFeat kf;
  rc = pack_feat(feat, part, &kf);
  if (rc != GG_OK) return rc;
  GG_REQUIRE(cache_stride >= kf.row_bytes && cache_stride % 4 == 0, "cache_stride %lld invalid",
             (long long)cache_stride);
  InplaceWs w;
  const size_t need_ws = inplace_ws_layout(cap, cache_rows, kp.P, (char*)ws, &w);
  GG_REQUIRE(ws && ws_bytes >= need_ws, "workspace of %zu bytes < %zu", ws_bytes, need_ws);
  bool v16 = aligned16(cache_d) && cache_stride % 16 == 0;
  for (int m = 0; m < kf.P; ++m)
    if (kf.rows[m] > 0) v16 = v16 && aligned16(kf.shard[m]) && kf.stride[m] % 16 == 0;
  StageArgs a;
  a.cap = cap;
  a.cache_rows = cache_rows;
  a.cache_stride = cache_stride;
  a.tile = copy_tile(tune, kf.row_bytes, 32768);
  a.pad_ = 0;
  a.geom = copy_geom(kf.row_bytes, v16 ? 16 : 4);
  GG_REQUIRE(((uintptr_t)occ_d & 15u) == 0 && ((uintptr_t)occ_prev_d & 15u) == 0,
             "occupancy maps must be 16-byte aligned");
  const int gridp = inplace_prep_blocks(cap, cache_rows);
  hipLaunchKernelGGL(k_inplace_prep, dim3(gridp), dim3(kBlock), 0, stream, bucket_ids_d,
                     owner_off_d, kp, a, prev_slot_of_d, w.old_slot, w.dcnt, w.dr, w.btot,
                     clear_ids_d, clear_count_d, slot_of_d, occ_prev_d, w.fcnt, occ_d, status_d);
  GG_LAUNCH_CHECK("k_inplace_prep");
  // the extent is known on the device only: blocks past its chunks return
  // at once, and the grid is capped so that they stay few
  const int64_t nch =
      occ_prev_d ? std::min<int64_t>(cdiv(cache_rows, kOccChunk), tune.emit_blocks) : 0;
  hipLaunchKernelGGL(k_inplace_emit, dim3((unsigned)std::max<int64_t>(nch, 1)), dim3(kBlock), 0, stream, occ_prev_d,
                     w.fcnt, w.btot, gridp, w.bpre, w.freel, w.nfree, a);
  GG_LAUNCH_CHECK("k_inplace_emit");
  const int64_t ntiles = cdiv(std::min(cap, cache_rows), a.tile);
  const int64_t gmax = host_shards(kf) > 0 ? tune.stage_host_blocks : tune.stage_blocks;
  const int grid = (int)std::min<int64_t>(std::max<int64_t>(cdiv(ntiles, kBlock / kWave), 1), gmax);
  StageStatsArgs sa;
  sa.prev_count = clear_count_d;
  sa.dcnt = w.dcnt;
  sa.stats = stats_d;
  sa.nfree = w.nfree;
  sa.occ_prev = occ_prev_d;
  sa.nblk_delta = gridp;
  sa.has_src = 1;
  // Cache rows are stored with ordinary stores: the gathers read them next.
  if (v16)
    hipLaunchKernelGGL((k_inplace_rows<16, false>), dim3(grid), dim3(kBlock), 0, stream,
                       bucket_ids_d, owner_off_d, kp, kf, a, (char*)cache_d, slot_of_d,
                       w.old_slot, w.dr, w.btot, w.bpre, gridp, w.freel, w.nfree, occ_prev_d,
                       occ_d, sa, status_d);
  else
    hipLaunchKernelGGL((k_inplace_rows<4, false>), dim3(grid), dim3(kBlock), 0, stream,
                       bucket_ids_d, owner_off_d, kp, kf, a, (char*)cache_d, slot_of_d,
                       w.old_slot, w.dr, w.btot, w.bpre, gridp, w.freel, w.nfree, occ_prev_d,
                       occ_d, sa, status_d);
  GG_LAUNCH_CHECK("k_inplace_rows");
  return GG_OK;
}
