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
  const int64_t n = stage_n(owner_off, part.P, a);
  __shared__ int64_t s_req[GG_MAX_PARTS], s_rows[GG_MAX_PARTS];
  if (threadIdx.x < GG_MAX_PARTS) {
    const int m = threadIdx.x;
    int64_t rows = 0;
    if (m < part.P) {
      int64_t lo = owner_off[m], hi = owner_off[m + 1];
      lo = lo < n ? lo : n;
      hi = hi < n ? hi : n;
      rows = hi > lo ? hi - lo : 0;
      if (has_src) rows = s_delta[m];    // only the delta is requested
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
    int64_t req = 0, fetched = 0;
    for (int m = 0; m < part.P; ++m) {
      req += s_req[m];
      fetched += s_rows[m];
    }
    stats->rows_total = n;
    stats->requests_total = req;
    stats->invalidated = prev_count ? prev_count[0] : 0;
    stats->retained = has_src ? n - fetched : 0;
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

template <int VB>
void launch_stage_rows(bool nt, int grid, hipStream_t stream, const int32_t* bucket,
                       const int64_t* owner_off, const KPart& kp, const KFeat& kf,
                       const StageArgs& a, char* cache, int32_t* slot_of, const char* src_cache,
                       const int32_t* old_slot, const StageStatsArgs& sa, int32_t* status) {
  if (nt)
    hipLaunchKernelGGL((k_stage_rows<VB, true>), dim3(grid), dim3(kBlock), 0, stream, bucket,
                       owner_off, kp, kf, a, cache, slot_of, src_cache, old_slot, sa, status);
  else
    hipLaunchKernelGGL((k_stage_rows<VB, false>), dim3(grid), dim3(kBlock), 0, stream, bucket,
                       owner_off, kp, kf, a, cache, slot_of, src_cache, old_slot, sa, status);
}

int stage_delta_blocks(int64_t cap) {
  return (int)std::min<int64_t>(std::max<int64_t>(cdiv(cap, kBlock), 1), 1024);
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
                             gg_stage_stats_t* stats_d, int32_t* status_d, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  GG_REQUIRE(owner_off_d && slot_of_d && stats_d && status_d, "NULL argument");
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
  a.tile = copy_tile(kf.row_bytes, 32768);
  a.pad_ = 0;
  a.geom = copy_geom(kf.row_bytes, v16 ? 16 : 4);
  static const bool nt = env_flag("GG_NT_STAGE", false);

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
  static const int host_cap = env_int("GG_STAGE_HOST_BLOCKS", 128);
  static const int hbm_cap = env_int("GG_STAGE_BLOCKS", 16384);
  int64_t gmax = hbm_cap;
  if (host_cap > 0 && host_shards(kf) > 0) gmax = host_cap;
  const int grid = (int)std::min<int64_t>(std::max<int64_t>(cdiv(ntiles, kBlock / kWave), 1), gmax);
  StageStatsArgs sa;
  sa.prev_count = clear_count_d;
  sa.dcnt = dcnt;
  sa.stats = stats_d;
  sa.nblk_delta = gridd;
  sa.has_src = src_cache_d ? 1 : 0;
  if (v16)
    launch_stage_rows<16>(nt, grid, stream, bucket_ids_d, owner_off_d, kp, kf, a, (char*)cache_d,
                          slot_of_d, (const char*)src_cache_d, old_slot, sa, status_d);
  else
    launch_stage_rows<4>(nt, grid, stream, bucket_ids_d, owner_off_d, kp, kf, a, (char*)cache_d,
                         slot_of_d, (const char*)src_cache_d, old_slot, sa, status_d);
  GG_LAUNCH_CHECK("k_stage_rows");
  return GG_OK;
}
