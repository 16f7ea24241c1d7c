// gg_gather_batch: per-batch feature assembly through the ID-to-slot remap,
// with the on-demand miss path.
//
// k_gather_rows: one wavefront per 64 consecutive output rows.  Each lane
// resolves its row (local shard, cache slot, or miss) and the wave copies
// all resolved rows with the row copy engine, writing out rows in order.
// Misses are compacted per block into the workspace together with per-block
// counts (no atomics on global memory, nothing to clear beforehand).
// k_gather_finish: serves the misses owner by owner from the owners' shards
// and reduces the per-block counts into the batch statistics.
#include <stdlib.h>
#include <string.h>

#include "gg_host.hpp"

namespace gg {
namespace {

constexpr int kRowsPerBlock = kBlock;  // 4 waves x 64 rows
constexpr int kFinishGrid = 512;

struct GatherArgs {
  int64_t n_cap;
  int64_t cache_stride;
  int64_t cache_rows;
  int64_t out_stride;
  int32_t nblk;
  int32_t nstat;   // ints of per-block statistics: 2 + P
  CopyGeom geom;
};

__device__ __forceinline__ int64_t gather_n(const int64_t* bounds, const GatherArgs& a) {
  const int64_t n = bounds[1] - bounds[0];
  return n < 0 ? 0 : (n < a.n_cap ? n : a.n_cap);
}

template <int VB, bool NT>
__global__ void __launch_bounds__(kBlock) k_gather_rows(const int32_t* in_ids, const int64_t* bounds,
                                                        KPart part, KFeat feat, GatherArgs a,
                                                        const char* cache, const int32_t* slot_of,
                                                        char* out, int32_t* blk_stat,
                                                        int32_t* miss_pos, int32_t* miss_id,
                                                        int32_t* status) {
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  __shared__ int32_t s_cnt[2 + GG_MAX_PARTS];  // local, hits, misses per owner
  __shared__ int32_t s_nmiss;
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  for (int t = threadIdx.x; t < 2 + GG_MAX_PARTS; t += blockDim.x) s_cnt[t] = 0;
  if (threadIdx.x == 0) s_nmiss = 0;
  __syncthreads();
  const int64_t n = gather_n(bounds, a);
  const int64_t begin = bounds[0];
  const int lane = lane_id();
  const int64_t r0 = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x / kWave) * kWave;
  const int64_t i = r0 + lane;
  const char* src = nullptr;
  bool miss = false, is_local = false, is_hit = false;
  int32_t u = -1, m = -1;
  int32_t st = 0;
  if (i < n) {
    u = in_ids[begin + i];
    if (u < 0 || (int64_t)u >= part.N) {
      st |= GG_DEV_BAD_ID;
    } else {
      m = owner_of(part, s_start, u);
      if (m == part.local) {
        const int64_t r = row_of(part, s_start, u, m);
        if (r < feat.rows[m]) {
          src = feat.shard[m] + r * feat.stride[m];
          is_local = true;
        } else {
          st |= GG_DEV_BAD_ROW;
        }
      } else {
        const int32_t s = slot_of[u];
        if (s >= 0 && (int64_t)s < a.cache_rows) {
          src = cache + (int64_t)s * a.cache_stride;
          is_hit = true;
        } else {
          if (s >= 0) st |= GG_DEV_BAD_ROW;
          miss = true;
        }
      }
    }
  }
  // Wave counts by ballot; misses per owner with one ballot per owner seen.
  const uint64_t ml = __ballot(is_local), mh = __ballot(is_hit), mm = __ballot(miss);
  if (lane == 0) {
    if (ml) atomicAdd(&s_cnt[0], (int32_t)__popcll(ml));
    if (mh) atomicAdd(&s_cnt[1], (int32_t)__popcll(mh));
  }
  for (uint64_t act = mm; act;) {
    const int leader = __ffsll((unsigned long long)act) - 1;
    const int32_t ol = __shfl(m, leader, kWave);
    const uint64_t sel = __ballot(miss && m == ol);
    if (lane == leader) atomicAdd(&s_cnt[2 + ol], (int32_t)__popcll(sel));
    act &= ~sel;
  }
  // Compact this wave's misses into the block's region of the workspace.
  if (mm) {
    int32_t wbase = 0;
    if (lane == 0) wbase = atomicAdd(&s_nmiss, (int32_t)__popcll(mm));
    wbase = __shfl(wbase, 0, kWave);
    if (miss) {
      const int64_t q = (int64_t)blockIdx.x * kRowsPerBlock + wbase + lanes_below(mm);
      miss_pos[q] = (int32_t)i;
      miss_id[q] = u;
    }
  }
  const int64_t left = n - r0;
  const int nrows = left <= 0 ? 0 : (left < kWave ? (int)left : kWave);
  if (nrows > 0) wave_copy_rows<VB, NT>(src, out + r0 * a.out_stride, a.out_stride, nrows, a.geom);
  if (st) set_status(status, st);
  __syncthreads();
  for (int t = threadIdx.x; t < a.nstat; t += blockDim.x)
    blk_stat[(int64_t)blockIdx.x * a.nstat + t] = s_cnt[t];
}

template <int VB, bool NT>
__global__ void __launch_bounds__(kBlock) k_gather_finish(const int64_t* bounds, KPart part, KFeat feat,
                                                          GatherArgs a, const int32_t* blk_stat,
                                                          const int32_t* miss_pos,
                                                          const int32_t* miss_id, char* out,
                                                          gg_gather_stats_t* stats,
                                                          int32_t* status) {
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  __shared__ unsigned long long s_sum[2 + GG_MAX_PARTS];
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  for (int t = threadIdx.x; t < 2 + GG_MAX_PARTS; t += blockDim.x) s_sum[t] = 0;
  __syncthreads();
  const int P = part.P;
  const int wid = threadIdx.x / kWave, lane = lane_id();
  int32_t st = 0;
  // Misses of gather block g, served from the owners' shards.
  for (int64_t g = blockIdx.x; g < a.nblk; g += gridDim.x) {
    int32_t nm = 0;
    for (int mm = 0; mm < P; ++mm) nm += blk_stat[g * a.nstat + 2 + mm];
    for (int32_t j0 = wid * kWave; j0 < nm; j0 += kBlock) {
      const int32_t j = j0 + lane;
      const char* src = nullptr;
      char* dst = nullptr;
      if (j < nm) {
        const int64_t q = g * kRowsPerBlock + j;
        const int32_t u = miss_id[q];
        const int32_t m = owner_of(part, s_start, u);
        const int64_t r = row_of(part, s_start, u, m);
        if (r < feat.rows[m]) {
          src = feat.shard[m] + r * feat.stride[m];
          dst = out + (int64_t)miss_pos[q] * a.out_stride;
        } else {
          st |= GG_DEV_BAD_ROW;
        }
      }
      const int nr = nm - j0 < kWave ? nm - j0 : kWave;
      wave_copy_rows_scatter<VB, NT>(src, dst, nr, a.geom);
    }
  }
  if (st) set_status(status, st);
  if (blockIdx.x != 0) return;
  // Block 0: batch statistics.
  for (int64_t e = threadIdx.x; e < (int64_t)a.nblk * a.nstat; e += blockDim.x) {
    const int32_t v = blk_stat[e];
    if (v) atomicAdd(&s_sum[e % a.nstat], (unsigned long long)v);
  }
  __syncthreads();
  if (threadIdx.x < GG_MAX_PARTS) {
    const int m = threadIdx.x;
    const int64_t rows = m < P ? (int64_t)s_sum[2 + m] : 0;
    stats->miss_rows[m] = rows;
    stats->miss_requests[m] = rows > 0 ? 1 : 0;
  }
  if (threadIdx.x == 0) {
    int64_t misses = 0;
    for (int m = 0; m < P; ++m) misses += (int64_t)s_sum[2 + m];
    stats->rows = gather_n(bounds, a);
    stats->local = (int64_t)s_sum[0];
    stats->hits = (int64_t)s_sum[1];
    stats->misses = misses;
  }
}

bool env_flag(const char* name, bool dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  return strcmp(v, "0") != 0;
}

template <int VB, bool NT>
void launch_gather(hipStream_t stream, const int32_t* in_ids, const int64_t* bounds, const KPart& kp,
                   const KFeat& kf, const GatherArgs& a, const char* cache, const int32_t* slot_of,
                   char* out, int32_t* blk_stat, int32_t* miss_pos, int32_t* miss_id,
                   gg_gather_stats_t* stats, int32_t* status) {
  hipLaunchKernelGGL((k_gather_rows<VB, NT>), dim3(a.nblk), dim3(kBlock), 0, stream, in_ids, bounds,
                     kp, kf, a, cache, slot_of, out, blk_stat, miss_pos, miss_id, status);
  hipLaunchKernelGGL((k_gather_finish<VB, NT>), dim3(std::min(a.nblk, kFinishGrid)), dim3(kBlock), 0,
                     stream, bounds, kp, kf, a, blk_stat, miss_pos, miss_id, out, stats, status);
}

struct GatherWs {
  int32_t* blk_stat;
  int32_t* miss_pos;
  int32_t* miss_id;
};

size_t gather_ws_layout(int64_t n_cap, int32_t P, char* base, GatherWs* out) {
  const int64_t nblk = std::max<int64_t>(1, cdiv(n_cap, kRowsPerBlock));
  Carve cv{base, 0, ~(size_t)0};
  GatherWs g;
  g.blk_stat = cv.take<int32_t>((size_t)(nblk * (2 + P)));
  g.miss_pos = cv.take<int32_t>((size_t)(nblk * kRowsPerBlock));
  g.miss_id = cv.take<int32_t>((size_t)(nblk * kRowsPerBlock));
  if (out) *out = g;
  return align_up(cv.used, 256);
}

}  // namespace
}  // namespace gg

using namespace gg;

extern "C" size_t gg_ws_gather(int64_t n_cap, int32_t num_parts) {
  return gather_ws_layout(n_cap, num_parts, nullptr, nullptr);
}

extern "C" int gg_gather_batch(const int32_t* in_ids_d, const int64_t* bounds_d, int64_t n_cap,
                               const gg_part_t* part, const gg_feat_t* feat, const void* cache_d,
                               int64_t cache_stride, int64_t cache_rows, const int32_t* slot_of_d,
                               void* out_d, int64_t out_stride, gg_gather_stats_t* stats_d,
                               int32_t* status_d, void* ws, size_t ws_bytes, hipStream_t stream) {
  GG_REQUIRE(bounds_d && slot_of_d && stats_d && status_d, "NULL argument");
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
  GatherWs gw;
  const size_t need_ws = gather_ws_layout(n_cap, kp.P, (char*)ws, &gw);
  GG_REQUIRE(ws && ws_bytes >= need_ws, "workspace of %zu bytes < %zu", ws_bytes, need_ws);
  bool v16 = aligned16(out_d) && out_stride % 16 == 0 &&
             (cache_rows == 0 || (aligned16(cache_d) && cache_stride % 16 == 0));
  for (int m = 0; m < kf.P; ++m)
    if (kf.rows[m] > 0) v16 = v16 && aligned16(kf.shard[m]) && kf.stride[m] % 16 == 0;
  GatherArgs a;
  a.n_cap = n_cap;
  a.cache_stride = cache_stride;
  a.cache_rows = cache_rows;
  a.out_stride = out_stride;
  a.nblk = (int32_t)std::max<int64_t>(1, cdiv(n_cap, kRowsPerBlock));
  a.nstat = 2 + kp.P;
  a.geom = copy_geom(kf.row_bytes, v16 ? 16 : 4);
  static const bool nt = env_flag("GG_NT_GATHER", true);
  const char* cache = (const char*)cache_d;
  char* out = (char*)out_d;
  if (v16) {
    if (nt)
      launch_gather<16, true>(stream, in_ids_d, bounds_d, kp, kf, a, cache, slot_of_d, out,
                              gw.blk_stat, gw.miss_pos, gw.miss_id, stats_d, status_d);
    else
      launch_gather<16, false>(stream, in_ids_d, bounds_d, kp, kf, a, cache, slot_of_d, out,
                               gw.blk_stat, gw.miss_pos, gw.miss_id, stats_d, status_d);
  } else {
    if (nt)
      launch_gather<4, true>(stream, in_ids_d, bounds_d, kp, kf, a, cache, slot_of_d, out,
                             gw.blk_stat, gw.miss_pos, gw.miss_id, stats_d, status_d);
    else
      launch_gather<4, false>(stream, in_ids_d, bounds_d, kp, kf, a, cache, slot_of_d, out,
                              gw.blk_stat, gw.miss_pos, gw.miss_id, stats_d, status_d);
  }
  GG_LAUNCH_CHECK("k_gather_rows/k_gather_finish");
  return GG_OK;
}
