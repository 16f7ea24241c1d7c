// gg_bucket_by_owner: stable partition of the hot set by partition owner.
//
// Three passes over the ids: per-block owner histograms, one exclusive scan
// over the (owner, block) counts in owner-major order, and a scatter in
// which every wavefront ranks its 64 ids among equal owners with ballots
// (one ballot per distinct owner present in the wave), so order is kept
// inside each owner.
//
// Range partitions first try the identity: when owners never decrease along
// the input (the ascending hot set always satisfies this), the input is
// already owner-major.  k_bucket_range copies it, writes owner_off from the
// owner changes and records per block whether its ids were in owner order;
// the general passes then run only if some block saw a decrease.  A caller
// that knows its input is in owner order (GG_BUCKET_OWNER_ORDERED) skips the
// general passes' launches altogether; a block that finds the order broken
// then raises GG_DEV_ORDER.
#include "gg_host.hpp"

namespace gg {
namespace {

constexpr int kIdsPerBlock = 4096;             // 16 per thread
constexpr int kIdsPerWave = kIdsPerBlock / 4;  // 1024 = 16 groups of 64

__device__ __forceinline__ int64_t bucket_n(const int64_t* hot_count, int64_t cap) {
  const int64_t n = hot_count[0];
  return n < cap ? n : cap;
}

// Owner-order check and identity bucketing for range partitions.  A block
// covers kRangeIds consecutive ids, four per thread, all loads issued
// before any store.  It copies them, writes the owner_off entries of every
// owner change it sees, and writes ok[blockIdx.x] = 1 when its ids were
// valid and in owner order.
constexpr int kRangePer = 4;
constexpr int kRangeIds = kBlock * kRangePer;

__global__ void __launch_bounds__(kBlock) k_bucket_range(const int32_t* ids, const int64_t* hot_count,
                                                         int64_t cap, KPart part, int32_t* out,
                                                         int64_t* owner_off, int32_t* ok,
                                                         int32_t order_bit, int32_t* status) {
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  __shared__ int32_t s_bad;
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  if (threadIdx.x == 0) s_bad = 0;
  __syncthreads();
  const int64_t n = bucket_n(hot_count, cap);
  const int P = part.P;
  if (n == 0 && blockIdx.x == 0)
    for (int m = threadIdx.x; m <= P; m += blockDim.x) owner_off[m] = 0;
  const int64_t i0 = (int64_t)blockIdx.x * kRangeIds + (int64_t)threadIdx.x * kRangePer;
  int32_t v[kRangePer + 1];  // v[0] = the id before this thread's first
#pragma unroll
  for (int j = 0; j <= kRangePer; ++j) {
    const int64_t i = i0 + j - 1;
    v[j] = (i >= 0 && i < n) ? ids[i] : -1;
  }
  int bad = 0, bad_id = 0;
  int32_t op = -1;
  if (i0 > 0 && i0 <= n) {
    const int32_t up = v[0];
    op = (up < 0 || (int64_t)up >= part.N) ? P : owner_of(part, s_start, up);
  }
#pragma unroll
  for (int j = 1; j <= kRangePer; ++j) {
    const int64_t i = i0 + j - 1;
    if (i >= n) break;
    const int32_t u = v[j];
    if (u < 0 || (int64_t)u >= part.N) {
      bad = bad_id = 1;
      op = P;
      continue;
    }
    const int32_t o = owner_of(part, s_start, u);
    if (op > o) bad = 1;
    for (int32_t m = op + 1; m <= o; ++m) owner_off[m] = i;
    if (i == n - 1)
      for (int32_t m = o + 1; m <= P; ++m) owner_off[m] = n;
    out[i] = u;
    op = o;
  }
  if (bad) atomicOr(&s_bad, bad_id ? 3 : 1);
  __syncthreads();
  if (threadIdx.x == 0) {
    if (ok) ok[blockIdx.x] = s_bad ? 0 : 1;
    // Trusted input: the general passes do not run, so report here.
    if (s_bad && order_bit) set_status(status, (s_bad & 2) ? (order_bit | GG_DEV_BAD_ID) : order_bit);
  }
}

// True when the identity pass of every block succeeded.
__device__ __forceinline__ bool range_done(const int32_t* ok, int32_t nok, int32_t* s_flag) {
  if (ok == nullptr) return false;
  if (threadIdx.x == 0) *s_flag = 1;
  __syncthreads();
  for (int x = threadIdx.x; x < nok; x += blockDim.x)
    if (ok[x] == 0) *s_flag = 0;
  __syncthreads();
  return *s_flag != 0;
}

__global__ void __launch_bounds__(kBlock) k_bucket_count(const int32_t* ids, const int64_t* hot_count,
                                                         int64_t cap, KPart part, int32_t* cnt,
                                                         int32_t nblk, const int32_t* ok,
                                                         int32_t nok, int32_t* status) {
  __shared__ int32_t s_flag;
  if (range_done(ok, nok, &s_flag)) return;
  __shared__ int32_t hist[GG_MAX_PARTS];
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  for (int t = threadIdx.x; t < GG_MAX_PARTS; t += blockDim.x) hist[t] = 0;
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  __syncthreads();
  const int64_t n = bucket_n(hot_count, cap);
  const int64_t i0 = (int64_t)blockIdx.x * kIdsPerBlock;
  int32_t st = 0;
  for (int it = 0; it < kIdsPerBlock / kBlock; ++it) {
    const int64_t i = i0 + it * kBlock + threadIdx.x;
    bool valid = false;
    int32_t m = 0;
    if (i < n) {
      const int32_t u = ids[i];
      if (u < 0 || (int64_t)u >= part.N) {
        st |= GG_DEV_BAD_ID;
      } else {
        valid = true;
        m = owner_of(part, s_start, u);
      }
    }
    wave_hist_add(hist, valid, m);
  }
  if (st) set_status(status, st);
  __syncthreads();
  for (int m = threadIdx.x; m < part.P; m += blockDim.x) cnt[(int64_t)m * nblk + blockIdx.x] = hist[m];
}

__global__ void __launch_bounds__(1024) k_bucket_scan(const int32_t* cnt, int64_t ncnt, int32_t nblk,
                                                      int32_t P, int64_t* off, int64_t* owner_off,
                                                      const int32_t* ok, int32_t nok) {
  __shared__ int32_t s_flag;
  if (range_done(ok, nok, &s_flag)) return;
  __shared__ int64_t lds[16];
  const int64_t total = block_scan_large(cnt, off, ncnt, 0, lds);
  __syncthreads();
  for (int m = threadIdx.x; m < P; m += blockDim.x) owner_off[m] = off[(int64_t)m * nblk];
  if (threadIdx.x == 0) owner_off[P] = total;
}

__global__ void __launch_bounds__(kBlock) k_bucket_scatter(const int32_t* ids, const int64_t* hot_count,
                                                           int64_t cap, KPart part, const int64_t* off,
                                                           int32_t nblk, const int32_t* ok,
                                                           int32_t nok, int32_t* out) {
  __shared__ int32_t s_flag;
  if (range_done(ok, nok, &s_flag)) return;
  __shared__ int32_t wcnt[4][GG_MAX_PARTS];
  __shared__ int64_t wbase[4][GG_MAX_PARTS];
  __shared__ int64_t s_start[GG_MAX_PARTS + 1];
  const int w = threadIdx.x / kWave, lane = lane_id();
  for (int t = threadIdx.x; t < 4 * GG_MAX_PARTS; t += blockDim.x) (&wcnt[0][0])[t] = 0;
  for (int t = threadIdx.x; t <= GG_MAX_PARTS; t += blockDim.x) s_start[t] = part.start[t];
  __syncthreads();
  const int64_t n = bucket_n(hot_count, cap);
  const int64_t i0 = (int64_t)blockIdx.x * kIdsPerBlock + (int64_t)w * kIdsPerWave;
  // Per-wave owner counts.
  for (int g = 0; g < kIdsPerWave / kWave; ++g) {
    const int64_t i = i0 + g * kWave + lane;
    bool valid = false;
    int32_t m = 0;
    if (i < n) {
      const int32_t u = ids[i];
      if (u >= 0 && (int64_t)u < part.N) {
        valid = true;
        m = owner_of(part, s_start, u);
      }
    }
    wave_hist_add(wcnt[w], valid, m);
  }
  __syncthreads();
  for (int t = threadIdx.x; t < 4 * part.P; t += blockDim.x) {
    const int ww = t / part.P, m = t - ww * part.P;
    int64_t b = off[(int64_t)m * nblk + blockIdx.x];
    for (int v = 0; v < ww; ++v) b += wcnt[v][m];
    wbase[ww][m] = b;
  }
  __syncthreads();
  // Ordered scatter: groups of 64 in id order, ranks by ballot per owner.
  // Lane m keeps the running output position of owner m.
  int64_t my_base = lane < part.P ? wbase[w][lane] : 0;
  for (int g = 0; g < kIdsPerWave / kWave; ++g) {
    const int64_t i = i0 + g * kWave + lane;
    int32_t u = -1, o = -1;
    bool valid = false;
    if (i < n) {
      u = ids[i];
      valid = u >= 0 && (int64_t)u < part.N;
      if (valid) o = owner_of(part, s_start, u);
    }
    uint64_t active = __ballot(valid);
    while (active) {
      const int leader = __ffsll((unsigned long long)active) - 1;
      const int32_t ol = __shfl(o, leader, kWave);
      const uint64_t mm = __ballot(valid && o == ol);
      const int64_t b = __shfl(my_base, ol, kWave);
      if (valid && o == ol) out[b + lanes_below(mm)] = u;
      if (lane == ol) my_base += __popcll(mm);
      active &= ~mm;
    }
  }
}

struct BucketWs {
  int32_t* cnt;
  int64_t* off;
  int32_t* ok;
};

size_t bucket_ws_layout(int64_t cap, int32_t P, char* base, BucketWs* out) {
  const int64_t nblk = std::max<int64_t>(1, cdiv(cap, kIdsPerBlock));
  Carve cv{base, 0, ~(size_t)0};
  BucketWs b;
  b.cnt = cv.take<int32_t>((size_t)(nblk * P));
  b.off = cv.take<int64_t>((size_t)(nblk * P));
  b.ok = cv.take<int32_t>((size_t)std::max<int64_t>(1, cdiv(cap, kRangeIds)));
  if (out) *out = b;
  return align_up(cv.used, 256);
}

}  // namespace
}  // namespace gg

using namespace gg;

extern "C" size_t gg_ws_bucket(int64_t cap, int32_t num_parts) {
  return bucket_ws_layout(cap, num_parts, nullptr, nullptr);
}

extern "C" int gg_bucket_by_owner(const int32_t* hot_ids_d, const int64_t* hot_count_d, int64_t cap,
                                  const gg_part_t* part, int32_t flags, int32_t* bucket_ids_d,
                                  int64_t* owner_off_d, int32_t* status_d, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  GG_REQUIRE(hot_count_d && owner_off_d && status_d, "NULL argument");
  GG_REQUIRE(cap >= 0 && cap < (1LL << 31), "capacity %lld unsupported", (long long)cap);
  GG_REQUIRE(cap == 0 || (hot_ids_d && bucket_ids_d), "NULL id buffer");
  GG_REQUIRE((flags & ~GG_BUCKET_OWNER_ORDERED) == 0, "unknown flags 0x%x", (unsigned)flags);
  KPart kp;
  int rc = pack_part(part, &kp);
  if (rc != GG_OK) return rc;
  BucketWs bw;
  const size_t need_ws = bucket_ws_layout(cap, kp.P, (char*)ws, &bw);
  GG_REQUIRE(ws && ws_bytes >= need_ws, "workspace of %zu bytes < %zu", ws_bytes, need_ws);
  const int32_t nblk = (int32_t)std::max<int64_t>(1, cdiv(cap, kIdsPerBlock));
  const int32_t nrange = (int32_t)std::max<int64_t>(1, cdiv(cap, kRangeIds));
  const int32_t* ok = nullptr;
  if (kp.kind == GG_PART_RANGE) {
    // Owner-ordered input under ranges is its own bucketing.  When the
    // caller vouches for the order, this pass is the whole call and an
    // input out of order is reported instead of repaired.
    const bool trusted = (flags & GG_BUCKET_OWNER_ORDERED) != 0;
    hipLaunchKernelGGL(k_bucket_range, dim3(nrange), dim3(kBlock), 0, stream, hot_ids_d, hot_count_d,
                       cap, kp, bucket_ids_d, owner_off_d, trusted ? nullptr : bw.ok,
                       trusted ? (int32_t)GG_DEV_ORDER : 0, status_d);
    GG_LAUNCH_CHECK("k_bucket_range");
    if (trusted) return GG_OK;
    ok = bw.ok;
  }
  hipLaunchKernelGGL(k_bucket_count, dim3(nblk), dim3(kBlock), 0, stream, hot_ids_d, hot_count_d, cap,
                     kp, bw.cnt, nblk, ok, nrange, status_d);
  GG_LAUNCH_CHECK("k_bucket_count");
  hipLaunchKernelGGL(k_bucket_scan, dim3(1), dim3(1024), 0, stream, bw.cnt, (int64_t)nblk * kp.P,
                     nblk, kp.P, bw.off, owner_off_d, ok, nrange);
  GG_LAUNCH_CHECK("k_bucket_scan");
  hipLaunchKernelGGL(k_bucket_scatter, dim3(nblk), dim3(kBlock), 0, stream, hot_ids_d, hot_count_d,
                     cap, kp, bw.off, nblk, ok, nrange, bucket_ids_d);
  GG_LAUNCH_CHECK("k_bucket_scatter");
  return GG_OK;
}
