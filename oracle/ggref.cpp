// ggref: CPU oracle of the per-window feature-fetch path.
//
// TEST INFRASTRUCTURE ONLY: loaded by the test suite, the smoke check and
// the benchmark's CPU-baseline leg, never by the product path.  Plain,
// single-threaded, written for clarity: std::set, std::sort and one memcpy
// per feature row.  It follows the paper (GreenGNN, arXiv 2606.02916) step
// by step; where the paper is silent the reading taken is stated at the
// function.  Nothing here is shared with the HIP library.

#include "ggref.h"

#include <algorithm>
#include <cmath>
#include <iterator>
#include <cstring>
#include <set>
#include <vector>

namespace {

// ---------------------------------------------------------------------------
// Philox4x32-10, from its definition in Salmon, Moraes, Dror and Shaw,
// "Parallel random numbers: as easy as 1, 2, 3" (SC'11), Sec. 3.2: ten
// rounds; each round multiplies words 0 and 2 by the two Philox-4x32
// multipliers, and the new block is (hi(R1) ^ x1 ^ k0, lo(R1),
// hi(R0) ^ x3 ^ k1, lo(R0)); the key is bumped by the Weyl constants
// (golden ratio and sqrt(3)-1, as 32-bit fractions) between rounds.
// ---------------------------------------------------------------------------
const uint32_t kPhiloxM0 = 0xD2511F53u;
const uint32_t kPhiloxM1 = 0xCD9E8D57u;
const uint32_t kWeyl0 = 0x9E3779B9u;
const uint32_t kWeyl1 = 0xBB67AE85u;

void philox_block(const uint32_t in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t x0 = in[0], x1 = in[1], x2 = in[2], x3 = in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += kWeyl0;
      k1 += kWeyl1;
    }
    const uint64_t p0 = (uint64_t)kPhiloxM0 * (uint64_t)x0;
    const uint64_t p1 = (uint64_t)kPhiloxM1 * (uint64_t)x2;
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t y0 = hi1 ^ x1 ^ k0;
    const uint32_t y1 = lo1;
    const uint32_t y2 = hi0 ^ x3 ^ k1;
    const uint32_t y3 = lo0;
    x0 = y0;
    x1 = y1;
    x2 = y2;
    x3 = y3;
  }
  out[0] = x0;
  out[1] = x1;
  out[2] = x2;
  out[3] = x3;
}

int64_t row_start(const ggref_csr_t* g, int64_t u) {
  if (g->row_ptr_bits == 32) return (int64_t)((const int32_t*)g->row_ptr)[u];
  return ((const int64_t*)g->row_ptr)[u];
}

std::vector<int32_t> sort_unique(std::vector<int32_t> v) {
  std::sort(v.begin(), v.end());
  v.erase(std::unique(v.begin(), v.end()), v.end());
  return v;
}

bool part_ok(const ggref_part_t* part) {
  if (!part || part->num_parts < 1 || part->num_parts > GGREF_MAX_PARTS) return false;
  if (part->local_owner < -1 || part->local_owner >= part->num_parts) return false;
  if (part->kind == GGREF_PART_RANGE) {
    if (part->range_start[0] != 0 || part->range_start[part->num_parts] != part->num_nodes) return false;
    for (int m = 0; m < part->num_parts; ++m)
      if (part->range_start[m + 1] < part->range_start[m]) return false;
  } else if (part->kind != GGREF_PART_MOD) {
    return false;
  }
  return true;
}

const char* src_row(const ggref_feat_t* feat, int32_t m, int64_t r) {
  return (const char*)feat->shard[m] + r * feat->row_stride[m];
}

}  // namespace

extern "C" {

void ggref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  philox_block(ctr, key, out);
}

// Lemire's multiply-shift map of a 32-bit word onto [0, bound), without the
// rejection step: floor(r * bound / 2^32).  bound <= 2^32.
uint64_t ggref_bounded(uint32_t r, uint64_t bound) {
  return ((uint64_t)r * bound) >> 32;
}

// Floyd's algorithm (Bentley and Floyd, "Programming pearls: a sample of
// brilliance", CACM 30(9), 1987).  For i = 0..k-1 with j = d-k+i, the i-th
// draw t[i] is uniform on [0, j]; it joins the set unless it is already
// there, in which case j joins instead.  The result has exactly k distinct
// positions of [0, d).
int ggref_floyd(int64_t d, int32_t k, const int64_t* t, int64_t* pos) {
  if (k < 1 || d <= k) return GGREF_ERR_ARG;
  std::set<int64_t> chosen;
  for (int32_t i = 0; i < k; ++i) {
    const int64_t j = d - k + i;
    if (t[i] < 0 || t[i] > j) return GGREF_ERR_ARG;
    if (chosen.count(t[i]))
      chosen.insert(j);
    else
      chosen.insert(t[i]);
  }
  int32_t n = 0;
  for (int64_t p : chosen) pos[n++] = p;
  return GGREF_OK;
}

int32_t ggref_owner(const ggref_part_t* part, int64_t u) {
  if (part->kind == GGREF_PART_MOD) return (int32_t)(u % part->num_parts);
  for (int32_t m = 0; m < part->num_parts; ++m)
    if (u >= part->range_start[m] && u < part->range_start[m + 1]) return m;
  return -1;
}

int64_t ggref_row(const ggref_part_t* part, int64_t u) {
  if (part->kind == GGREF_PART_MOD) return u / part->num_parts;
  const int32_t m = ggref_owner(part, u);
  return m < 0 ? -1 : u - part->range_start[m];
}

// Sampling of one window (Sec. IV-A step 2; the paper takes the sampler
// from DGL).  Readings where the paper is silent:
//  * fanout[l] applies at hop l+1, seed side first;
//  * sampling is without replacement: a node of degree d <= k keeps all
//    its neighbours in CSR order, a node with d > k keeps the k positions
//    chosen by Floyd's algorithm, ascending;
//  * nested frontiers: F_0 = the batch's distinct seeds, F_{l+1} = F_l
//    together with every neighbour sampled at hop l+1, so N_b = F_L;
//  * draw i of node u at hop l in global batch b uses word i mod 4 of the
//    Philox block with counter (u, b, epoch, (l << 16) | (i div 4)) and
//    key (low, high 32 bits of rng_seed); the bounded map gives the Floyd
//    draw on [0, d-k+i].
int ggref_sample_window(const ggref_csr_t* csr, const int32_t* seeds, const int64_t* seed_off,
                        int32_t W, const int32_t* fanout, int32_t L, uint64_t rng_seed,
                        int32_t epoch, int64_t batch0, int32_t* frontier_ids,
                        int64_t frontier_cap, int64_t* frontier_off, int32_t* nbr_ids,
                        int64_t nbr_cap, int64_t* nbr_off, int64_t* need) {
  if (!csr || W < 1 || L < 1 || !seed_off || !fanout) return GGREF_ERR_ARG;
  for (int32_t l = 0; l < L; ++l)
    if (fanout[l] < 1 || fanout[l] > 4 * 65536) return GGREF_ERR_ARG;
  const int64_t N = csr->num_nodes;
  const uint32_t key[2] = {(uint32_t)rng_seed, (uint32_t)(rng_seed >> 32)};

  // frontier[b][l] and sampled[b][l] for every batch of the window.
  std::vector<std::vector<std::vector<int32_t>>> frontier(W), sampled(W);
  for (int32_t b = 0; b < W; ++b) {
    frontier[b].resize(L + 1);
    sampled[b].resize(L);
    std::vector<int32_t> s0;
    for (int64_t i = seed_off[b]; i < seed_off[b + 1]; ++i) {
      if (seeds[i] < 0 || seeds[i] >= N) return GGREF_ERR_RANGE;
      s0.push_back(seeds[i]);
    }
    frontier[b][0] = sort_unique(s0);
    const uint32_t bglob = (uint32_t)(batch0 + b);
    for (int32_t l = 0; l < L; ++l) {
      const int32_t k = fanout[l];
      std::vector<int32_t> next = frontier[b][l];
      std::vector<int32_t>& out = sampled[b][l];
      for (int32_t u : frontier[b][l]) {
        const int64_t beg = row_start(csr, u);
        const int64_t d = row_start(csr, (int64_t)u + 1) - beg;
        std::vector<int64_t> positions;
        if (d <= k) {
          for (int64_t p = 0; p < d; ++p) positions.push_back(p);
        } else {
          if (d > 0xFFFFFFFFLL) return GGREF_ERR_RANGE;
          std::vector<int64_t> t(k), pos(k);
          for (int32_t i = 0; i < k; ++i) {
            const uint32_t ctr[4] = {(uint32_t)u, bglob, (uint32_t)epoch,
                                     ((uint32_t)l << 16) | (uint32_t)(i / 4)};
            uint32_t block[4];
            philox_block(ctr, key, block);
            t[i] = (int64_t)ggref_bounded(block[i % 4], (uint64_t)(d - k + i + 1));
          }
          if (ggref_floyd(d, k, t.data(), pos.data()) != GGREF_OK) return GGREF_ERR_ARG;
          positions = pos;
        }
        for (int64_t p : positions) {
          const int32_t v = csr->col_idx[beg + p];
          if (v < 0 || v >= N) return GGREF_ERR_RANGE;
          out.push_back(v);
          next.push_back(v);
        }
        for (int64_t p = (int64_t)positions.size(); p < k; ++p) out.push_back(-1);
      }
      frontier[b][l + 1] = sort_unique(next);
    }
  }

  // Level-major layout.
  int64_t fpos = 0, npos = 0;
  for (int32_t l = 0; l <= L; ++l)
    for (int32_t b = 0; b < W; ++b) fpos += (int64_t)frontier[b][l].size();
  for (int32_t l = 0; l < L; ++l)
    for (int32_t b = 0; b < W; ++b) npos += (int64_t)sampled[b][l].size();
  if (need) {
    need[0] = fpos;
    need[1] = npos;
  }
  if (fpos > frontier_cap || npos > nbr_cap) return GGREF_ERR_CAPACITY;
  fpos = 0;
  for (int32_t l = 0; l <= L; ++l)
    for (int32_t b = 0; b < W; ++b) {
      frontier_off[l * W + b] = fpos;
      for (int32_t u : frontier[b][l]) frontier_ids[fpos++] = u;
    }
  frontier_off[(L + 1) * W] = fpos;
  npos = 0;
  for (int32_t l = 0; l < L; ++l)
    for (int32_t b = 0; b < W; ++b) {
      nbr_off[l * W + b] = npos;
      for (int32_t v : sampled[b][l]) nbr_ids[npos++] = v;
    }
  nbr_off[L * W] = npos;
  return GGREF_OK;
}

// Hot set H_k of one window (Sec. IV-A window simulation: the most
// frequently accessed remote nodes of the window).  freq(u) counts the
// batches of the window whose N_b holds u.  n_hot < 0 keeps every remote
// node of the window (the union); otherwise the first n_hot in order of
// decreasing freq, ties broken by smaller id.
int ggref_build_hotset(const int32_t* frontier_ids, const int64_t* frontier_off, int32_t W,
                       int32_t L, const ggref_part_t* part, int64_t n_hot, int64_t hot_num,
                       int64_t hot_den, int32_t* hot_ids, int32_t* hot_freq, int64_t cap,
                       int64_t* hot_count) {
  if (!part_ok(part) || W < 1 || L < 0) return GGREF_ERR_ARG;
  if (hot_den < 0 || hot_den > (1LL << 31) ||
      (hot_den > 0 && (n_hot != -1 || hot_num < 0 || hot_num > hot_den)))
    return GGREF_ERR_ARG;
  std::vector<int32_t> remote;
  for (int32_t b = 0; b < W; ++b) {
    const int64_t s = (int64_t)L * W + b;
    for (int64_t i = frontier_off[s]; i < frontier_off[s + 1]; ++i) {
      const int32_t u = frontier_ids[i];
      if (ggref_owner(part, u) != part->local_owner) remote.push_back(u);
    }
  }
  std::sort(remote.begin(), remote.end());
  std::vector<std::pair<int32_t, int32_t>> uf;  // (id, freq), id ascending
  for (size_t i = 0; i < remote.size();) {
    size_t j = i;
    while (j < remote.size() && remote[j] == remote[i]) ++j;
    uf.push_back({remote[i], (int32_t)(j - i)});
    i = j;
  }
  if (hot_den > 0) {   // the top hot_num / hot_den of the U distinct remote nodes, rounded up
    const int64_t U = (int64_t)uf.size();
    n_hot = (U * hot_num + hot_den - 1) / hot_den;
  }
  if (n_hot >= 0 && n_hot < (int64_t)uf.size()) {
    std::stable_sort(uf.begin(), uf.end(),
                     [](const std::pair<int32_t, int32_t>& a, const std::pair<int32_t, int32_t>& b) {
                       return a.second > b.second;
                     });
    uf.resize((size_t)n_hot);
    std::sort(uf.begin(), uf.end());
  }
  if (hot_count) *hot_count = (int64_t)uf.size();
  if ((int64_t)uf.size() > cap) return GGREF_ERR_CAPACITY;
  for (size_t i = 0; i < uf.size(); ++i) {
    hot_ids[i] = uf[i].first;
    if (hot_freq) hot_freq[i] = uf[i].second;
  }
  return GGREF_OK;
}

// Owner grouping (Sec. IV-A rebuild events, Sec. IV-C: one bulk request per
// partition owner).  count[m] = members of owner m; owner_off is its
// exclusive scan; members keep their input order inside each owner.
int ggref_bucket_by_owner(const int32_t* hot_ids, int64_t hot_count, const ggref_part_t* part,
                          int32_t* bucket_ids, int64_t* owner_off) {
  if (!part_ok(part) || hot_count < 0) return GGREF_ERR_ARG;
  const int32_t P = part->num_parts;
  std::vector<int64_t> count(P, 0);
  for (int64_t i = 0; i < hot_count; ++i) {
    const int32_t m = ggref_owner(part, hot_ids[i]);
    if (m < 0) return GGREF_ERR_RANGE;
    ++count[m];
  }
  owner_off[0] = 0;
  for (int32_t m = 0; m < P; ++m) owner_off[m + 1] = owner_off[m] + count[m];
  std::vector<int64_t> cursor(owner_off, owner_off + P);
  for (int64_t i = 0; i < hot_count; ++i) {
    const int32_t m = ggref_owner(part, hot_ids[i]);
    bucket_ids[cursor[m]++] = hot_ids[i];
  }
  return GGREF_OK;
}

// Bulk staging of the window cache (Sec. IV-C; Algorithm 1 WarmCache).
// The node's slot in the cache it came from is read first (the source remap
// may be slot_of itself); then the listed remap entries are cleared; then,
// for every owner, the bucket's rows are filled in bucket order.  Without a
// source cache every row is one owner's bulk request; with one, rows the
// source cache holds are copied from it and only the rebuild delta of
// Sec. IV-A, Delta_{k,m} = (H_k in owner m) minus C_{k-1}, is requested,
// one request per owner whose delta is non-empty (Eq. (1) indicator).
// delta_rows[m] always counts the rows of bucket m absent from the source
// (or, without one, from the current) remap.
int ggref_stage_bulk(const int32_t* bucket_ids, const int64_t* owner_off,
                     const ggref_part_t* part, const ggref_feat_t* feat, void* cache,
                     int64_t cache_stride, int64_t cache_rows, int32_t* slot_of,
                     const int32_t* clear_ids, int64_t clear_count, const void* src_cache,
                     const int32_t* src_slot_of, ggref_stage_stats_t* stats) {
  if (!part_ok(part) || !feat || feat->num_parts != part->num_parts) return GGREF_ERR_ARG;
  const int32_t P = part->num_parts;
  std::memset(stats, 0, sizeof(*stats));
  const int64_t total = owner_off[P];
  if (total > cache_rows) return GGREF_ERR_CAPACITY;
  const int32_t* before = src_slot_of ? src_slot_of : slot_of;
  std::vector<int32_t> old_slot((size_t)total);
  for (int64_t s = 0; s < total; ++s) old_slot[(size_t)s] = before[bucket_ids[s]];
  for (int64_t i = 0; i < clear_count; ++i) slot_of[clear_ids[i]] = -1;
  stats->invalidated = clear_count;
  for (int32_t m = 0; m < P; ++m) {
    for (int64_t s = owner_off[m]; s < owner_off[m + 1]; ++s) {
      const int32_t u = bucket_ids[s];
      if (ggref_owner(part, u) != m) return GGREF_ERR_RANGE;
      const int64_t r = ggref_row(part, u);
      if (r < 0 || r >= feat->shard_rows[m]) return GGREF_ERR_RANGE;
      const int32_t old = old_slot[(size_t)s];
      if (old < 0) ++stats->delta_rows[m];
      char* dst = (char*)cache + s * cache_stride;
      if (src_cache && old >= 0) {
        std::memcpy(dst, (const char*)src_cache + (int64_t)old * cache_stride,
                    (size_t)feat->row_bytes);
        ++stats->retained;
      } else {
        std::memcpy(dst, src_row(feat, m, r), (size_t)feat->row_bytes);
        ++stats->rows[m];
      }
      slot_of[u] = (int32_t)s;
    }
    stats->bytes[m] = stats->rows[m] * feat->row_bytes;
    stats->requests[m] = stats->rows[m] > 0 ? 1 : 0;
    stats->requests_total += stats->requests[m];
  }
  stats->rows_total = total;
  return GGREF_OK;
}

// Delta staging into one persistent cache (Sec. IV-A; Algorithm 1
// WarmCache(H_{k+1} \ C)): what the previous window cached stays in place,
// and only the rebuild delta is fetched, into the lowest free slots.
int ggref_stage_inplace(const int32_t* bucket_ids, const int64_t* owner_off,
                        const ggref_part_t* part, const ggref_feat_t* feat, void* cache,
                        int64_t cache_stride, int64_t cache_rows, int32_t* slot_of,
                        const int32_t* clear_ids, int64_t clear_count,
                        const int32_t* prev_slot_of, ggref_stage_stats_t* stats) {
  if (!part_ok(part) || !feat || feat->num_parts != part->num_parts) return GGREF_ERR_ARG;
  if (prev_slot_of == slot_of) return GGREF_ERR_ARG;
  const int32_t P = part->num_parts;
  const int64_t N = part->num_nodes;
  std::memset(stats, 0, sizeof(*stats));
  // The slots the previous window occupies; the rest are free, ascending.
  std::vector<char> used((size_t)cache_rows, 0);
  if (prev_slot_of)
    for (int64_t u = 0; u < N; ++u) {
      const int32_t s = prev_slot_of[u];
      if (s >= cache_rows) return GGREF_ERR_RANGE;
      if (s >= 0) used[(size_t)s] = 1;
    }
  std::vector<int64_t> free_slots;
  for (int64_t s = 0; s < cache_rows; ++s)
    if (!used[(size_t)s]) free_slots.push_back(s);
  for (int64_t i = 0; i < clear_count; ++i) slot_of[clear_ids[i]] = -1;
  stats->invalidated = clear_count;
  size_t next_free = 0;
  bool short_of_slots = false;
  for (int32_t m = 0; m < P; ++m) {
    for (int64_t s = owner_off[m]; s < owner_off[m + 1]; ++s) {
      const int32_t u = bucket_ids[s];
      if (ggref_owner(part, u) != m) return GGREF_ERR_RANGE;
      const int64_t r = ggref_row(part, u);
      if (r < 0 || r >= feat->shard_rows[m]) return GGREF_ERR_RANGE;
      const int32_t old = prev_slot_of ? prev_slot_of[u] : -1;
      if (old >= 0) {
        slot_of[u] = old;
        ++stats->retained;
        continue;
      }
      ++stats->delta_rows[m];
      if (next_free == free_slots.size()) {
        // No free slot is left: the row is not cached this window, so a
        // gather serves it as a miss.
        slot_of[u] = -1;
        short_of_slots = true;
        continue;
      }
      const int64_t slot = free_slots[next_free++];
      std::memcpy((char*)cache + slot * cache_stride, src_row(feat, m, r), (size_t)feat->row_bytes);
      slot_of[u] = (int32_t)slot;
      ++stats->rows[m];
    }
    stats->bytes[m] = stats->rows[m] * feat->row_bytes;
    stats->requests[m] = (stats->rows[m] > 0) ? 1 : 0;
    stats->requests_total += stats->requests[m];
  }
  stats->rows_total = owner_off[P];
  return short_of_slots ? GGREF_ERR_CAPACITY : GGREF_OK;
}

// Per-batch feature assembly (Algorithm 1, inner loop): a local node is
// read from the local shard, a cached remote node from its cache slot, and
// every other node is a residual miss.  Misses are grouped by owner, input
// order kept, and each non-empty group is one on-demand request
// (the indicator of Eq. (2)); its rows go straight to their output rows.
int ggref_gather_batch(const int32_t* in_ids, int64_t n, const ggref_part_t* part,
                       const ggref_feat_t* feat, const void* cache, int64_t cache_stride,
                       int64_t cache_rows, const int32_t* slot_of, void* out, int64_t out_stride,
                       ggref_gather_stats_t* stats) {
  if (!part_ok(part) || !feat || feat->num_parts != part->num_parts || n < 0) return GGREF_ERR_ARG;
  const int32_t P = part->num_parts;
  std::memset(stats, 0, sizeof(*stats));
  std::vector<std::vector<int64_t>> miss(P);
  for (int64_t i = 0; i < n; ++i) {
    const int32_t u = in_ids[i];
    if (u < 0 || u >= part->num_nodes) return GGREF_ERR_RANGE;
    const int32_t m = ggref_owner(part, u);
    char* dst = (char*)out + i * out_stride;
    if (m == part->local_owner) {
      const int64_t r = ggref_row(part, u);
      if (r >= feat->shard_rows[m]) return GGREF_ERR_RANGE;
      std::memcpy(dst, src_row(feat, m, r), (size_t)feat->row_bytes);
      ++stats->local;
    } else if (slot_of[u] >= 0) {
      if (slot_of[u] >= cache_rows) return GGREF_ERR_RANGE;
      std::memcpy(dst, (const char*)cache + (int64_t)slot_of[u] * cache_stride,
                  (size_t)feat->row_bytes);
      ++stats->hits;
    } else {
      miss[m].push_back(i);
    }
  }
  for (int32_t m = 0; m < P; ++m) {
    stats->miss_rows[m] = (int64_t)miss[m].size();
    stats->miss_requests[m] = miss[m].empty() ? 0 : 1;
    stats->misses += (int64_t)miss[m].size();
    for (int64_t i : miss[m]) {
      const int64_t r = ggref_row(part, in_ids[i]);
      if (r >= feat->shard_rows[m]) return GGREF_ERR_RANGE;
      std::memcpy((char*)out + i * out_stride, src_row(feat, m, r), (size_t)feat->row_bytes);
    }
  }
  stats->rows = n;
  return GGREF_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Trace simulator (Sec. IV-A simulation, Sec. IV-B, Sec. V).
// ---------------------------------------------------------------------------
namespace {

// Prices one communication event whose owners move x[m] rows: every owner
// with rows pays one initiation plus its linear payload (the summand of
// Eq. (1) and Eq. (2)); the event lasts the longer of its slowest owner's
// transfer and all its rows at the aggregate bandwidth ceiling.  Owners
// are taken in ascending order.
double price_event(const std::vector<int64_t>& x, const ggref_part_t* part,
                   const ggref_sim_coeffs_t* c, int64_t* events, int64_t* rows, double* t) {
  double energy = 0.0, slowest = 0.0;
  int64_t moved = 0;
  for (int32_t m = 0; m < part->num_parts; ++m) {
    if (m == part->local_owner || x[m] == 0) continue;   // only remote owners with a transfer
    const double xm = (double)x[m];
    energy = energy + (c->eps_init[m] + c->eps_row[m] * xm);
    const double tm = c->lam_init[m] + c->lam_row[m] * xm;
    if (tm > slowest) slowest = tm;
    moved += x[m];
    *events += 1;
  }
  *rows += moved;
  if (moved > 0) {
    const double ceiling = (double)moved * c->row_bytes / c->bw_bytes_per_s;
    *t = *t + (slowest > ceiling ? slowest : ceiling);
  }
  return energy;
}

}  // namespace

int ggref_simulate_epoch(const int32_t* trace_ids, const int64_t* trace_off, int64_t n_batches,
                         int32_t W, int64_t n_hot, int64_t hot_num, int64_t hot_den,
                         const ggref_part_t* part, const ggref_sim_coeffs_t* coeffs,
                         ggref_sim_acc_t* acc) {
  if (!part_ok(part) || !coeffs || !acc || W < 1 || n_batches < 0 ||
      !(coeffs->bw_bytes_per_s > 0.0))
    return GGREF_ERR_ARG;
  std::memset(acc, 0, sizeof(*acc));
  const int32_t P = part->num_parts;
  std::vector<int32_t> cache;   // C_{k-1}, ascending; C_0 is empty
  const int64_t K = (n_batches + W - 1) / W;
  for (int64_t k = 0; k < K; ++k) {
    const int64_t b0 = k * W, b1 = std::min<int64_t>(n_batches, b0 + W);
    const int32_t Wk = (int32_t)(b1 - b0);
    // H_k from the window's N_b (level 0 of a one-level layout).
    std::vector<int32_t> hot((size_t)std::max<int64_t>(trace_off[b1] - trace_off[b0], 1));
    int64_t nh = 0;
    int rc = ggref_build_hotset(trace_ids, trace_off + b0, Wk, 0, part, n_hot, hot_num, hot_den,
                                hot.data(), nullptr, (int64_t)hot.size(), &nh);
    if (rc != GGREF_OK) return rc;
    hot.resize((size_t)nh);
    // Rebuild event: Delta_{k,m} = (H_k in owner m) \ C_{k-1}.
    std::vector<int32_t> delta;
    std::set_difference(hot.begin(), hot.end(), cache.begin(), cache.end(),
                        std::back_inserter(delta));
    std::vector<int64_t> x(P, 0);
    for (int32_t u : delta) ++x[ggref_owner(part, u)];
    acc->e_rebuild = acc->e_rebuild + price_event(x, part, coeffs, &acc->rebuild_events,
                                                  &acc->rebuild_rows, &acc->t_stall);
    // Miss events: M_{b,m} = (N_b in owner m) \ H_k for remote m.
    for (int64_t b = b0; b < b1; ++b) {
      std::vector<int32_t> remote;
      for (int64_t i = trace_off[b]; i < trace_off[b + 1]; ++i)
        if (ggref_owner(part, trace_ids[i]) != part->local_owner) remote.push_back(trace_ids[i]);
      std::vector<int32_t> miss;
      std::set_difference(remote.begin(), remote.end(), hot.begin(), hot.end(),
                          std::back_inserter(miss));
      std::fill(x.begin(), x.end(), 0);
      for (int32_t u : miss) ++x[ggref_owner(part, u)];
      acc->e_miss = acc->e_miss + price_event(x, part, coeffs, &acc->miss_events,
                                              &acc->miss_rows, &acc->t_stall);
      acc->remote_rows += (int64_t)remote.size();
      acc->hits += (int64_t)(remote.size() - miss.size());
    }
    cache = hot;   // C_k = H_k (Algorithm 1: the cache holds the window's hot set)
    acc->windows += 1;
    acc->batches += Wk;
    acc->e_stall = coeffs->p_idle * acc->t_stall;
    acc->e_phy = (acc->e_rebuild + acc->e_miss) + acc->e_stall;
  }
  return GGREF_OK;
}

// ---------------------------------------------------------------------------
// GraphSAGE consumer of X_b (mean aggregator), in fp64.
// ---------------------------------------------------------------------------
namespace {

// IEEE 754 binary16 to double, from the bit fields.
double half_to_double(uint16_t h) {
  const int sign = (h >> 15) & 1, exp = (h >> 10) & 31, man = h & 1023;
  double v;
  if (exp == 0)
    v = std::ldexp((double)man, -24);                  // subnormal (or zero)
  else if (exp == 31)
    v = man ? std::nan("") : INFINITY;
  else
    v = std::ldexp((double)(1024 + man), exp - 25);    // (1 + man/1024) * 2^(exp-15)
  return sign ? -v : v;
}

}  // namespace

int ggref_sage_forward(const int32_t* frontier_ids, const int64_t* frontier_off,
                       const int32_t* nbr_ids, const int64_t* nbr_off, int32_t W, int32_t L,
                       const int32_t* fanout, const void* x, int32_t x_dtype, int64_t x_stride,
                       const ggref_sage_layer_t* layers, double* out, double* out_abs) {
  if (W < 1 || L < 1 || (x_dtype != 0 && x_dtype != 1) || !layers || !out) return GGREF_ERR_ARG;
  for (int32_t j = 0; j < L; ++j) {
    if (layers[j].d_in < 1 || layers[j].d_out < 1) return GGREF_ERR_ARG;
    if (j > 0 && layers[j].d_in != layers[j - 1].d_out) return GGREF_ERR_ARG;
  }
  const int64_t esz = x_dtype == 0 ? 4 : 2;
  if (x_stride < layers[0].d_in * esz) return GGREF_ERR_ARG;
  const int32_t d_last = layers[L - 1].d_out;
  for (int32_t b = 0; b < W; ++b) {
    // h^0 = X_b over F_L(b)
    const int64_t sL = (int64_t)L * W + b;
    const int64_t nL = frontier_off[sL + 1] - frontier_off[sL];
    const int64_t xrow0 = frontier_off[sL] - frontier_off[(int64_t)L * W];
    int32_t d = layers[0].d_in;
    std::vector<double> h((size_t)(nL * d)), ha((size_t)(nL * d));
    for (int64_t i = 0; i < nL; ++i) {
      const char* row = (const char*)x + (xrow0 + i) * x_stride;
      for (int32_t c = 0; c < d; ++c) {
        double v;
        if (x_dtype == 0) {
          float f;
          std::memcpy(&f, row + 4 * c, 4);
          v = f;
        } else {
          uint16_t bits;
          std::memcpy(&bits, row + 2 * c, 2);
          v = half_to_double(bits);
        }
        h[(size_t)(i * d + c)] = v;
        ha[(size_t)(i * d + c)] = std::fabs(v);
      }
    }
    for (int32_t j = 1; j <= L; ++j) {
      const int32_t lvl = L - j;                      // output level; input level lvl + 1
      const ggref_sage_layer_t& ly = layers[j - 1];
      const int64_t sin = (int64_t)(lvl + 1) * W + b, sout = (int64_t)lvl * W + b;
      const int32_t* Fin = frontier_ids + frontier_off[sin];
      const int64_t nin = frontier_off[sin + 1] - frontier_off[sin];
      const int32_t* Fout = frontier_ids + frontier_off[sout];
      const int64_t nout = frontier_off[sout + 1] - frontier_off[sout];
      const int32_t k = fanout[lvl];
      const int32_t* S = nbr_ids + nbr_off[(int64_t)lvl * W + b];
      if (nbr_off[(int64_t)lvl * W + b + 1] - nbr_off[(int64_t)lvl * W + b] != nout * k)
        return GGREF_ERR_RANGE;
      auto pos = [&](int32_t u) -> int64_t {          // row of u in h (F_in ascending)
        const int32_t* p = std::lower_bound(Fin, Fin + nin, u);
        return (p != Fin + nin && *p == u) ? (int64_t)(p - Fin) : -1;
      };
      const int32_t dout = ly.d_out;
      std::vector<double> g((size_t)(nout * dout)), ga((size_t)(nout * dout));
      std::vector<double> mean((size_t)d), meana((size_t)d);
      for (int64_t i = 0; i < nout; ++i) {
        const int64_t pv = pos(Fout[i]);
        if (pv < 0) return GGREF_ERR_RANGE;
        std::fill(mean.begin(), mean.end(), 0.0);
        std::fill(meana.begin(), meana.end(), 0.0);
        int32_t cnt = 0;
        for (int32_t t = 0; t < k; ++t) {
          const int32_t u = S[i * k + t];
          if (u < 0) continue;
          const int64_t pu = pos(u);
          if (pu < 0) return GGREF_ERR_RANGE;
          for (int32_t c = 0; c < d; ++c) {
            mean[(size_t)c] += h[(size_t)(pu * d + c)];
            meana[(size_t)c] += ha[(size_t)(pu * d + c)];
          }
          ++cnt;
        }
        if (cnt > 0)
          for (int32_t c = 0; c < d; ++c) {
            mean[(size_t)c] /= cnt;
            meana[(size_t)c] /= cnt;
          }
        for (int32_t o = 0; o < dout; ++o) {
          double y = ly.bias ? (double)ly.bias[o] : 0.0;
          double ya = std::fabs(y);
          for (int32_t c = 0; c < d; ++c) {
            const double ws = ly.w_self[(size_t)c * dout + o], wn = ly.w_neigh[(size_t)c * dout + o];
            y += ws * h[(size_t)(pv * d + c)] + wn * mean[(size_t)c];
            ya += std::fabs(ws) * ha[(size_t)(pv * d + c)] + std::fabs(wn) * meana[(size_t)c];
          }
          if (ly.relu && y < 0) y = 0;
          g[(size_t)(i * dout + o)] = y;
          ga[(size_t)(i * dout + o)] = ya;
        }
      }
      h.swap(g);
      ha.swap(ga);
      d = dout;
    }
    const int64_t n0 = frontier_off[b + 1] - frontier_off[b];
    const int64_t orow0 = frontier_off[b] - frontier_off[0];
    for (int64_t i = 0; i < n0 * d_last; ++i) {
      out[orow0 * d_last + i] = h[(size_t)i];
      if (out_abs) out_abs[orow0 * d_last + i] = ha[(size_t)i];
    }
  }
  return GGREF_OK;
}
