// Host-side helpers of libgg: argument checks, error reporting, kernel
// argument packing and workspace carving.
#pragma once

#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include <algorithm>

#include "gg.h"
#include "gg_dev.hpp"

namespace gg {

void set_error(const char* fmt, ...);

#define GG_REQUIRE(cond, ...)        \
  do {                               \
    if (!(cond)) {                   \
      ::gg::set_error(__VA_ARGS__);  \
      return GG_ERR_ARG;             \
    }                                \
  } while (0)

#define GG_LAUNCH_CHECK(what)                                                           \
  do {                                                                                  \
    hipError_t e_ = hipGetLastError();                                                  \
    if (e_ != hipSuccess) {                                                             \
      ::gg::set_error("%s: launch failed: %s", what, hipGetErrorString(e_));           \
      return GG_ERR_HIP;                                                                \
    }                                                                                   \
  } while (0)

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t a, size_t b) { return (a + b - 1) / b * b; }

// Checks a partition book and packs it for the kernels.
int pack_part(const gg_part_t* part, KPart* out);

// Checks feature shards against a partition book and packs them.
int pack_feat(const gg_feat_t* feat, const gg_part_t* part, KFeat* out);

// Rows a wavefront takes per step of a row copy: the largest power of two
// up to 64 whose rows fit in max_bytes, so that wide rows still spread over
// every wave of the grid.
inline int32_t tile_rows(int32_t row_bytes, int32_t max_bytes) {
  int32_t t = 64;
  while (t > 1 && (int64_t)t * row_bytes > max_bytes) t >>= 1;
  return t;
}

// Rows a wavefront takes per step of a row copy: as many as fit in
// max_bytes, up to 64.  Any count works, since the copy engine spreads a
// tile's 16-byte chunks over all lanes; 20 rows of 400 bytes (500 chunks)
// fill two steps of 256 loads to 98%, where 16 rows (400 chunks) fill
// them to 78%.
inline int32_t fill_rows(int32_t row_bytes, int32_t max_bytes) {
  const int64_t t = row_bytes > 0 ? max_bytes / row_bytes : 64;
  return (int32_t)(t < 1 ? 1 : (t > 64 ? 64 : t));
}

// Launch-shape defaults (gg_tuning_t fields left 0).
constexpr int kGatherBlocksDefault = 1024;   // gather blocks per launch
constexpr int kGatherLoadsAlone = 8;         // row loads in flight per lane
constexpr int kGatherLoadsShared = 4;        // ... under GG_GATHER_SHARED
constexpr int kStageBlocksDefault = 16384;   // most staging blocks (device shards)
constexpr int kStageHostBlocksDefault = 128; // ... when a shard is in host memory
constexpr int kEmitBlocksMax = 512;          // most in-place free-list blocks
constexpr int kHotMaxChunks = 4096;          // most hot-set chunks
constexpr int64_t kByteMapMaxBytes = 512LL << 20;  // largest sampler byte map
constexpr int kMarkSlicesDefault = 8;        // most LDS mark slices per batch
constexpr int kMarkSliceChunksDefault = 8;   // 8 KB chunks per mark slice
constexpr int kMarkBlockLanes = 256;         // lanes per mark block

// gg_tuning_t checked and resolved against the defaults.
struct Tune {
  int32_t tile_rows;          // 0: by row width
  int32_t gather_blocks;
  int32_t gather_loads;       // 0: by GG_GATHER_SHARED
  int32_t stage_blocks;
  int32_t stage_host_blocks;
  int32_t emit_blocks;
  int32_t hot_max_chunks;
  int64_t bytemap_max_bytes;  // -1: no byte map
  int32_t sample_order;       // GG_SAMPLE_*
  int32_t sample_tile_runs;   // 0: per hop
  int32_t mark_slices_max;    // -1: marks by atomics (or the byte map)
  int32_t mark_slice_chunks;  // 8 KB chunks of a batch's set per mark slice
  int32_t mark_block;         // lanes per mark block: 256 or 1024
  int64_t mark_min_slots;     // a hop before the last: LDS marks from this slot bound per batch
  int32_t mark_min_batches;   // LDS marks from this many batches; 0: by the alternative
};

// Resolves `t` (NULL: every default) into *out; GG_ERR_ARG (with a message)
// for a value outside its range.
int resolve_tuning(const gg_tuning_t* t, Tune* out);

// pow2 ? tile_rows(row_bytes, max_bytes) : fill_rows(row_bytes, max_bytes),
// or the tuning's tile_rows when set (1 makes a wavefront copy one row per
// step).
int32_t copy_tile(const Tune& tune, int32_t row_bytes, int32_t max_bytes, bool pow2 = true);

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Number of shards with rows whose memory is pinned host memory (read by
// the kernels over PCIe rather than from HBM).
int host_shards(const KFeat& f);

// Bump allocator over the caller's workspace.
struct Carve {
  char* base;
  size_t used;
  size_t cap;
  template <typename T>
  T* take(size_t count) {
    used = align_up(used, 256);
    T* p = (T*)(base + used);
    used += count * sizeof(T);
    return p;
  }
  bool ok() const { return used <= cap; }
};

}  // namespace gg
