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

// pow2 ? tile_rows(row_bytes, max_bytes) : fill_rows(row_bytes, max_bytes),
// or, when GG_TILE_ROWS is set (read at every call), that count, at most 64
// (1 makes a wavefront copy one row per step).
int32_t copy_tile(int32_t row_bytes, int32_t max_bytes, bool pow2 = true);

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Tuning switches read once from the environment: a flag is on unless "0".
bool env_flag(const char* name, bool dflt);
int env_int(const char* name, int dflt);

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
