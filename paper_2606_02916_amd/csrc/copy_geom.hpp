// Geometry of the row copy engine: how a tile of rows is cut into VB-byte
// chunks (VB = 16 or 4) and how a chunk index maps back to its row.  Plain
// integer code, shared by the host (which fills the struct) and the kernels
// (which decode chunk indices); it needs no HIP header, so a host program
// can check the map for every row width the library accepts.
#pragma once

#include <stdint.h>

#ifdef __HIPCC__
#define GG_HD __host__ __device__
#else
#define GG_HD
#endif

namespace gg {

struct CopyGeom {
  int32_t row_bytes;
  uint32_t cpr;       // full VB-byte chunks per row
  uint32_t magic;     // div_magic(cpr)
  uint32_t tail;      // 4-byte words after the full chunks (VB = 16 only)
  uint32_t tmagic;    // div_magic(tail)
};

// Multiplier for c / d as the high word of c * magic: magic = ceil(2^32 / d).
// With e = magic * d - 2^32 (0 <= e < d) the quotient is exact while
// c * e < 2^32; a tile has at most 64 rows, so c < 64 d and d <= 8192
// suffices (d is at most 32768 / 4).  A divisor of 1 has no 32-bit
// multiplier (2^32 does not fit), so it is marked by magic = 0 and
// chunk_row returns c itself; d = 0 (no chunks) also gives 0 and is never
// decoded.
GG_HD inline uint32_t div_magic(uint32_t d) {
  return d > 1 ? (uint32_t)(((1ULL << 32) + d - 1) / d) : 0u;
}

// Row of chunk c, for a divisor whose multiplier is `magic`.
GG_HD inline uint32_t chunk_row(uint32_t c, uint32_t magic) {
  return magic ? (uint32_t)(((uint64_t)c * magic) >> 32) : c;
}

inline CopyGeom copy_geom(int32_t row_bytes, int vb) {
  CopyGeom g;
  g.row_bytes = row_bytes;
  g.cpr = (uint32_t)(row_bytes / vb);
  g.tail = vb == 16 ? (uint32_t)((row_bytes % 16) / 4) : 0u;
  g.magic = div_magic(g.cpr);
  g.tmagic = div_magic(g.tail);
  return g;
}

}  // namespace gg
