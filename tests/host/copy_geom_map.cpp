// Checks the row copy engine's chunk-to-row map (copy_geom.hpp) on the
// host, for every row width libgg accepts (4 .. 32768 bytes, multiples of
// 4) and both vector widths (16-byte chunks plus 4-byte tail words, and
// 4-byte chunks): for a tile of 64 rows, every chunk index c must decode
// to row c / cpr and column c mod cpr, and every tail word to row
// c / tail, and the chunks and tail words of one row must cover exactly
// its bytes.  Prints the number of widths checked and exits non-zero on
// the first mismatch.
#include <stdint.h>
#include <stdio.h>

#include "copy_geom.hpp"

static int check_div(uint32_t d, uint32_t magic, int rb, int vb, const char* what) {
  const uint32_t n = 64u * d;   // chunks of a full 64-row tile
  for (uint32_t c = 0; c < n; ++c) {
    const uint32_t r = gg::chunk_row(c, magic);
    if (r != c / d || c - r * d != c % d) {
      printf("row_bytes %d vb %d %s: chunk %u -> row %u, want %u\n", rb, vb, what, c, r, c / d);
      return 1;
    }
  }
  return 0;
}

int main() {
  int widths = 0;
  for (int rb = 4; rb <= 32768; rb += 4) {
    for (int vb = 16; vb >= 4; vb -= 12) {
      const gg::CopyGeom g = gg::copy_geom(rb, vb);
      const int64_t covered = (int64_t)g.cpr * vb + (int64_t)g.tail * 4;
      if (g.row_bytes != rb || covered != rb) {
        printf("row_bytes %d vb %d: chunks cover %lld bytes\n", rb, vb, (long long)covered);
        return 1;
      }
      if (g.cpr && check_div(g.cpr, g.magic, rb, vb, "chunk")) return 1;
      if (g.tail && check_div(g.tail, g.tmagic, rb, vb, "tail")) return 1;
    }
    ++widths;
  }
  printf("%d\n", widths);
  return 0;
}
