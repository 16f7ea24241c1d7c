/* Exhaustive check of the oracle's bounded map for one small bound B: calls
 * ggref_bounded for every 32-bit word and prints
 *   min_count max_count n_values monotone first last out_of_range
 * where counts are the preimage sizes of each value in [0, B). */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

uint64_t ggref_bounded(uint32_t r, uint64_t bound);

#define NCHUNK 256

int main(int argc, char** argv) {
  if (argc < 2) return 2;
  const uint64_t B = strtoull(argv[1], 0, 10);
  if (B < 1 || B > 64) return 2;
  static uint64_t cnt[NCHUNK][65];
  static uint64_t lo[NCHUNK], hi[NCHUNK];
  static int mono[NCHUNK], oor[NCHUNK];
  memset(cnt, 0, sizeof(cnt));
  const uint64_t span = (1ull << 32) / NCHUNK;
#pragma omp parallel for schedule(dynamic, 1)
  for (int c = 0; c < NCHUNK; ++c) {
    uint64_t prev = ggref_bounded((uint32_t)(c * span), B);
    lo[c] = prev;
    mono[c] = 1;
    oor[c] = 0;
    for (uint64_t r = c * span; r < (c + 1) * span; ++r) {
      uint64_t t = ggref_bounded((uint32_t)r, B);
      if (t >= B) { oor[c] = 1; t = B; }
      cnt[c][t]++;
      if (t < prev) mono[c] = 0;
      prev = t;
    }
    hi[c] = prev;
  }
  int monotone = 1, out_of_range = 0;
  uint64_t tot[65] = {0};
  for (int c = 0; c < NCHUNK; ++c) {
    monotone &= mono[c];
    out_of_range |= oor[c];
    if (c > 0 && lo[c] < hi[c - 1]) monotone = 0;
    for (uint64_t t = 0; t <= B; ++t) tot[t] += cnt[c][t];
  }
  uint64_t mn = ~0ull, mx = 0, nv = 0;
  for (uint64_t t = 0; t < B; ++t) {
    if (tot[t] < mn) mn = tot[t];
    if (tot[t] > mx) mx = tot[t];
    nv += tot[t] > 0;
  }
  printf("%llu %llu %llu %d %llu %llu %d\n", (unsigned long long)mn, (unsigned long long)mx,
         (unsigned long long)nv, monotone, (unsigned long long)lo[0],
         (unsigned long long)hi[NCHUNK - 1], out_of_range);
  return 0;
}
