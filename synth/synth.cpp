// Seeded synthetic inputs for the per-window feature-fetch path.
//
// This library only produces inputs: R-MAT power-law graphs in CSR form,
// random node relabellings, permutations for train splits and epoch orders,
// and dense feature matrices.  It contains none of the arithmetic of the
// feature-fetch method itself (no sampling, hot set, bucketing, staging or
// gathering), and both the CPU oracle and the HIP path consume what it
// writes.  Every value is a pure function of (seed, stream, index), so the
// output does not depend on the thread count.
//
// Random words come from SplitMix64 (Steele, Lea and Flood, OOPSLA 2014),
// used as a counter-based hash.  It is deliberately a different generator
// from the Philox stream that the sampler draws from.

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <thread>
#include <vector>

namespace {

inline uint64_t mix64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

// Word i of the stream (seed, stream).
inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
  return mix64(seed * 0xD1B54A32D192ED03ULL ^ mix64(stream));
}
inline uint64_t word64(uint64_t seed, uint64_t stream, uint64_t i) {
  return mix64(stream_key(seed, stream) + i);
}

int num_threads() {
  unsigned hc = std::thread::hardware_concurrency();
  if (hc == 0) hc = 4;
  return (int)std::min<unsigned>(hc, 16u);
}

// Runs f(i) for i in [0, n) on the worker threads.  Items are handed out in
// grains; `heavy` marks loops whose items are large chunks of work, which
// are spread one at a time and never run serially.
template <class F>
void parallel_for(int64_t n, F f, bool heavy = false) {
  int nt = num_threads();
  if (n < 4096 && !heavy) nt = 1;
  std::vector<std::thread> th;
  std::atomic<int64_t> next{0};
  const int64_t grain =
      heavy ? 1 : std::max<int64_t>(1, std::min<int64_t>(1 << 16, n / (nt * 8) + 1));
  for (int t = 0; t < nt; ++t) {
    th.emplace_back([&]() {
      for (;;) {
        int64_t b = next.fetch_add(grain);
        if (b >= n) break;
        int64_t e = std::min(n, b + grain);
        for (int64_t i = b; i < e; ++i) f(i);
      }
    });
  }
  for (auto& t : th) t.join();
}

// Bijection on [0, n): a 4-round Feistel network on the smallest even-width
// power-of-two domain that covers n, with cycle walking back into [0, n).
struct Perm {
  uint64_t n;
  int half;
  uint64_t mask;
  uint64_t keys[4];
};

Perm make_perm(uint64_t n, uint64_t seed, uint64_t stream) {
  Perm p;
  p.n = n;
  int bits = 2;
  while ((1ULL << bits) < n) ++bits;
  if (bits & 1) ++bits;
  p.half = bits / 2;
  p.mask = (1ULL << p.half) - 1;
  for (int i = 0; i < 4; ++i) p.keys[i] = word64(seed, stream, (uint64_t)i);
  return p;
}

inline uint64_t perm_apply(const Perm& p, uint64_t x) {
  do {
    uint64_t L = x >> p.half, R = x & p.mask;
    for (int i = 0; i < 4; ++i) {
      uint64_t t = L ^ (mix64(R ^ p.keys[i]) & p.mask);
      L = R;
      R = t;
    }
    x = (L << p.half) | R;
  } while (x >= p.n);
  return x;
}

enum : uint64_t {
  STREAM_RMAT = 1,
  STREAM_RELABEL = 2,
  STREAM_FEAT = 3,
};

// One R-MAT candidate edge.  Each level draws one 32-bit word and picks a
// quadrant of the adjacency matrix with probabilities (a, b, c, 1-a-b-c).
inline void rmat_candidate(uint64_t key, uint64_t c, int scale, uint32_t t1, uint32_t t2,
                           uint32_t t3, uint64_t* src, uint64_t* dst) {
  uint64_t s = 0, d = 0;
  uint64_t w = 0;
  const uint64_t base = c * (uint64_t)((scale + 1) / 2);
  for (int lv = 0; lv < scale; ++lv) {
    if ((lv & 1) == 0) w = mix64(key + base + (uint64_t)(lv / 2));
    const uint32_t r = (lv & 1) ? (uint32_t)(w >> 32) : (uint32_t)w;
    // Quadrants in order (0,0), (0,1), (1,0), (1,1) below t1, t2, t3, 2^32.
    const uint64_t g1 = r >= t1, g2 = r >= t2, g3 = r >= t3;
    s = (s << 1) | g2;
    d = (d << 1) | (g1 ^ g2 ^ g3);
  }
  *src = s;
  *dst = d;
}

}  // namespace

extern "C" {

int synth_version() { return 1; }

// Writes a bijection of [0, n) into out[n]: out[i] = perm(i).
void synth_permutation(int64_t n, uint64_t seed, uint64_t stream, int64_t* out) {
  Perm p = make_perm((uint64_t)n, seed, stream + 100);
  parallel_for(n, [&](int64_t i) { out[i] = (int64_t)perm_apply(p, (uint64_t)i); });
}

// R-MAT graph with exactly `num_edges` directed edges over `num_nodes`
// nodes.  Candidates whose endpoints fall outside [0, num_nodes) are
// rejected; accepted candidates are kept in candidate order until
// `num_edges` are found.  With relabel != 0, node ids go through a random
// bijection.  The CSR is written with rows (sources) ascending and the
// neighbours of each row sorted ascending; self loops and repeated edges
// are kept.  row_ptr has num_nodes + 1 entries.
// Returns 0 on success, -1 if the candidate budget ran out.
int synth_rmat_csr(int64_t num_nodes, int64_t num_edges, double a, double b, double c,
                   uint64_t seed, int relabel, int64_t* row_ptr, int32_t* col_idx) {
  int scale = 1;
  while ((1LL << scale) < num_nodes) ++scale;
  const double two32 = 4294967296.0;
  const uint32_t t1 = (uint32_t)std::min(two32 - 1, a * two32);
  const uint32_t t2 = (uint32_t)std::min(two32 - 1, (a + b) * two32);
  const uint32_t t3 = (uint32_t)std::min(two32 - 1, (a + b + c) * two32);
  const int64_t CH = 1 << 18;
  const uint64_t rkey = stream_key(seed, STREAM_RMAT);

  // Pass 1: count accepted candidates per chunk until the budget covers E.
  std::vector<int64_t> chunk_cnt;
  int64_t have = 0;
  int64_t nchunks = 0;
  const int64_t max_chunks = (num_edges / CH + 1) * 64 + 64;
  while (have < num_edges) {
    int64_t add = std::max<int64_t>(16, (num_edges - have) / CH + 1);
    add = add + add / 4 + 1;
    if (nchunks + add > max_chunks) add = max_chunks - nchunks;
    if (add <= 0) return -1;
    chunk_cnt.resize((size_t)(nchunks + add));
    const int64_t first = nchunks;
    parallel_for(add, [&](int64_t k) {
      const int64_t ch = first + k;
      int64_t cnt = 0;
      for (int64_t i = 0; i < CH; ++i) {
        uint64_t s, d;
        rmat_candidate(rkey, (uint64_t)(ch * CH + i), scale, t1, t2, t3, &s, &d);
        cnt += (s < (uint64_t)num_nodes && d < (uint64_t)num_nodes);
      }
      chunk_cnt[(size_t)ch] = cnt;
    }, true);
    for (int64_t k = 0; k < add; ++k) have += chunk_cnt[(size_t)(first + k)];
    nchunks += add;
  }
  std::vector<int64_t> chunk_off((size_t)nchunks + 1, 0);
  for (int64_t k = 0; k < nchunks; ++k) chunk_off[(size_t)k + 1] = chunk_off[(size_t)k] + chunk_cnt[(size_t)k];
  int64_t used = 0;
  while (used < nchunks && chunk_off[(size_t)used] < num_edges) ++used;

  // Pass 2: regenerate the used chunks and write accepted edges in order.
  std::vector<int32_t> es((size_t)num_edges), ed((size_t)num_edges);
  Perm rp = make_perm((uint64_t)num_nodes, seed, STREAM_RELABEL);
  parallel_for(used, [&](int64_t ch) {
    int64_t pos = chunk_off[(size_t)ch];
    for (int64_t i = 0; i < CH && pos < num_edges; ++i) {
      uint64_t s, d;
      rmat_candidate(rkey, (uint64_t)(ch * CH + i), scale, t1, t2, t3, &s, &d);
      if (s < (uint64_t)num_nodes && d < (uint64_t)num_nodes) {
        if (relabel) {
          s = perm_apply(rp, s);
          d = perm_apply(rp, d);
        }
        es[(size_t)pos] = (int32_t)s;
        ed[(size_t)pos] = (int32_t)d;
        ++pos;
      }
    }
  }, true);

  // Counting sort by source, then sort each row.
  std::vector<std::atomic<int64_t>> deg((size_t)num_nodes);
  parallel_for(num_nodes, [&](int64_t u) { deg[(size_t)u].store(0, std::memory_order_relaxed); });
  parallel_for(num_edges, [&](int64_t e) { deg[(size_t)es[(size_t)e]].fetch_add(1, std::memory_order_relaxed); });
  row_ptr[0] = 0;
  for (int64_t u = 0; u < num_nodes; ++u) row_ptr[u + 1] = row_ptr[u] + deg[(size_t)u].load(std::memory_order_relaxed);
  parallel_for(num_nodes, [&](int64_t u) { deg[(size_t)u].store(row_ptr[u], std::memory_order_relaxed); });
  parallel_for(num_edges, [&](int64_t e) {
    int64_t p = deg[(size_t)es[(size_t)e]].fetch_add(1, std::memory_order_relaxed);
    col_idx[p] = ed[(size_t)e];
  });
  parallel_for(num_nodes, [&](int64_t u) { std::sort(col_idx + row_ptr[u], col_idx + row_ptr[u + 1]); });
  return 0;
}

// Float to IEEE binary16, round to nearest even (finite inputs).
static inline uint16_t f32_to_f16(float f) {
  uint32_t x;
  std::memcpy(&x, &f, 4);
  uint32_t sign = (x >> 16) & 0x8000u;
  int32_t exp = (int32_t)((x >> 23) & 0xFF) - 127 + 15;
  uint32_t mant = x & 0x7FFFFFu;
  if (exp >= 31) return (uint16_t)(sign | 0x7C00u);
  if (exp <= 0) {
    if (exp < -10) return (uint16_t)sign;
    mant |= 0x800000u;
    int shift = 14 - exp;
    uint32_t h = mant >> shift;
    uint32_t rem = mant & ((1u << shift) - 1);
    uint32_t halfway = 1u << (shift - 1);
    if (rem > halfway || (rem == halfway && (h & 1u))) ++h;
    return (uint16_t)(sign | h);
  }
  uint32_t h = ((uint32_t)exp << 10) | (mant >> 13);
  uint32_t rem = mant & 0x1FFFu;
  if (rem > 0x1000u || (rem == 0x1000u && (h & 1u))) ++h;
  return (uint16_t)(sign | h);
}

// Feature rows for nodes [u_begin, u_end): row u is written at
// out + (u - u_begin) * stride_bytes.  dtype 0 = fp32, 1 = fp16.
// dist 0 = N(0,1) (Box-Muller, two values per draw), 1 = U(-1,1).
// Padding bytes between row_bytes and the stride are zero.
void synth_features(int64_t u_begin, int64_t u_end, int32_t dim, int32_t dtype, int32_t dist,
                    int64_t stride_bytes, uint64_t seed, void* out) {
  const int64_t row_bytes = (int64_t)dim * (dtype == 0 ? 4 : 2);
  const uint64_t key = stream_key(seed, STREAM_FEAT);
  parallel_for(u_end - u_begin, [&](int64_t k) {
    const int64_t u = u_begin + k;
    char* row = (char*)out + k * stride_bytes;
    for (int32_t j = 0; j < dim; j += 2) {
      const uint64_t w = mix64(key + (uint64_t)u * (uint64_t)dim + (uint64_t)j);
      const double u1 = ((double)(w >> 11) + 0.5) * (1.0 / 9007199254740992.0);
      float v[2];
      if (dist == 0) {
        const uint64_t w2 = mix64(w ^ 0x5851F42D4C957F2DULL);
        const double u2 = (double)(w2 >> 11) * (1.0 / 9007199254740992.0);
        const double r = std::sqrt(-2.0 * std::log(u1)), th = 6.283185307179586 * u2;
        v[0] = (float)(r * std::cos(th));
        v[1] = (float)(r * std::sin(th));
      } else {
        const uint64_t w2 = mix64(w ^ 0x5851F42D4C957F2DULL);
        v[0] = (float)(2.0 * u1 - 1.0);
        v[1] = (float)(2.0 * (((double)(w2 >> 11) + 0.5) * (1.0 / 9007199254740992.0)) - 1.0);
      }
      for (int t = 0; t < 2 && j + t < dim; ++t) {
        if (dtype == 0) {
          std::memcpy(row + (int64_t)(j + t) * 4, &v[t], 4);
        } else {
          const uint16_t h = f32_to_f16(v[t]);
          std::memcpy(row + (int64_t)(j + t) * 2, &h, 2);
        }
      }
    }
    if (stride_bytes > row_bytes) std::memset(row + row_bytes, 0, (size_t)(stride_bytes - row_bytes));
  });
}

}  // extern "C"
