// gg_build_hotset: the hot set of one window from the W bit sets N_b.
//
// For every 32-node word the W batch words are summed into bit-sliced
// counters (plane p holds bit p of every node's freq), so freq, the union
// and the comparisons freq > f / freq == f are a handful of bitwise ops per
// word.  With a budget n_hot the frequency histogram fixes a threshold f*
// and a remainder r: the hot set is every remote node with freq > f* plus
// the r smallest ids with freq == f*, which is the n_hot most frequent with
// ties broken by smaller id.  Ids come out ascending because words are
// visited in id order.
#include <stdlib.h>

#include "gg_host.hpp"

namespace gg {
namespace {

constexpr int kPlanes = 7;  // freq <= GG_MAX_W = 64 needs 7 bits

struct HotArgs {
  int64_t wpb;
  int64_t cap;
  int32_t W;
  int32_t fstar;   // used when params == nullptr
  int64_t r;       // used when params == nullptr
  int32_t passes;  // kHotWords-word passes per chunk
  int32_t nch;     // chunks (at most kHotMaxChunks)
};

__device__ __forceinline__ void bs_add(uint32_t (&pl)[kPlanes], uint32_t x) {
  uint32_t carry = x;
#pragma unroll
  for (int p = 0; p < kPlanes; ++p) {
    const uint32_t t = pl[p] & carry;
    pl[p] ^= carry;
    carry = t;
  }
}

// Masks of the nodes of a word whose freq is > f and == f.
__device__ __forceinline__ void bs_cmp(const uint32_t (&pl)[kPlanes], uint32_t f, uint32_t* gt,
                                       uint32_t* eq) {
  uint32_t g = 0u, e = 0xFFFFFFFFu;
#pragma unroll
  for (int p = kPlanes - 1; p >= 0; --p) {
    if ((f >> p) & 1u) {
      e &= pl[p];
    } else {
      g |= e & pl[p];
      e &= ~pl[p];
    }
  }
  *gt = g;
  *eq = e;
}

__device__ __forceinline__ uint32_t bs_freq(const uint32_t (&pl)[kPlanes], int bit) {
  uint32_t f = 0;
#pragma unroll
  for (int p = 0; p < kPlanes; ++p) f |= ((pl[p] >> bit) & 1u) << p;
  return f;
}

// Bits of word w that belong to remote nodes (owner != local).
__device__ __forceinline__ uint32_t remote_mask(const KPart& p, int64_t w) {
  if (p.local < 0) return 0xFFFFFFFFu;
  const int64_t u0 = w * 32;
  uint32_t local = 0;
  if (p.kind == GG_PART_MOD) {
    const int32_t r0 = (int32_t)(u0 - (int64_t)mod_div(p, (uint32_t)u0) * p.P);
    int j = p.local - r0;
    if (j < 0) j += p.P;
    for (; j < 32; j += p.P) local |= 1u << j;
  } else {
    const int64_t lo = p.start[p.local], hi = p.start[p.local + 1];
    const int64_t a = lo > u0 ? lo : u0;
    const int64_t b = hi < u0 + 32 ? hi : u0 + 32;
    if (b > a) {
      const int n = (int)(b - a), s = (int)(a - u0);
      local = (n == 32 ? 0xFFFFFFFFu : ((1u << n) - 1u)) << s;
    }
  }
  return ~local;
}

// One 32-node word per thread and pass: a block (chunk) covers `passes`
// runs of kHotWords consecutive words.  Chunks stay at most kHotMaxChunks,
// so every emit block can sum the counts of the chunks before it itself
// (at most 16 loads per thread and array); a 2.45M-node window is 304
// chunks of one pass, a 111M-node one 3,388 chunks of four.
constexpr int kHotWords = kBlock;
constexpr int kHotMaxIds = kHotWords * 32;  // ids one pass can emit
static_assert(kHotMaxChunks == 4096, "emit blocks sum at most 16 counts per thread");

// Sums word w of every batch's set into the planes, eight loads in flight.
__device__ __forceinline__ void load_planes(const uint32_t* bits, const HotArgs& a, int64_t w,
                                            uint32_t (&pl)[kPlanes]) {
#pragma unroll
  for (int p = 0; p < kPlanes; ++p) pl[p] = 0u;
  int32_t b = 0;
  for (; b + 8 <= a.W; b += 8) {
    uint32_t x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = bits[(int64_t)(b + j) * a.wpb + w];
#pragma unroll
    for (int j = 0; j < 8; ++j) bs_add(pl, x[j]);
  }
  for (; b < a.W; ++b) bs_add(pl, bits[(int64_t)b * a.wpb + w]);
}

// The planes of word w restricted to remote nodes.
__device__ __forceinline__ void remote_planes(const uint32_t* bits, const KPart& part,
                                              const HotArgs& a, int64_t w, uint32_t (&pl)[kPlanes]) {
  load_planes(bits, a, w, pl);
  const uint32_t m = remote_mask(part, w);
#pragma unroll
  for (int q = 0; q < kPlanes; ++q) pl[q] &= m;
}

// Per-chunk histogram of freq over the remote nodes of the window.
__global__ void __launch_bounds__(kBlock) k_hot_hist(const uint32_t* bits, KPart part, HotArgs a,
                                                     int32_t* chunk_hist) {
  __shared__ int32_t hist[GG_MAX_W + 2];
  for (int t = threadIdx.x; t < GG_MAX_W + 2; t += blockDim.x) hist[t] = 0;
  __syncthreads();
  const int c = blockIdx.x;
  for (int32_t q = 0; q < a.passes; ++q) {
    const int64_t w = ((int64_t)c * a.passes + q) * kHotWords + threadIdx.x;
    uint32_t pl[kPlanes];
    if (w < a.wpb) {
      remote_planes(bits, part, a, w, pl);
    } else {
#pragma unroll
      for (int p = 0; p < kPlanes; ++p) pl[p] = 0u;
    }
    for (int32_t f = 1; f <= a.W; ++f) {
      uint32_t g, e;
      bs_cmp(pl, (uint32_t)f, &g, &e);
      const int n = wave_sum(__popc(e));
      if (lane_id() == 0 && n) atomicAdd(&hist[f], n);
    }
  }
  __syncthreads();
  for (int t = threadIdx.x; t <= a.W; t += blockDim.x) chunk_hist[(int64_t)c * (a.W + 1) + t] = hist[t];
}

// One block: total histogram, then the threshold f* and remainder r.
// With den > 0 the budget is ceil(total * num / den) of the window's total
// distinct remote nodes (exact integer arithmetic).
__global__ void __launch_bounds__(1024) k_hot_select(const int32_t* chunk_hist, int32_t nch,
                                                     int32_t W, int64_t n_hot, int64_t num,
                                                     int64_t den, int64_t* params) {
  __shared__ int64_t hist[GG_MAX_W + 2];
  for (int t = threadIdx.x; t < GG_MAX_W + 2; t += blockDim.x) hist[t] = 0;
  __syncthreads();
  for (int32_t f = 1; f <= W; ++f) {
    int64_t v = 0;
    for (int64_t c = threadIdx.x; c < nch; c += blockDim.x) v += chunk_hist[c * (W + 1) + f];
    v = wave_sum(v);
    if (lane_id() == 0 && v) atomicAdd((unsigned long long*)&hist[f], (unsigned long long)v);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t total = 0;
    for (int32_t f = 1; f <= W; ++f) total += hist[f];
    if (den > 0) n_hot = (total * num + den - 1) / den;
    int64_t fstar = 0, r = 0;
    if (n_hot >= total) {
      fstar = 0;
    } else if (n_hot == 0) {
      fstar = W + 1;
    } else {
      int64_t cum = 0;
      for (int32_t f = W; f >= 1; --f) {
        if (cum + hist[f] >= n_hot) {
          fstar = f;
          r = n_hot - cum;
          break;
        }
        cum += hist[f];
      }
    }
    params[0] = fstar;
    params[1] = r;
  }
}

__device__ __forceinline__ void get_sel(const HotArgs& a, const int64_t* params, uint32_t* fstar,
                                        int64_t* r) {
  if (params) {
    *fstar = (uint32_t)params[0];
    *r = params[1];
  } else {
    *fstar = (uint32_t)a.fstar;
    *r = a.r;
  }
}

// Masks of the remote nodes of a word with freq > f* and freq == f*.
__device__ __forceinline__ void sel_masks(const uint32_t (&pl)[kPlanes], uint32_t fstar,
                                          uint32_t* gm, uint32_t* em) {
  bs_cmp(pl, fstar, gm, em);
  if (fstar == 0) *em = 0u;  // freq == 0 is not a member
}

// The planes of word w restricted to remote nodes, or none past the set.
__device__ __forceinline__ void word_masks(const uint32_t* bits, const KPart& part,
                                           const HotArgs& a, int64_t w, uint32_t fstar,
                                           uint32_t (&pl)[kPlanes], uint32_t* gm, uint32_t* em) {
  if (w < a.wpb) {
    remote_planes(bits, part, a, w, pl);
    sel_masks(pl, fstar, gm, em);
  } else {
#pragma unroll
    for (int p = 0; p < kPlanes; ++p) pl[p] = 0u;
    *gm = *em = 0u;
  }
}

// Per-chunk counts of nodes with freq > f* and freq == f*.
__global__ void __launch_bounds__(kBlock) k_hot_count(const uint32_t* bits, KPart part, HotArgs a,
                                                      const int64_t* params, int32_t* cnt_gt,
                                                      int32_t* cnt_eq) {
  __shared__ int32_t lds[2][kBlock / kWave];
  const int c = blockIdx.x;
  uint32_t fstar;
  int64_t r;
  get_sel(a, params, &fstar, &r);
  int ng = 0, ne = 0;
  for (int32_t q = 0; q < a.passes; ++q) {
    uint32_t pl[kPlanes], g, e;
    word_masks(bits, part, a, ((int64_t)c * a.passes + q) * kHotWords + threadIdx.x, fstar, pl,
               &g, &e);
    ng += __popc(g);
    ne += __popc(e);
  }
  ng = wave_sum(ng);
  ne = wave_sum(ne);
  if (lane_id() == 0) {
    lds[0][threadIdx.x / kWave] = ng;
    lds[1][threadIdx.x / kWave] = ne;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    cnt_gt[c] = lds[0][0] + lds[0][1] + lds[0][2] + lds[0][3];
    cnt_eq[c] = lds[1][0] + lds[1][1] + lds[1][2] + lds[1][3];
  }
}

// Sums of two values over the block.
__device__ __forceinline__ void block_sum2(int64_t& x, int64_t& y, int64_t (*lds)[2]) {
  x = wave_sum(x);
  y = wave_sum(y);
  const int w = threadIdx.x / kWave;
  if (lane_id() == 0) {
    lds[w][0] = x;
    lds[w][1] = y;
  }
  __syncthreads();
  x = y = 0;
  for (int q = 0; q < kBlock / kWave; ++q) {
    x += lds[q][0];
    y += lds[q][1];
  }
  __syncthreads();
}

// Writes the chunk's selected ids (and their freq) ascending.  The block
// first sums the counts of the chunks before its own (its place in the
// list; block 0 sums them all and writes the hot-set count).  Each thread
// owns one word per pass; a pass's ids are assembled in LDS at their
// block-local positions and then written out as one contiguous run.
__global__ void __launch_bounds__(kBlock) k_hot_emit(const uint32_t* bits, KPart part, HotArgs a,
                                                     const int64_t* params, const int32_t* cnt_gt,
                                                     const int32_t* cnt_eq, int32_t* hot_ids,
                                                     int32_t* hot_freq, int64_t* hot_count,
                                                     int32_t* status) {
  __shared__ int32_t s_out[kHotMaxIds];
  __shared__ int64_t lds[kBlock / kWave];
  __shared__ int64_t lds2[kBlock / kWave][2];
  const int c = blockIdx.x;
  uint32_t fstar;
  int64_t r;
  get_sel(a, params, &fstar, &r);
  // chunks before c (all chunks for block 0's totals)
  const int upto = c == 0 ? a.nch : c;
  int64_t pg = 0, pe = 0;
  for (int t = threadIdx.x; t < upto; t += kBlock) {
    pg += cnt_gt[t];
    pe += cnt_eq[t];
  }
  block_sum2(pg, pe, lds2);
  if (c == 0) {
    if (threadIdx.x == 0) {
      const int64_t total = pg + (pe < r ? pe : r);
      hot_count[0] = total < a.cap ? total : a.cap;
      hot_count[1] = total;
      if (total > a.cap) set_status(status, GG_DEV_CAPACITY);
    }
    pg = pe = 0;
  }
  int64_t eq_before = pe;                          // freq == f* ids before this pass
  int64_t pos0 = pg + (pe < r ? pe : r);           // output position of this pass
  for (int32_t q = 0; q < a.passes; ++q) {
    const int64_t w = ((int64_t)c * a.passes + q) * kHotWords + threadIdx.x;
    uint32_t pl[kPlanes], gm, em;
    word_masks(bits, part, a, w, fstar, pl, &gm, &em);
    const int ne = __popc(em);
    int64_t etot;
    // freq == f* nodes are taken in id order until r of them are in.
    const int64_t eq_rank0 = eq_before + block_excl_scan<kBlock>((int64_t)ne, lds, &etot);
    int64_t take = r - eq_rank0;
    take = take < 0 ? 0 : (take > ne ? ne : take);
    uint32_t sel = gm;
    for (uint32_t e = em; take > 0; --take) {
      sel |= e & (0u - e);  // lowest remaining id
      e &= e - 1u;
    }
    int64_t btot;
    const int64_t lpos = block_excl_scan<kBlock>((int64_t)__popc(sel), lds, &btot);
    for (int pass = 0; pass < (hot_freq ? 2 : 1); ++pass) {
      int32_t* dst = pass == 0 ? hot_ids : hot_freq;
      int64_t p = lpos;
      for (uint32_t m = sel; m; m &= m - 1u) {
        const int bit = __ffs(m) - 1;
        s_out[p++] = pass == 0 ? (int32_t)(w * 32 + bit) : (int32_t)bs_freq(pl, bit);
      }
      __syncthreads();
      for (int64_t i = threadIdx.x; i < btot; i += kBlock) {
        const int64_t o = pos0 + i;
        if (o < a.cap) dst[o] = s_out[i];
      }
      __syncthreads();
    }
    eq_before += etot;
    pos0 += btot;
  }
}

struct HotWs {
  int32_t* chunk_hist;
  int32_t* cnt_gt;
  int32_t* cnt_eq;
  int64_t* params;
};

// Passes per chunk and chunks for a window of num_nodes nodes.  The chunk
// limit is the tuning's hot_max_chunks (at most kHotMaxChunks); a lower one
// lets small graphs exercise multi-pass chunks, and the workspace layout
// depends on it.
void hot_chunks(int64_t num_nodes, const Tune& tune, int32_t* passes, int32_t* nch) {
  const int64_t runs = gg_bits_words(num_nodes) / kHotWords;
  const int64_t maxc = tune.hot_max_chunks;
  const int64_t p = std::max<int64_t>(1, cdiv(runs, maxc));
  *passes = (int32_t)p;
  *nch = (int32_t)cdiv(runs, p);
}

size_t hot_ws_layout(int64_t num_nodes, int32_t W, const Tune& tune, char* base, HotWs* out) {
  int32_t passes, nch;
  hot_chunks(num_nodes, tune, &passes, &nch);
  Carve cv{base, 0, ~(size_t)0};
  HotWs h;
  h.chunk_hist = cv.take<int32_t>((size_t)nch * (W + 1));
  h.cnt_gt = cv.take<int32_t>((size_t)nch);
  h.cnt_eq = cv.take<int32_t>((size_t)nch);
  h.params = cv.take<int64_t>(4);
  if (out) *out = h;
  return align_up(cv.used, 256);
}

}  // namespace
}  // namespace gg

using namespace gg;

extern "C" size_t gg_ws_hotset(int64_t num_nodes, int32_t W, const gg_tuning_t* tuning) {
  Tune tune;
  if (resolve_tuning(tuning, &tune) != GG_OK) return 0;
  return hot_ws_layout(num_nodes, W, tune, nullptr, nullptr);
}

extern "C" int gg_build_hotset(const uint32_t* frontier_bits_d, int32_t W, const gg_part_t* part,
                               int64_t n_hot, int64_t hot_num, int64_t hot_den,
                               int32_t* hot_ids_d, int32_t* hot_freq_d, int64_t cap,
                               int64_t* hot_count_d, const gg_tuning_t* tuning,
                               int32_t* status_d, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  GG_REQUIRE(frontier_bits_d && hot_count_d && status_d && (cap == 0 || hot_ids_d),
             "NULL argument");
  Tune tune;
  if (resolve_tuning(tuning, &tune) != GG_OK) return GG_ERR_ARG;
  GG_REQUIRE(W >= 1 && W <= GG_MAX_W, "W = %d outside 1..%d", W, GG_MAX_W);
  GG_REQUIRE(cap >= 0, "negative capacity");
  GG_REQUIRE(hot_den >= 0 && hot_den <= (1LL << 31), "hot_den %lld outside 0..2^31",
             (long long)hot_den);
  GG_REQUIRE(hot_den == 0 || (n_hot == -1 && hot_num >= 0 && hot_num <= hot_den),
             "a relative budget needs n_hot = -1 and 0 <= hot_num <= hot_den");
  GG_REQUIRE(aligned16(frontier_bits_d), "frontier_bits must be 16-byte aligned");
  KPart kp;
  int rc = pack_part(part, &kp);
  if (rc != GG_OK) return rc;
  GG_REQUIRE(kp.N >= 1, "empty graph");
  HotWs hw;
  const size_t need_ws = hot_ws_layout(kp.N, W, tune, (char*)ws, &hw);
  GG_REQUIRE(ws && ws_bytes >= need_ws, "workspace of %zu bytes < %zu", ws_bytes, need_ws);
  const int64_t wpb = gg_bits_words(kp.N);
  int32_t passes, nch;
  hot_chunks(kp.N, tune, &passes, &nch);
  HotArgs a;
  a.wpb = wpb;
  a.cap = cap;
  a.W = W;
  a.fstar = 0;
  a.r = 0;
  a.passes = passes;
  a.nch = nch;
  const int64_t* params = nullptr;
  if (n_hot == 0) {
    a.fstar = W + 1;
  } else if (n_hot > 0 || hot_den > 0) {
    hipLaunchKernelGGL(k_hot_hist, dim3(nch), dim3(kBlock), 0, stream, frontier_bits_d, kp, a,
                       hw.chunk_hist);
    GG_LAUNCH_CHECK("k_hot_hist");
    hipLaunchKernelGGL(k_hot_select, dim3(1), dim3(1024), 0, stream, hw.chunk_hist, nch, W, n_hot,
                       hot_num, hot_den, hw.params);
    GG_LAUNCH_CHECK("k_hot_select");
    params = hw.params;
  }
  hipLaunchKernelGGL(k_hot_count, dim3(nch), dim3(kBlock), 0, stream, frontier_bits_d, kp, a, params,
                     hw.cnt_gt, hw.cnt_eq);
  GG_LAUNCH_CHECK("k_hot_count");
  hipLaunchKernelGGL(k_hot_emit, dim3(nch), dim3(kBlock), 0, stream, frontier_bits_d, kp, a, params,
                     hw.cnt_gt, hw.cnt_eq, hot_ids_d, hot_freq_d, hot_count_d, status_d);
  GG_LAUNCH_CHECK("k_hot_emit");
  return GG_OK;
}
