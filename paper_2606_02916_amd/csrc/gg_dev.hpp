// Device-side building blocks of libgg (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "copy_geom.hpp"
#include "gg.h"

namespace gg {

constexpr int kWave = 64;
constexpr int kBlock = 256;                  // 4 wavefronts
constexpr int kChunkWords = 2048;            // bit-set words per compaction block
constexpr int kWordsPerThread = kChunkWords / kBlock;

// ---------------------------------------------------------------------------
// Partition book, passed by value.  MOD uses a multiply-shift for u div P
// (exact for u < 2^34 and P <= 64); RANGE finds the last start <= u by a
// binary search over the P starts (the table is padded with N up to 64).
// ---------------------------------------------------------------------------
struct KPart {
  int32_t P;
  int32_t kind;
  int32_t local;
  int32_t step0;  // RANGE: largest power of two <= max(P - 1, 1)
  int64_t N;
  uint64_t div_magic;
  int64_t start[GG_MAX_PARTS + 1];  // entries past P hold N
};

__device__ __forceinline__ int32_t mod_div(const KPart& p, uint32_t u) {
  return (int32_t)(((uint64_t)u * p.div_magic) >> 40);
}

// start: the 65-entry table (kernarg or LDS copy).
__device__ __forceinline__ int32_t owner_of(const KPart& p, const int64_t* start, int32_t u) {
  if (p.kind == GG_PART_MOD) {
    const int32_t q = mod_div(p, (uint32_t)u);
    return u - q * p.P;
  }
  int32_t idx = 0;
  for (int step = p.step0; step >= 1; step >>= 1)
    if (start[idx + step] <= (int64_t)u) idx += step;
  return idx;
}

__device__ __forceinline__ int64_t row_of(const KPart& p, const int64_t* start, int32_t u,
                                          int32_t owner) {
  if (p.kind == GG_PART_MOD) return (int64_t)mod_div(p, (uint32_t)u);
  return (int64_t)u - start[owner];
}

// ---------------------------------------------------------------------------
// Feature shards, passed by value.
// ---------------------------------------------------------------------------
struct KFeat {
  int32_t row_bytes;
  int32_t P;
  const char* shard[GG_MAX_PARTS];
  int64_t stride[GG_MAX_PARTS];
  int64_t rows[GG_MAX_PARTS];
};

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC'11): ten rounds of two
// 32x32->64 multiplies; the key advances by the Weyl increments each round.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t lo0 = M0 * c.x, hi0 = __umulhi(M0, c.x);
    const uint32_t lo1 = M1 * c.z, hi1 = __umulhi(M1, c.z);
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    k0 += W0;
    k1 += W1;
  }
  return c;
}

__device__ __forceinline__ void set_status(int32_t* status, int32_t bits) {
  atomicOr(status, bits);
}

// ---------------------------------------------------------------------------
// Wave and block primitives.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

// Number of set bits of `mask` in lanes below this one.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Lane index of the (r+1)-th set bit of mask (r < popcount(mask)).
__device__ __forceinline__ int nth_set_lane(uint64_t mask, int r) {
  int lo = 0;
#pragma unroll
  for (int w = 32; w >= 1; w >>= 1) {
    // set bits below lane lo + w
    const uint64_t below = (lo + w >= 64) ? mask : (mask & ((1ull << (lo + w)) - 1ull));
    if (__popcll(below) <= r) lo += w;
  }
  return lo;
}

template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v) {
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const T t = __shfl_up(v, o, kWave);
    if (lane >= o) v += t;
  }
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = kWave / 2; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Exclusive scan over a block of NT threads; lds must hold NT/64 entries.
// Every thread of the block must call it.
template <int NT, typename T>
__device__ __forceinline__ T block_excl_scan(T v, T* lds, T* total) {
  constexpr int NW = NT / kWave;
  const int wid = (int)threadIdx.x / kWave;
  const T inc = wave_incl_scan(v);
  if (lane_id() == kWave - 1) lds[wid] = inc;
  __syncthreads();
  T base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const T x = lds[w];
    base += (w < wid) ? x : (T)0;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return base + inc - v;
}

// Exclusive scan of in[0..n) into out[0..n) plus `base`, by one block of
// NT threads, 16 consecutive items per thread per tile; lds holds NT/64
// entries.  Returns the sum.
template <int NT = 1024>
__device__ __forceinline__ int64_t block_scan_large(const int32_t* in, int64_t* out, int64_t n,
                                                    int64_t base, int64_t* lds16) {
  constexpr int IT = 16;
  int64_t carry = base;
  for (int64_t t0 = 0; t0 < n; t0 += (int64_t)NT * IT) {
    int32_t loc[IT];
    int64_t sum = 0;
    const int64_t i0 = t0 + (int64_t)threadIdx.x * IT;
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int64_t i = i0 + j;
      loc[j] = i < n ? in[i] : 0;
      sum += loc[j];
    }
    int64_t tot;
    const int64_t ex = block_excl_scan<NT>(sum, lds16, &tot);
    int64_t run = carry + ex;
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int64_t i = i0 + j;
      if (i < n) out[i] = run;
      run += loc[j];
    }
    carry += tot;
  }
  return carry - base;
}

// hist[key] += number of active lanes with `valid` and that key: one LDS
// atomic per distinct key present in the wave.  Call from every active lane.
__device__ __forceinline__ void wave_hist_add(int32_t* hist, bool valid, int32_t key) {
  const int lane = lane_id();
  for (uint64_t act = __ballot(valid); act;) {
    const int leader = __ffsll((unsigned long long)act) - 1;
    const int32_t kl = __shfl(key, leader, kWave);
    const uint64_t sel = __ballot(valid && key == kl);
    if (lane == leader) atomicAdd(&hist[kl], (int32_t)__popcll(sel));
    act &= ~sel;
  }
}

// ---------------------------------------------------------------------------
// Row copy engine.  A wavefront copies up to 64 rows: lane r supplies the
// source of row r (nullptr = skip that row) and the rows land at
// dst0 + r * dst_stride.  The row bytes are cut into VB-byte chunks that are
// spread over the wave, so consecutive lanes move consecutive chunks of one
// row and then of the next: every load and store instruction covers a
// contiguous run of up to 1 KB, and short rows do not leave lanes idle.
// Chunk c belongs to row c / cpr, computed by chunk_row (copy_geom.hpp).
// ---------------------------------------------------------------------------
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ void st16(char* p, u32x4 v) {
  if (NT)
    __builtin_nontemporal_store(v, (u32x4*)p);
  else
    *(u32x4*)p = v;
}

template <bool NT>
__device__ __forceinline__ void st4(char* p, uint32_t v) {
  if (NT)
    __builtin_nontemporal_store(v, (uint32_t*)p);
  else
    *(uint32_t*)p = v;
}

template <int VB, bool NT, int U = (VB == 16 ? 4 : 8)>
__device__ __forceinline__ void wave_copy_rows(const char* src, char* dst0, int64_t dst_stride,
                                               int nrows, const CopyGeom& g) {
  const int lane = lane_id();
  const uint32_t total = (uint32_t)nrows * g.cpr;
  const long long srcl = (long long)src;
  for (uint32_t base = 0; base < total; base += kWave * U) {
    if (VB == 16) {
      // Destinations are recomputed at the stores: holding U 64-bit
      // pointers across the loads would cost 2U registers.
      u32x4 v[U];
      bool ok[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const uint32_t c = base + (uint32_t)(j * kWave + lane);
        const uint32_t r = chunk_row(c, g.magic);
        const uint32_t col = c - r * g.cpr;
        const char* sp = (const char*)__shfl(srcl, (int)(r & 63u), kWave);
        ok[j] = (c < total) && (sp != nullptr);
        if (ok[j]) v[j] = *(const u32x4*)(sp + (int64_t)col * 16);
      }
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const uint32_t c = base + (uint32_t)(j * kWave + lane);
        const uint32_t r = chunk_row(c, g.magic);
        const uint32_t col = c - r * g.cpr;
        if (ok[j]) st16<NT>(dst0 + (int64_t)r * dst_stride + (int64_t)col * 16, v[j]);
      }
    } else {
      uint32_t v[U];
      char* dp[U];
      bool ok[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const uint32_t c = base + (uint32_t)(j * kWave + lane);
        const uint32_t r = chunk_row(c, g.magic);
        const uint32_t col = c - r * g.cpr;
        const char* sp = (const char*)__shfl(srcl, (int)(r & 63u), kWave);
        ok[j] = (c < total) && (sp != nullptr);
        dp[j] = dst0 + (int64_t)r * dst_stride + (int64_t)col * 4;
        if (ok[j]) v[j] = *(const uint32_t*)(sp + (int64_t)col * 4);
      }
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (ok[j]) st4<NT>(dp[j], v[j]);
    }
  }
  if (VB == 16 && g.tail) {
    const uint32_t ttotal = (uint32_t)nrows * g.tail;
    const int64_t off0 = (int64_t)g.cpr * 16;
    for (uint32_t base = 0; base < ttotal; base += kWave) {
      const uint32_t c = base + (uint32_t)lane;
      const uint32_t r = chunk_row(c, g.tmagic);
      const uint32_t w = c - r * g.tail;
      const char* sp = (const char*)__shfl(srcl, (int)(r & 63u), kWave);
      if (c < ttotal && sp != nullptr) {
        const uint32_t v = *(const uint32_t*)(sp + off0 + (int64_t)w * 4);
        st4<NT>(dst0 + (int64_t)r * dst_stride + off0 + (int64_t)w * 4, v);
      }
    }
  }
}

// As wave_copy_rows, with a destination per row: lane r supplies both the
// source and the destination of row r (a nullptr source skips the row).
template <int VB, bool NT, int U = (VB == 16 ? 4 : 8)>
__device__ __forceinline__ void wave_copy_rows_to(const char* src, char* dst, int nrows,
                                                  const CopyGeom& g) {
  const int lane = lane_id();
  const uint32_t total = (uint32_t)nrows * g.cpr;
  const long long srcl = (long long)src, dstl = (long long)dst;
  for (uint32_t base = 0; base < total; base += kWave * U) {
    if (VB == 16) {
      u32x4 v[U];
      char* dp[U];
      bool ok[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const uint32_t c = base + (uint32_t)(j * kWave + lane);
        const uint32_t r = chunk_row(c, g.magic);
        const uint32_t col = c - r * g.cpr;
        const char* sp = (const char*)__shfl(srcl, (int)(r & 63u), kWave);
        dp[j] = (char*)__shfl(dstl, (int)(r & 63u), kWave) + (int64_t)col * 16;
        ok[j] = (c < total) && (sp != nullptr);
        if (ok[j]) v[j] = *(const u32x4*)(sp + (int64_t)col * 16);
      }
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (ok[j]) st16<NT>(dp[j], v[j]);
    } else {
      uint32_t v[U];
      char* dp[U];
      bool ok[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const uint32_t c = base + (uint32_t)(j * kWave + lane);
        const uint32_t r = chunk_row(c, g.magic);
        const uint32_t col = c - r * g.cpr;
        const char* sp = (const char*)__shfl(srcl, (int)(r & 63u), kWave);
        dp[j] = (char*)__shfl(dstl, (int)(r & 63u), kWave) + (int64_t)col * 4;
        ok[j] = (c < total) && (sp != nullptr);
        if (ok[j]) v[j] = *(const uint32_t*)(sp + (int64_t)col * 4);
      }
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (ok[j]) st4<NT>(dp[j], v[j]);
    }
  }
  if (VB == 16 && g.tail) {
    const uint32_t ttotal = (uint32_t)nrows * g.tail;
    const int64_t off0 = (int64_t)g.cpr * 16;
    for (uint32_t base = 0; base < ttotal; base += kWave) {
      const uint32_t c = base + (uint32_t)lane;
      const uint32_t r = chunk_row(c, g.tmagic);
      const uint32_t w = c - r * g.tail;
      const char* sp = (const char*)__shfl(srcl, (int)(r & 63u), kWave);
      char* dp = (char*)__shfl(dstl, (int)(r & 63u), kWave);
      if (c < ttotal && sp != nullptr) {
        const uint32_t v = *(const uint32_t*)(sp + off0 + (int64_t)w * 4);
        st4<NT>(dp + off0 + (int64_t)w * 4, v);
      }
    }
  }
}

}  // namespace gg
