// The consumer of X_b: GraphSAGE layers with the mean aggregator over the
// sampled blocks of a window (Algorithm 1 forward pass; Sec. VI-A model).
//
// Each layer runs as two launches over all W batches at once:
//  * k_sage_project: Z = H [W_self | W_neigh] for every input row, a dense
//    fp32 product on MFMA (v_mfma_f32_16x16x4f32).  Each wave owns 16 rows
//    and loads them straight into registers, 16 bytes per lane; the weights
//    sit in LDS;
//  * k_sage_aggregate: out_v = act(Z_self[v] + mean_{u in S(v)} Z_neigh[u] +
//    bias).  The mean commutes with the linear map, so averaging the
//    projected rows (d_out wide) equals projecting the averaged input rows
//    (d_in wide) up to rounding, and reads 64-byte rows instead of d_in-wide
//    ones.
// A node's row in the input level is its position in that level's ascending
// frontier.  For the first layer (input level N_b) the position is a rank in
// the batch's N_b bit set: a prefix count per word (k_rank_local,
// k_rank_chunks) plus a popcount.  Deeper layers binary-search the (small)
// frontier.  Nothing of size N per level is needed.
#include <hip/hip_fp16.h>

#include "gg_host.hpp"

namespace gg {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kSageBlock = 256;          // 4 waves
constexpr int kTileRows = 64;            // 16 rows per wave
constexpr int kWLdsFloats = 16384;       // 64 KB of weights in LDS at most
constexpr int kRankChunk = 2048;         // bit-set words per rank chunk (divides gg_bits_words)

// ---------------------------------------------------------------------------
// Rank of a node in its batch's N_b bit set.
// ---------------------------------------------------------------------------

// rank[w] = {set bits of the words before w inside w's chunk, word w}: the
// word travels with its prefix so that a rank lookup is one 8-byte load;
// csum[b][c] = bits of chunk c of batch b.
__global__ void __launch_bounds__(kSageBlock) k_rank_local(const uint32_t* bits, int64_t wpb,
                                                           int64_t nch, int2* rank,
                                                           int32_t* csum) {
  __shared__ int32_t lds[kSageBlock / kWave];
  const int b = blockIdx.y;
  const int64_t c = blockIdx.x;
  const int64_t w0 = (int64_t)b * wpb + c * kRankChunk + (int64_t)threadIdx.x * 8;
  uint32_t wd[8];
  int32_t s = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    wd[j] = bits[w0 + j];
    s += __popc(wd[j]);
  }
  int32_t tot;
  int32_t run = block_excl_scan<kSageBlock>(s, lds, &tot);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    rank[w0 + j] = make_int2(run, (int32_t)wd[j]);
    run += __popc(wd[j]);
  }
  if (threadIdx.x == 0) csum[(int64_t)b * nch + c] = tot;
}

// Exclusive scan of each batch's chunk counts, in place.
__global__ void __launch_bounds__(kSageBlock) k_rank_chunks(int32_t* csum, int64_t nch) {
  __shared__ int32_t lds[kSageBlock / kWave];
  int32_t* cs = csum + (int64_t)blockIdx.x * nch;
  int32_t carry = 0;
  for (int64_t i0 = 0; i0 < nch; i0 += kSageBlock) {
    const int64_t i = i0 + threadIdx.x;
    const int32_t v = i < nch ? cs[i] : 0;
    int32_t tot;
    const int32_t ex = block_excl_scan<kSageBlock>(v, lds, &tot);
    if (i < nch) cs[i] = carry + ex;
    carry += tot;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Projection Z = H [W_self | W_neigh] on MFMA.
// ---------------------------------------------------------------------------
struct ProjArgs {
  const char* h;        // input rows of the level, back to back
  int64_t h_stride;     // bytes
  int32_t K;            // d_in
  int32_t K16;          // K rounded up to 16
  int32_t kc;           // weight rows per LDS chunk (multiple of 16)
  int32_t d_out;
  int32_t ldz;          // floats per Z row (NT * 16)
  const float* w_self;  // [K][d_out]
  const float* w_neigh;
  float* z;
  const int64_t* off;   // frontier_off
  int64_t seg0;         // first segment of the input level
  int32_t W;
  int64_t rows_cap;
};

// Four consecutive elements of a row starting at column c (zero past K).
template <int XT, bool VEC>
__device__ __forceinline__ f32x4 load4(const char* row, int c, int K) {
  f32x4 v = {0.f, 0.f, 0.f, 0.f};
  if (VEC && c + 3 < K) {
    if (XT == GG_F32) {
      v = *(const f32x4*)(row + (int64_t)c * 4);
    } else {
      const __half2* p = (const __half2*)(row + (int64_t)c * 2);
      const float2 lo = __half22float2(p[0]), hi = __half22float2(p[1]);
      v = f32x4{lo.x, lo.y, hi.x, hi.y};
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (c + e < K)
        v[e] = XT == GG_F32 ? ((const float*)row)[c + e]
                            : __half2float(((const __half*)row)[c + e]);
  }
  return v;
}

// The contraction over K is evaluated in a permuted order: in the 16-column
// group q, lane group g = lane / 16 holds columns q + 4g .. q + 4g + 3 of its
// row (one 16-byte load) and feeds them to four MFMA steps, while the B
// operand of lane 16g + j is the weight row with the same column index.
// Every product A[i][k] B[k][j] is taken exactly once.
template <int NT, int XT, bool VEC>
__global__ void __launch_bounds__(kSageBlock) k_sage_project(ProjArgs a, int32_t* status) {
  extern __shared__ float Ws[];   // a.kc rows of NT * 16 weights
  constexpr int ncol = NT * 16;
  int64_t n = a.off[a.seg0 + a.W] - a.off[a.seg0];
  if (n > a.rows_cap) {
    if (blockIdx.x == 0 && threadIdx.x == 0) set_status(status, GG_DEV_CAPACITY);
    n = a.rows_cap;
  }
  const int lane = lane_id();
  const int wv = (int)threadIdx.x / kWave;
  const int g = lane >> 4, il = lane & 15;
  const int n2 = 2 * a.d_out;
  const bool whole = a.kc >= a.K16;
  auto load_w = [&](int k0) {
    for (int e = threadIdx.x; e < a.kc * ncol; e += kSageBlock) {
      const int kk = e / ncol, c = e - kk * ncol;
      const int k = k0 + kk;
      float v = 0.f;
      if (k < a.K) {
        if (c < a.d_out)
          v = a.w_self[(int64_t)k * a.d_out + c];
        else if (c < n2)
          v = a.w_neigh[(int64_t)k * a.d_out + (c - a.d_out)];
      }
      Ws[e] = v;
    }
  };
  if (whole) {
    load_w(0);
    __syncthreads();
  }
  for (int64_t row0 = (int64_t)blockIdx.x * kTileRows; row0 < n;
       row0 += (int64_t)gridDim.x * kTileRows) {
    const int64_t r = row0 + wv * 16 + il;
    const bool rok = r < n;
    const char* rp = a.h + (rok ? r : 0) * a.h_stride;
    f32x4 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < a.K16; k0 += a.kc) {
      if (!whole) {
        __syncthreads();
        load_w(k0);
        __syncthreads();
      }
      const int kend = a.K16 - k0 < a.kc ? a.K16 - k0 : a.kc;
      constexpr int U = 4;   // 16-column groups whose loads are issued together
      for (int q = 0; q < kend; q += 16 * U) {
        f32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int qq = q + 16 * u;
          v[u] = (rok && qq < kend) ? load4<XT, VEC>(rp, k0 + qq + 4 * g, a.K)
                                    : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int qq = q + 16 * u;
          if (qq >= kend) break;
          const float* wrow = Ws + (int64_t)(qq + 4 * g) * ncol + il;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
#pragma unroll
            for (int t = 0; t < NT; ++t)
              acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(v[u][e], wrow[e * ncol + t * 16],
                                                            acc[t], 0, 0, 0);
          }
        }
      }
    }
    // D[i][j] of tile t sits in lane 16 * (i / 4) + j, element i % 4.
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int col = t * 16 + il;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int64_t row = row0 + wv * 16 + 4 * g + rr;
        if (row < n && col < n2) a.z[row * a.ldz + col] = acc[t][rr];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Mean aggregation of the projected rows.
// ---------------------------------------------------------------------------
struct AggArgs {
  const int32_t* fids;
  const int64_t* off;
  const int32_t* nbr;
  const int64_t* noff;
  int32_t W;
  int32_t lvl;          // output level; the input level is lvl + 1
  int32_t k;            // fanout of hop lvl
  const float* z;
  int32_t ldz;
  int32_t d_out;
  const float* bias;
  int32_t relu;
  float* out;           // output rows of level lvl, back to back, d_out floats each
  int64_t z_cap;        // rows of z that were computed
  int64_t out_cap;
  // rank lookup in the N_b bit sets (input level = N_b), else binary search
  int32_t use_rank;
  const int2* rank;     // {prefix in chunk, word} per bit-set word
  const int32_t* cpre;
  int64_t wpb;
  int64_t nch;
};

__device__ __forceinline__ int64_t find_sorted(const int32_t* a, int64_t n, int32_t v) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (a[mid] < v)
      lo = mid + 1;
    else
      hi = mid;
  }
  return (lo < n && a[lo] == v) ? lo : -1;
}

__device__ __forceinline__ int32_t row_in_level(const AggArgs& a, int b, const int32_t* Fin,
                                                int64_t nin, int32_t u) {
  int64_t p;
  if (a.use_rank) {
    const int64_t wi = (int64_t)(uint32_t)u >> 5;
    if (u < 0 || wi >= a.wpb) return -1;
    const int64_t w = (int64_t)b * a.wpb + wi;
    const int2 rw = a.rank[w];
    const int32_t cpre = a.cpre[(int64_t)b * a.nch + wi / kRankChunk];
    const uint32_t word = (uint32_t)rw.y, bit = 1u << (u & 31);
    if (!(word & bit)) return -1;
    p = (int64_t)rw.x + cpre + __popc(word & (bit - 1u));
    if (p >= nin) return -1;
  } else {
    p = find_sorted(Fin, nin, u);
  }
  return (int32_t)p;
}

// Grid (blocks, W): block column b serves batch b.  Sixteen lanes per output
// node: lane j of the group resolves neighbour slots j and j + 16, then the
// group sums the projected neighbour rows, 16 columns at a time.  The
// neighbour loop is unrolled to KMAX >= k so that all of a column's row
// loads are in flight together; the sum still runs in slot order.
template <int KMAX>
__global__ void __launch_bounds__(kSageBlock) k_sage_aggregate(AggArgs a, int32_t* status) {
  const int b = blockIdx.y;
  const int64_t sout = (int64_t)a.lvl * a.W + b, sin = sout + a.W;
  const int64_t o0 = a.off[sout], nout = a.off[sout + 1] - o0;
  const int64_t i0 = a.off[sin], nin = a.off[sin + 1] - i0;
  const int64_t orow0 = o0 - a.off[(int64_t)a.lvl * a.W];
  const int64_t zrow0 = i0 - a.off[(int64_t)(a.lvl + 1) * a.W];
  const int32_t* Fin = a.fids + i0;
  const int32_t* Fout = a.fids + o0;
  const int32_t* S = a.nbr + a.noff[sout];
  const int64_t nslots = a.noff[sout + 1] - a.noff[sout];   // nout * k unless clamped
  const int lane = lane_id();
  const int sub = (int)threadIdx.x >> 4, sl = (int)threadIdx.x & 15;
  const int gbase = lane & 48;   // first lane of this group within the wave
  int32_t st = 0;
  for (int64_t i = (int64_t)blockIdx.x * (kSageBlock / 16) + sub; i < nout;
       i += (int64_t)gridDim.x * (kSageBlock / 16)) {
    int32_t pv = row_in_level(a, b, Fin, nin, Fout[i]);
    int32_t p0 = -1, p1 = -1;
    if (sl < a.k && i * a.k + sl < nslots) {
      const int32_t u = S[i * a.k + sl];
      if (u >= 0) {
        p0 = row_in_level(a, b, Fin, nin, u);
        if (p0 < 0) st |= GG_DEV_BAD_ID;
      }
    }
    if (sl + 16 < a.k && i * a.k + sl + 16 < nslots) {
      const int32_t u = S[i * a.k + sl + 16];
      if (u >= 0) {
        p1 = row_in_level(a, b, Fin, nin, u);
        if (p1 < 0) st |= GG_DEV_BAD_ID;
      }
    }
    if (pv < 0) st |= GG_DEV_BAD_ID;
    if (zrow0 + pv >= a.z_cap) pv = -1;
    if (p0 >= 0 && zrow0 + p0 >= a.z_cap) p0 = -1;
    if (p1 >= 0 && zrow0 + p1 >= a.z_cap) p1 = -1;
    int32_t pt[KMAX];
    int cnt = 0;
#pragma unroll
    for (int t = 0; t < KMAX; ++t) {
      pt[t] = __shfl(t < 16 ? p0 : p1, gbase + (t & 15), kWave);
      if (t >= a.k) pt[t] = -1;
      cnt += pt[t] >= 0;
    }
    const float inv = cnt ? 1.0f / (float)cnt : 0.f;
    const int64_t orow = orow0 + i;
    for (int c0 = 0; c0 < a.d_out; c0 += 16) {
      const int c = c0 + sl;
      const bool cok = c < a.d_out;
      const float self = (cok && pv >= 0) ? a.z[(zrow0 + pv) * a.ldz + c] : 0.f;
      float v[KMAX];
#pragma unroll
      for (int t = 0; t < KMAX; ++t)
        v[t] = (cok && pt[t] >= 0) ? a.z[(zrow0 + pt[t]) * a.ldz + a.d_out + c] : 0.f;
      float sum = 0.f;
#pragma unroll
      for (int t = 0; t < KMAX; ++t)
        if (pt[t] >= 0) sum += v[t];
      if (cok && pv >= 0) {
        float y = self + sum * inv + (a.bias ? a.bias[c] : 0.f);
        if (a.relu && y < 0.f) y = 0.f;
        if (orow < a.out_cap) a.out[orow * a.d_out + c] = y;
      }
    }
    if (orow >= a.out_cap) st |= GG_DEV_CAPACITY;
  }
  if (st) set_status(status, st);
}

int ldz_tiles(int32_t d_out) {
  const int need = (2 * d_out + 15) / 16;
  int nt = 1;
  while (nt < need) nt <<= 1;
  return nt;
}

struct SageWs {
  float* z;
  float* h[2];
  int2* rank;
  int32_t* csum;
};

size_t sage_ws_layout(int64_t num_nodes, int32_t W, int64_t rows_cap, int32_t L,
                      const gg_sage_layer_t* layers, char* base, SageWs* out) {
  int32_t dmax = 1, ntmax = 1;
  for (int32_t j = 0; j < L; ++j) {
    dmax = std::max(dmax, layers[j].d_out);
    ntmax = std::max(ntmax, ldz_tiles(layers[j].d_out));
  }
  const size_t r = (size_t)std::max<int64_t>(rows_cap, 1);
  const int64_t wpb = gg_bits_words(num_nodes);
  const int64_t nch = wpb / kRankChunk;
  Carve cv{base, 0, ~(size_t)0};
  float* z = cv.take<float>(r * (size_t)ntmax * 16);
  float* h0 = cv.take<float>(r * (size_t)dmax);
  float* h1 = cv.take<float>(r * (size_t)dmax);
  int2* rank = cv.take<int2>((size_t)W * (size_t)wpb);
  int32_t* csum = cv.take<int32_t>((size_t)W * (size_t)std::max<int64_t>(nch, 1));
  if (out) *out = SageWs{z, {h0, h1}, rank, csum};
  return align_up(cv.used, 256);
}

template <int NT, int XT>
void launch_project_v(bool vec, const ProjArgs& a, int grid, size_t lds, int32_t* status,
                      hipStream_t stream) {
  if (vec)
    hipLaunchKernelGGL((k_sage_project<NT, XT, true>), dim3(grid), dim3(kSageBlock), lds, stream,
                       a, status);
  else
    hipLaunchKernelGGL((k_sage_project<NT, XT, false>), dim3(grid), dim3(kSageBlock), lds, stream,
                       a, status);
}

template <int NT>
void launch_project(int xt, bool vec, const ProjArgs& a, int grid, size_t lds, int32_t* status,
                    hipStream_t stream) {
  if (xt == GG_F32)
    launch_project_v<NT, GG_F32>(vec, a, grid, lds, status, stream);
  else
    launch_project_v<NT, GG_F16>(vec, a, grid, lds, status, stream);
}

}  // namespace
}  // namespace gg

using namespace gg;

extern "C" size_t gg_ws_sage(int64_t num_nodes, int32_t W, int64_t rows_cap, int32_t L,
                             const gg_sage_layer_t* layers_h) {
  if (num_nodes < 1 || W < 1 || W > GG_MAX_W || rows_cap < 0 || L < 1 || L > GG_MAX_LAYERS ||
      !layers_h)
    return 0;
  return sage_ws_layout(num_nodes, W, rows_cap, L, layers_h, nullptr, nullptr);
}

extern "C" int gg_sage_forward(const gg_wsample_t* smp, int64_t num_nodes, int32_t W, int32_t L,
                               const int32_t* fanout_h, const void* x_d, int32_t x_dtype,
                               int64_t x_stride, int64_t rows_cap, const gg_sage_layer_t* layers_h,
                               float* out_d, int64_t out_rows_cap, int32_t* status_d, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  GG_REQUIRE(smp && fanout_h && x_d && layers_h && out_d && status_d, "NULL argument");
  GG_REQUIRE(smp->frontier_ids && smp->frontier_off && smp->nbr_ids && smp->nbr_off &&
                 smp->frontier_bits,
             "sampling outputs are NULL");
  GG_REQUIRE(num_nodes >= 1 && num_nodes <= INT32_MAX, "num_nodes %lld invalid",
             (long long)num_nodes);
  GG_REQUIRE(W >= 1 && W <= GG_MAX_W, "W = %d outside 1..%d", W, GG_MAX_W);
  GG_REQUIRE(L >= 1 && L <= GG_MAX_LAYERS, "L = %d outside 1..%d", L, GG_MAX_LAYERS);
  GG_REQUIRE(x_dtype == GG_F32 || x_dtype == GG_F16, "x_dtype %d unsupported", x_dtype);
  GG_REQUIRE(rows_cap >= 0 && out_rows_cap >= 0, "negative capacity");
  const int64_t esz = x_dtype == GG_F32 ? 4 : 2;
  GG_REQUIRE(((uintptr_t)x_d % esz) == 0 && x_stride % esz == 0, "x is not %lld-byte aligned",
             (long long)esz);
  for (int32_t l = 0; l < L; ++l)
    GG_REQUIRE(fanout_h[l] >= 1 && fanout_h[l] <= GG_MAX_FANOUT, "fanout[%d] = %d invalid", l,
               fanout_h[l]);
  for (int32_t j = 0; j < L; ++j) {
    const gg_sage_layer_t& ly = layers_h[j];
    GG_REQUIRE(ly.w_self && ly.w_neigh, "layer %d weights are NULL", j);
    GG_REQUIRE(ly.d_out >= 1 && ly.d_out <= GG_SAGE_MAX_DIM, "layer %d: d_out = %d outside 1..%d",
               j, ly.d_out, GG_SAGE_MAX_DIM);
    if (j == 0)
      GG_REQUIRE(ly.d_in >= 1 && ly.d_in <= GG_SAGE_MAX_IN && ly.d_in * esz <= x_stride,
                 "layer 0: d_in = %d does not fit rows of %lld bytes", ly.d_in,
                 (long long)x_stride);
    else
      GG_REQUIRE(ly.d_in == layers_h[j - 1].d_out, "layer %d: d_in %d != previous d_out %d", j,
                 ly.d_in, layers_h[j - 1].d_out);
  }
  GG_REQUIRE(aligned16(smp->frontier_bits), "frontier_bits must be 16-byte aligned");
  const size_t need = sage_ws_layout(num_nodes, W, rows_cap, L, layers_h, nullptr, nullptr);
  GG_REQUIRE(ws && ws_bytes >= need, "workspace of %zu bytes < %zu", ws_bytes, need);
  SageWs sw;
  sage_ws_layout(num_nodes, W, rows_cap, L, layers_h, (char*)ws, &sw);
  const int64_t wpb = gg_bits_words(num_nodes);
  const int64_t nch = wpb / kRankChunk;

  // ranks in the N_b bit sets
  hipLaunchKernelGGL(k_rank_local, dim3((unsigned)nch, W), dim3(kSageBlock), 0, stream,
                     smp->frontier_bits, wpb, nch, sw.rank, sw.csum);
  GG_LAUNCH_CHECK("k_rank_local");
  hipLaunchKernelGGL(k_rank_chunks, dim3(W), dim3(kSageBlock), 0, stream, sw.csum, nch);
  GG_LAUNCH_CHECK("k_rank_chunks");

  const int proj_grid = (int)std::min<int64_t>(std::max<int64_t>(cdiv(rows_cap, kTileRows), 1), 8192);
  const int agg_bx = (int)std::min<int64_t>(
      std::max<int64_t>(cdiv(rows_cap, (int64_t)W * (kSageBlock / 16)), 1), 1024);
  for (int32_t j = 1; j <= L; ++j) {
    const gg_sage_layer_t& ly = layers_h[j - 1];
    const int32_t lvl = L - j;
    ProjArgs pa;
    int xt;
    if (j == 1) {
      pa.h = (const char*)x_d;
      pa.h_stride = x_stride;
      xt = x_dtype;
    } else {
      pa.h = (const char*)sw.h[(j - 2) & 1];
      pa.h_stride = (int64_t)layers_h[j - 2].d_out * 4;
      xt = GG_F32;
    }
    const int vb = xt == GG_F32 ? 16 : 8;   // bytes of four elements
    const bool vec = ((uintptr_t)pa.h % vb) == 0 && pa.h_stride % vb == 0;
    const int nt = ldz_tiles(ly.d_out);
    pa.K = ly.d_in;
    pa.K16 = (ly.d_in + 15) / 16 * 16;
    const int kc_max = kWLdsFloats / (nt * 16) / 16 * 16;
    pa.kc = std::min(pa.K16, kc_max);
    pa.d_out = ly.d_out;
    pa.ldz = nt * 16;
    pa.w_self = ly.w_self;
    pa.w_neigh = ly.w_neigh;
    pa.z = sw.z;
    pa.off = smp->frontier_off;
    pa.seg0 = (int64_t)(lvl + 1) * W;
    pa.W = W;
    pa.rows_cap = rows_cap;
    const size_t lds = (size_t)pa.kc * nt * 16 * sizeof(float);
    switch (nt) {
      case 1: launch_project<1>(xt, vec, pa, proj_grid, lds, status_d, stream); break;
      case 2: launch_project<2>(xt, vec, pa, proj_grid, lds, status_d, stream); break;
      case 4: launch_project<4>(xt, vec, pa, proj_grid, lds, status_d, stream); break;
      case 8: launch_project<8>(xt, vec, pa, proj_grid, lds, status_d, stream); break;
      default: launch_project<16>(xt, vec, pa, proj_grid, lds, status_d, stream); break;
    }
    GG_LAUNCH_CHECK("k_sage_project");
    AggArgs aa;
    aa.fids = smp->frontier_ids;
    aa.off = smp->frontier_off;
    aa.nbr = smp->nbr_ids;
    aa.noff = smp->nbr_off;
    aa.W = W;
    aa.lvl = lvl;
    aa.k = fanout_h[lvl];
    aa.z = sw.z;
    aa.ldz = nt * 16;
    aa.d_out = ly.d_out;
    aa.bias = ly.bias;
    aa.relu = ly.relu ? 1 : 0;
    aa.z_cap = rows_cap;
    if (j < L) {
      aa.out = sw.h[(j - 1) & 1];
      aa.out_cap = rows_cap;
    } else {
      aa.out = out_d;
      aa.out_cap = out_rows_cap;
    }
    aa.use_rank = j == 1 ? 1 : 0;   // the first layer's input level is N_b
    aa.rank = sw.rank;
    aa.cpre = sw.csum;
    aa.wpb = wpb;
    aa.nch = nch;
    if (aa.k <= 8)
      hipLaunchKernelGGL(k_sage_aggregate<8>, dim3(agg_bx, W), dim3(kSageBlock), 0, stream, aa,
                         status_d);
    else if (aa.k <= 16)
      hipLaunchKernelGGL(k_sage_aggregate<16>, dim3(agg_bx, W), dim3(kSageBlock), 0, stream, aa,
                         status_d);
    else
      hipLaunchKernelGGL(k_sage_aggregate<32>, dim3(agg_bx, W), dim3(kSageBlock), 0, stream, aa,
                         status_d);
    GG_LAUNCH_CHECK("k_sage_aggregate");
  }
  return GG_OK;
}
