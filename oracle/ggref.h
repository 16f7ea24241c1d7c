/*
 * ggref: the CPU oracle of the per-window feature-fetch path.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, single-threaded C++
 * implementation of what the path computes, written from the paper's
 * definitions (GreenGNN, arXiv 2606.02916: Sec. IV-A trace collection and
 * window simulation, Sec. IV-C / Algorithm 1 runtime execution, Eq. (1)-(2)
 * request indicators).  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load it.  It shares no code, header
 * or constant table with the HIP library; the two agree only through the
 * documented data layout of the results.
 *
 * Every call works on host pointers, runs synchronously and returns 0 on
 * success or a negative error code.
 *
 * Parity pins (tests under tests/ check each against something other than
 * this code): Philox4x32-10 against an independent published
 * implementation; the bounded map against its exact preimage counts; Floyd
 * against brute-force enumeration of every draw sequence; the sampler
 * against the BFS ball and per-row invariants; the hot set, buckets, stage
 * and gather against brute-force set arithmetic and the unsharded feature
 * matrix; the paper's worked request count (Sec. IV-C, 48 per-batch
 * requests become 3 bulk transfers).
 */
#ifndef GGREF_H
#define GGREF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GGREF_MAX_PARTS 64
#define GGREF_OK 0
#define GGREF_ERR_ARG (-1)
#define GGREF_ERR_CAPACITY (-2)
#define GGREF_ERR_RANGE (-3)

enum { GGREF_PART_MOD = 0, GGREF_PART_RANGE = 1 };

typedef struct ggref_csr {
  int64_t num_nodes;
  int64_t num_edges;
  const void* row_ptr; /* num_nodes + 1 entries, int32 or int64 */
  int32_t row_ptr_bits; /* 32 or 64 */
  int32_t pad_;
  const int32_t* col_idx; /* num_edges entries */
} ggref_csr_t;

/* Partition book: every node has exactly one owner (Sec. IV notation). */
typedef struct ggref_part {
  int32_t num_parts;
  int32_t kind; /* MOD: owner = u mod P, row = u div P.
                   RANGE: owner = m with start[m] <= u < start[m+1], row = u - start[m]. */
  int32_t local_owner; /* the owner that is this worker, or -1 for none */
  int32_t pad_;
  int64_t num_nodes;
  int64_t range_start[GGREF_MAX_PARTS + 1];
} ggref_part_t;

/* Feature shards: owner m's rows live at shard[m] + row * row_stride[m]. */
typedef struct ggref_feat {
  int32_t row_bytes;
  int32_t num_parts;
  const void* shard[GGREF_MAX_PARTS];
  int64_t row_stride[GGREF_MAX_PARTS];
  int64_t shard_rows[GGREF_MAX_PARTS];
} ggref_feat_t;

typedef struct ggref_stage_stats {
  int64_t rows_total;
  int64_t requests_total;
  int64_t invalidated;
  int64_t retained; /* rows copied from the source cache instead of an owner */
  int64_t requests[GGREF_MAX_PARTS];
  int64_t rows[GGREF_MAX_PARTS];
  int64_t bytes[GGREF_MAX_PARTS];
  int64_t delta_rows[GGREF_MAX_PARTS];
} ggref_stage_stats_t;

typedef struct ggref_gather_stats {
  int64_t rows;
  int64_t local;
  int64_t hits;
  int64_t misses;
  int64_t miss_requests[GGREF_MAX_PARTS];
  int64_t miss_rows[GGREF_MAX_PARTS];
} ggref_gather_stats_t;

/* Philox4x32-10 block function (Salmon, Moraes, Dror and Shaw, SC'11):
 * out = philox(ctr, key). */
void ggref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* Maps a 32-bit word onto [0, bound): floor(r * bound / 2^32). */
uint64_t ggref_bounded(uint32_t r, uint64_t bound);

/* Floyd's k-of-d sample from already-bounded draws: t[i] must lie in
 * [0, d-k+i].  Writes the k chosen positions ascending into pos[k].
 * Requires d > k >= 1. */
int ggref_floyd(int64_t d, int32_t k, const int64_t* t, int64_t* pos);

/* Owner and local row of node u. */
int32_t ggref_owner(const ggref_part_t* part, int64_t u);
int64_t ggref_row(const ggref_part_t* part, int64_t u);

/* Neighbour sampling for the W batches of one window (Sec. IV-A step 2).
 * seeds[seed_off[b] .. seed_off[b+1]) are batch b's seed nodes.
 * Output layout, level-major: segment s = l*W + b holds frontier F_l of
 * batch b at frontier_ids[frontier_off[s] .. frontier_off[s+1]), ascending;
 * frontier_off has (L+1)*W + 1 entries.  Segment l*W + b of nbr_ids holds,
 * for each frontier node of F_l (in order), fanout[l] sampled neighbour ids
 * padded with -1; nbr_off has L*W + 1 entries.  need[0], need[1] receive
 * the entries required; returns GGREF_ERR_CAPACITY if a capacity is short. */
int ggref_sample_window(const ggref_csr_t* csr, const int32_t* seeds, const int64_t* seed_off,
                        int32_t W, const int32_t* fanout, int32_t L, uint64_t rng_seed,
                        int32_t epoch, int64_t batch0, int32_t* frontier_ids,
                        int64_t frontier_cap, int64_t* frontier_off, int32_t* nbr_ids,
                        int64_t nbr_cap, int64_t* nbr_off, int64_t* need);

/* Hot set of a window (Sec. IV-A window simulation): the remote nodes of
 * the window's input sets N_b = frontier segment (L, b), with freq(u) = the
 * number of batches whose N_b holds u.  n_hot < 0 keeps all of them;
 * otherwise the n_hot most frequent (ties: smaller id first).  With
 * hot_den > 0 (and n_hot = -1) the budget is the top hot_num / hot_den of
 * the window's U distinct remote nodes, rounded up: ceil(U * hot_num /
 * hot_den) (the "top 10%" of Sec. I).  Output ascending by id. */
int ggref_build_hotset(const int32_t* frontier_ids, const int64_t* frontier_off, int32_t W,
                       int32_t L, const ggref_part_t* part, int64_t n_hot, int64_t hot_num,
                       int64_t hot_den, int32_t* hot_ids, int32_t* hot_freq, int64_t cap,
                       int64_t* hot_count);

/* Stable partition of the hot set by owner: owner-major, input order kept
 * inside each owner; owner_off has P+1 entries. */
int ggref_bucket_by_owner(const int32_t* hot_ids, int64_t hot_count, const ggref_part_t* part,
                          int32_t* bucket_ids, int64_t* owner_off);

/* Window cache rebuild (Sec. IV-A rebuild events, Eq. (1); Sec. IV-C;
 * Algorithm 1 WarmCache).  The rows of the bucketed hot set go to cache
 * slots in bucket order and slot_of points at them, after the entries
 * clear_ids[0 .. clear_count) of slot_of are set to -1.  Without a source
 * cache (src_cache == NULL) every row is requested from its owner.  With
 * one, a row whose node the source remap src_slot_of (which may be slot_of
 * itself, read before clearing) holds is copied from the source cache, and
 * only the rebuild delta Delta_{k,m} = (H_k in owner m) \ C_{k-1} is
 * requested from the owners: one request per owner whose delta is
 * non-empty. */
int ggref_stage_bulk(const int32_t* bucket_ids, const int64_t* owner_off,
                     const ggref_part_t* part, const ggref_feat_t* feat, void* cache,
                     int64_t cache_stride, int64_t cache_rows, int32_t* slot_of,
                     const int32_t* clear_ids, int64_t clear_count, const void* src_cache,
                     const int32_t* src_slot_of, ggref_stage_stats_t* stats);

/* Delta staging into one persistent cache (Sec. IV-A rebuild events,
 * Eq. (1); Algorithm 1 WarmCache(H_{k+1} \ C)).  The entries
 * clear_ids[0 .. clear_count) of slot_of are set to -1 first.  A node of
 * the bucketed hot set that the previous window's remap prev_slot_of
 * (num_nodes entries, or NULL for a first window) holds keeps that slot,
 * and its row stays where it is.  Every other node is the rebuild delta: it
 * is requested from its owner (one request per owner whose delta is
 * non-empty) and takes, in bucket order, the lowest cache slot that
 * prev_slot_of does not hold.  When the free slots run out, the delta rows
 * left over are not cached (slot_of = -1, nothing copied, not counted in
 * rows/bytes/requests, still counted in delta_rows), the call completes
 * and returns GGREF_ERR_CAPACITY. */
int ggref_stage_inplace(const int32_t* bucket_ids, const int64_t* owner_off,
                        const ggref_part_t* part, const ggref_feat_t* feat, void* cache,
                        int64_t cache_stride, int64_t cache_rows, int32_t* slot_of,
                        const int32_t* clear_ids, int64_t clear_count,
                        const int32_t* prev_slot_of, ggref_stage_stats_t* stats);

/* Assembles one batch's input features (Algorithm 1, cache lookup, residual
 * misses, on-demand fetch): out row i = feature row of in_ids[i]. */
int ggref_gather_batch(const int32_t* in_ids, int64_t n, const ggref_part_t* part,
                       const ggref_feat_t* feat, const void* cache, int64_t cache_stride,
                       int64_t cache_rows, const int32_t* slot_of, void* out, int64_t out_stride,
                       ggref_gather_stats_t* stats);

/* Coefficients of the analytical energy model (Sec. IV-B), per owner m;
 * a "row" is one node's feature row.  eps_payload(m, x) = eps_row[m] * x,
 * lam_payload(m, x) = lam_row[m] * x. */
typedef struct ggref_sim_coeffs {
  double eps_init[GGREF_MAX_PARTS];
  double eps_row[GGREF_MAX_PARTS];
  double lam_init[GGREF_MAX_PARTS];
  double lam_row[GGREF_MAX_PARTS];
  double bw_bytes_per_s;
  double row_bytes;
  double p_idle;
} ggref_sim_coeffs_t;

typedef struct ggref_sim_acc {
  int64_t windows;
  int64_t batches;
  int64_t rebuild_events;
  int64_t rebuild_rows;
  int64_t miss_events;
  int64_t miss_rows;
  int64_t remote_rows;
  int64_t hits;
  double e_rebuild;
  double e_miss;
  double t_stall;
  double e_stall;
  double e_phy;
} ggref_sim_acc_t;

/* The paper's trace simulator for one window size W (Sec. IV-A simulation,
 * Sec. IV-B Eqs. (1)-(3), Sec. V trace simulator).  trace_ids /
 * trace_off hold the epoch's N_b, batch b at [trace_off[b],
 * trace_off[b+1]), each ascending and distinct.  For each window k: H_k =
 * the hot set under the budget (n_hot, hot_num / hot_den) as above; the
 * rebuild delta Delta_{k,m} = (H_k in owner m) \ C_{k-1}, C_0 empty and
 * C_k = H_k; per batch the misses M_{b,m} = (remote N_b in owner m) \ H_k.
 * Every non-empty set is one event priced by Eq. (1) or (2); an event lasts
 * the longer of its slowest owner's transfer and its rows at the aggregate
 * bandwidth; E_stall = p_idle * total duration (Eq. (3)). */
int ggref_simulate_epoch(const int32_t* trace_ids, const int64_t* trace_off, int64_t n_batches,
                         int32_t W, int64_t n_hot, int64_t hot_num, int64_t hot_den,
                         const ggref_part_t* part, const ggref_sim_coeffs_t* coeffs,
                         ggref_sim_acc_t* acc);

/* One GraphSAGE layer with the mean aggregator: for a node v with sampled
 * neighbours S(v), out = act(W_self^T h_v + W_neigh^T mean_{u in S(v)} h_u
 * + bias), the mean of an empty S(v) being 0; act = ReLU when relu != 0.
 * Weights are row-major [d_in][d_out]. */
typedef struct ggref_sage_layer {
  int32_t d_in;
  int32_t d_out;
  int32_t relu;
  const float* w_self;
  const float* w_neigh;
  const float* bias;
} ggref_sage_layer_t;

/* The consumer of X_b (Algorithm 1: forward pass on the assembled tensor;
 * Sec. VI-A: GraphSAGE): L mean-aggregator layers over each batch's sampled
 * blocks.  Layer j (1..L) computes h^j for the nodes of F_{L-j} from h^{j-1}
 * over F_{L-j+1}, with S(v) = v's sampled neighbours at hop L-j; h^0 = X_b.
 * x holds the rows of N_b = F_L of all W batches back to back (batch b's at
 * row frontier_off[L*W+b] - frontier_off[L*W]), layers[0].d_in elements of
 * x_dtype (0 = fp32, 1 = fp16) per row at x_stride bytes.  out receives
 * the rows of F_0 (the seeds) of all batches back to back, layers[L-1].d_out
 * doubles per row; out_abs (may be NULL) the same forward pass on absolute
 * values (|x|, |W|, |bias|, no activation), a magnitude bound used to size
 * rounding-error tolerances.  Arithmetic in fp64. */
int ggref_sage_forward(const int32_t* frontier_ids, const int64_t* frontier_off,
                       const int32_t* nbr_ids, const int64_t* nbr_off, int32_t W, int32_t L,
                       const int32_t* fanout, const void* x, int32_t x_dtype, int64_t x_stride,
                       const ggref_sage_layer_t* layers, double* out, double* out_abs);

#ifdef __cplusplus
}
#endif
#endif
