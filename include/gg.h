/*
 * gg.h -- C ABI of libgg, the MI355X (gfx950) per-window feature-fetch path.
 *
 * The method is GreenGNN's window-based caching (arXiv 2606.02916): the
 * epoch is cut into windows of W consecutive sampled mini-batches
 * (Sec. IV-A); each window's remote receptive-field nodes form a hot set
 * that is staged into a local cache with one bulk request per partition
 * owner, and every mini-batch then reads its input features from the cache,
 * with an on-demand path for the residual misses (Sec. IV-C, Algorithm 1).
 * The five calls below are the steps of that path for one window:
 *
 *   gg_sample_window    neighbour sampling of the W batches (Sec. IV-A step 2)
 *   gg_build_hotset     hot set H_k of the window (Sec. IV-A window simulation)
 *   gg_bucket_by_owner  H_k grouped by partition owner (Sec. IV-A rebuild events)
 *   gg_stage_bulk       one bulk copy per non-empty owner into the cache (Sec. IV-C)
 *   gg_gather_batch     per-batch assembly: local rows, cache hits, misses
 *                       (Algorithm 1 inner loop; Eq. (2) request indicators)
 *
 * Conventions shared by every call:
 *  - Pointers ending in _d are device pointers (memory from hipMalloc, or
 *    pinned host memory from hipHostMalloc used through its device
 *    address); pointers ending in _h are host pointers read during the call.
 *    The caller owns every buffer and keeps it alive until the work queued
 *    on `stream` has finished.
 *  - Calls only enqueue work on `stream`; they never allocate, never
 *    synchronise and keep no state between calls (the library reads no
 *    environment and holds no global settings: launch tuning is an
 *    argument, gg_tuning_t).  Scratch memory is the caller's workspace `ws`
 *    of at least the size returned by the matching gg_ws_* function; its
 *    contents need no initialisation.
 *  - Return value: GG_OK, or a GG_ERR_* code when a host-visible argument
 *    is invalid (nothing is enqueued then) or a launch failed;
 *    gg_last_error() gives a message (per thread).
 *  - Data-dependent failures found on the device (a capacity too small, a
 *    node id or a feature row out of range) never write outside a buffer:
 *    the kernels OR a GG_DEV_* bit into the caller's sticky status word
 *    *status_d (int32, zeroed by the caller) and clamp.  Read it once per
 *    window.
 *  - Node ids are int32 in [0, num_nodes).  Feature rows are opaque bytes;
 *    row_bytes must be a multiple of 4 and at most 32768.  The 16-byte
 *    vector copy path is used when every base pointer and stride involved
 *    is a multiple of 16, a 4-byte path otherwise.
 */
#ifndef GG_H
#define GG_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GG_VERSION 1

#define GG_MAX_PARTS 64   /* partition owners */
#define GG_MAX_LAYERS 4   /* sampling hops L */
#define GG_MAX_W 64       /* batches per window */
#define GG_MAX_FANOUT 32  /* neighbours drawn per node and hop */
#define GG_MAX_ROW_BYTES 32768

/* Return codes. */
#define GG_OK 0
#define GG_ERR_ARG 1
#define GG_ERR_CAPACITY 2
#define GG_ERR_HIP 3
#define GG_ERR_UNSUPPORTED 4

/* Bits of the sticky device status word. */
#define GG_DEV_CAPACITY 1   /* an output capacity was too small; results clamped */
#define GG_DEV_BAD_ID 2     /* a seed or neighbour id outside [0, num_nodes) */
#define GG_DEV_BAD_ROW 4    /* a feature row or cache slot outside its shard or cache */
#define GG_DEV_BAD_DEGREE 8 /* a node degree of 2^32 or more */
#define GG_DEV_ORDER 16     /* ids declared owner-ordered were not; bucketing output invalid */

/* Graph in CSR form (device): row u holds the sampled-from neighbours of u
 * at col_idx[row_ptr[u] .. row_ptr[u+1]). */
typedef struct gg_csr {
  int64_t num_nodes;     /* < 2^31 */
  int64_t num_edges;
  const void* row_ptr;   /* num_nodes + 1 entries of int32 or int64 */
  int32_t row_ptr_bits;  /* 32 or 64 */
  int32_t pad_;
  const int32_t* col_idx;
} gg_csr_t;

/* Partition book (Sec. IV notation: each node belongs to exactly one owner).
 * Passed by value to the kernels; range_start is read on the host. */
enum { GG_PART_MOD = 0, GG_PART_RANGE = 1 };
typedef struct gg_part {
  int32_t num_parts;    /* P, 1..GG_MAX_PARTS */
  int32_t kind;         /* GG_PART_MOD: owner = u mod P, row = u div P.
                           GG_PART_RANGE: owner = m with range_start[m] <= u <
                           range_start[m+1], row = u - range_start[m]. */
  int32_t local_owner;  /* this worker's own partition, or -1 (all remote) */
  int32_t pad_;
  int64_t num_nodes;
  int64_t range_start[GG_MAX_PARTS + 1]; /* RANGE only: 0 = start[0] <= ... <= start[P] = num_nodes */
} gg_part_t;

/* Feature shards: owner m's row r is row_bytes bytes at
 * shard[m] + r * row_stride[m] (device memory, or pinned host memory through
 * its device address for remote owners kept in host memory). */
typedef struct gg_feat {
  int32_t row_bytes;
  int32_t num_parts;
  const void* shard[GG_MAX_PARTS];
  int64_t row_stride[GG_MAX_PARTS];
  int64_t shard_rows[GG_MAX_PARTS];
} gg_feat_t;

/* Outputs of gg_sample_window (all device, caller allocated).
 * Level-major layout: segment s = l*W + b (l = 0..L, b = 0..W-1) holds the
 * frontier F_l of batch b, ascending, at
 * frontier_ids[frontier_off[s] .. frontier_off[s+1]); F_0 is the batch's
 * distinct seeds and N_b = F_L is the batch's input node set.
 * Segment l*W + b (l < L) of nbr_ids holds fanout[l] entries per node of
 * F_l, in frontier order: the sampled neighbour ids, then -1 padding.
 * frontier_bits holds, for every batch b, the bit set of N_b:
 * bit (u & 31) of word frontier_bits[b * gg_bits_words(num_nodes) + (u >> 5)].
 * need[0], need[1] receive the frontier and neighbour entries required;
 * offsets are clamped to the capacities. */
typedef struct gg_wsample {
  int32_t* frontier_ids;
  int64_t frontier_cap;
  int64_t* frontier_off;   /* (L+1)*W + 1 entries */
  int32_t* nbr_ids;
  int64_t nbr_cap;
  int64_t* nbr_off;        /* L*W + 1 entries */
  uint32_t* frontier_bits; /* W * gg_bits_words(num_nodes) words */
  int64_t* need;           /* 2 entries */
} gg_wsample_t;

/* Per-window staging statistics (device). */
typedef struct gg_stage_stats {
  int64_t rows_total;        /* cache rows filled */
  int64_t requests_total;
  int64_t invalidated;       /* remap entries cleared */
  int64_t retained;          /* rows copied from the source cache */
  int64_t requests[GG_MAX_PARTS];   /* 1 per owner with rows requested */
  int64_t rows[GG_MAX_PARTS];       /* rows requested from owner m */
  int64_t bytes[GG_MAX_PARTS];
  int64_t delta_rows[GG_MAX_PARTS]; /* |bucket_m(H_k) \ C_{k-1}|, Sec. IV-A rebuild delta */
} gg_stage_stats_t;

/* Per-batch gather statistics (device). */
typedef struct gg_gather_stats {
  int64_t rows;
  int64_t local;
  int64_t hits;
  int64_t misses;
  int64_t miss_requests[GG_MAX_PARTS]; /* indicator of M_{b,m} != empty, Eq. (2) */
  int64_t miss_rows[GG_MAX_PARTS];
} gg_gather_stats_t;

/* Launch tuning.  Results never depend on it: it only changes how the work
 * is spread over the chip (for sweeps of the launch shape, and for tests
 * that reach code paths small inputs would not).  Every call that takes a
 * `tuning` pointer accepts NULL (all defaults), and a field left 0 keeps
 * its default; values outside the stated ranges are GG_ERR_ARG.  A call
 * and the gg_ws_* function that sized its workspace must be given the same
 * values (the hot-set chunk limit, the byte-map and mark-slice limits and
 * the gather's block count change workspace layouts). */
typedef struct gg_tuning {
  int32_t tile_rows;         /* rows a wavefront copies per step, 1..64 (staging and gathers);
                                default: as many as fit in 32 KB (staging) or 8 KB (gathers),
                                a power of two except for a GG_GATHER_SHARED gather */
  int32_t gather_blocks;     /* blocks of one gather launch, shared by its segments,
                                8..65536 (default 1024) */
  int32_t gather_loads;      /* 16-byte row loads in flight per lane in a gather: 2, 4 or 8
                                (default 8, or 4 with GG_GATHER_SHARED) */
  int32_t stage_blocks;      /* most blocks of a staging copy, 1..65536 (default 16384) */
  int32_t stage_host_blocks; /* most blocks of a staging copy when a shard lives in host
                                memory, 1..65536, or -1 for stage_blocks (default 128) */
  int32_t emit_blocks;       /* most blocks of gg_stage_inplace's free-list emit, 1..512
                                (default 512) */
  int32_t hot_max_chunks;    /* most chunks of gg_build_hotset's passes, 1..4096 (default
                                4096; fewer make every chunk span several passes) */
  int32_t bytemap_max_mb;    /* largest byte map (MB) into which the sampler's last hop marks
                                its draws, 1..65536, or -1 for none (default 512) */
  int32_t sample_order;      /* GG_SAMPLE_BATCH_ORDER (default): one lane per frontier entry,
                                batch by batch.  GG_SAMPLE_TILES_LAST: the last hop in node
                                tiles (a wavefront samples one tile of consecutive node ids in
                                every batch of the window, so the batches share the CSR lines
                                they fetch: less HBM traffic, which pays when other kernels
                                share the memory system).  GG_SAMPLE_TILES_ALL: every hop in
                                node tiles.  The workspace holds the tiles' table unless
                                batch order. */
  int32_t sample_tile_runs;  /* node tiles of this many runs of 256 ids, a power of two up to
                                64; 0: sized per hop from its entry count */
  int32_t mark_slices_max;   /* the sampler marks each hop's draws into the bit sets in a pass of
                                its own, one block per slice of a batch's set held in LDS (up to
                                64 KB: 524,288 node ids), when a batch's set has at most this many
                                slices, 1..4096; -1: never (the hop marks with atomic ORs, or
                                the last hop into the byte map).  Default 8 */
  int32_t mark_slice_chunks; /* chunks of 65,536 node ids (8 KB of a set) per mark slice, 1..8
                                (default 8) */
  int32_t mark_block;        /* lanes of a mark block: 256 (default) or 1024; a block keeps
                                32 KB of slot loads in flight */
  int32_t mark_min_slots;    /* a hop before the last marks through LDS slices only when its
                                bound on neighbour slots per batch, min(N, B * prod_{i<l}
                                (k_i + 1)) * k_l with B the largest batch, is at least this
                                (a smaller hop marks with atomics, which cost less than a
                                pass over the slices); 0: the words of a slice (16,384 by
                                default); -1: every hop */
  int32_t mark_min_batches;  /* a hop marks through LDS slices only in a call of at least this
                                many batches (a pass takes about as long for one batch as for
                                many, where atomics and the byte map scale with the batches);
                                0: 8 where the last hop could use the byte map, else 4;
                                -1: any */
} gg_tuning_t;
#define GG_SAMPLE_BATCH_ORDER 0
#define GG_SAMPLE_TILES_LAST 1
#define GG_SAMPLE_TILES_ALL 2

/* Words per batch of frontier_bits (a multiple of 2048). */
int64_t gg_bits_words(int64_t num_nodes);

/* Worst-case capacities of the sampling outputs for W batches of at most
 * max_batch seeds: sum over l of min(num_nodes, max_batch * prod_{i<l}
 * (fanout[i] + 1)) frontier entries per batch, and that bound times fanout[l]
 * neighbour entries. */
int gg_sample_caps(int64_t num_nodes, int32_t W, int64_t max_batch, const int32_t* fanout_h,
                   int32_t L, int64_t* frontier_cap, int64_t* nbr_cap);

/* Workspace sizes in bytes.  Each serves every call of its entry point with
 * at most the given batches (W), segments (nseg), rows (cap, n_cap) and
 * cache rows, so one workspace sized for a window serves a shorter last
 * window too. */
size_t gg_ws_sample(int64_t num_nodes, int32_t W, const gg_tuning_t* tuning);
size_t gg_ws_hotset(int64_t num_nodes, int32_t W, const gg_tuning_t* tuning);
size_t gg_ws_bucket(int64_t cap, int32_t num_parts);
size_t gg_ws_stage(int64_t cap, int32_t num_parts);
size_t gg_ws_stage_inplace(int64_t cap, int64_t cache_rows, int32_t num_parts);
size_t gg_ws_gather(int64_t n_cap, int32_t nseg, int32_t num_parts, const gg_tuning_t* tuning);

/* Neighbour sampling of one window (Sec. IV-A step 2: one epoch of
 * deterministic sampling under fixed seeds fixes every later access).
 * seeds_d[seed_off_h[b] .. seed_off_h[b+1]) are batch b's seed nodes
 * (b = 0..W-1; seed_off_h[0] = 0).  Hop l (0-based) draws fanout_h[l] <=
 * GG_MAX_FANOUT distinct neighbours of every node of F_l without
 * replacement: all neighbours in CSR order when the degree d is at most
 * fanout_h[l], else the positions chosen by Floyd's algorithm from a
 * Philox4x32-10 stream (key = rng_seed; counter = (u, batch0 + b, epoch,
 * (l << 16) | i/4), word i mod 4 for draw i, mapped onto [0, d-k+i] by
 * floor(r * (d-k+i+1) / 2^32)), ascending.  F_{l+1} is F_l together with
 * the neighbours drawn at hop l.  batch0 is the epoch-global index of the
 * window's first batch, so N_b does not depend on W.  The marks that make
 * F_{l+1} from a hop's draws are the same bits whichever way they are made:
 * through LDS slices of each batch's set in a pass of their own (where a
 * set has at most tuning->mark_slices_max slices of 64 KB, the hop is large
 * enough and the call has enough batches: see gg_tuning_t), else with
 * atomic ORs, or at the last hop into a byte map (one byte per node and
 * batch) when W * 32 * gg_bits_words(num_nodes) is at most
 * tuning->bytemap_max_mb (512 MB by default).  gg_ws_sample includes the
 * byte map of any call of at most W batches that takes it. */
int gg_sample_window(const gg_csr_t* csr, const int32_t* seeds_d, const int64_t* seed_off_h,
                     int32_t W, const int32_t* fanout_h, int32_t L, uint64_t rng_seed,
                     int32_t epoch, int64_t batch0, const gg_wsample_t* out,
                     const gg_tuning_t* tuning, int32_t* status_d, void* ws, size_t ws_bytes,
                     hipStream_t stream);

/* gg_sample_window in two calls, so that a caller can write the window's
 * N_b lists on another stream while the hot set is built from the bit sets
 * (the hot set, buckets and staging read only frontier_bits; the lists are
 * first read by the gathers).  part GG_SAMPLE_PART_BITS enqueues everything
 * but the compaction of the last level: once it completes, frontier_bits
 * holds every batch's N_b, and the lists, offsets and neighbour slots of
 * levels 0..L-1 are written.  part GG_SAMPLE_PART_LAST enqueues that
 * compaction: F_L into frontier_ids, its offsets, and need.  The second
 * call must start after the first completes (stream order, or an event
 * across streams) and be given the same arguments, ws included, whose
 * contents carry the level counts from one call to the other; nothing may
 * reuse ws or frontier_bits before it completes.  Any other part is
 * GG_ERR_ARG. */
#define GG_SAMPLE_PART_BITS 1
#define GG_SAMPLE_PART_LAST 2
int gg_sample_window_part(const gg_csr_t* csr, const int32_t* seeds_d, const int64_t* seed_off_h,
                          int32_t W, const int32_t* fanout_h, int32_t L, uint64_t rng_seed,
                          int32_t epoch, int64_t batch0, const gg_wsample_t* out, int32_t part,
                          const gg_tuning_t* tuning, int32_t* status_d, void* ws,
                          size_t ws_bytes, hipStream_t stream);

/* Hot set of the window (Sec. IV-A: the most frequently accessed remote
 * nodes of the window).  Input: the W bit sets N_b written by
 * gg_sample_window (frontier_bits_d).  freq(u) = number of batches whose N_b
 * holds u; a node is remote when its owner is not part->local_owner.
 * n_hot < 0 keeps every remote node of the window (the union); n_hot >= 0
 * keeps the n_hot most frequent (ties: smaller id first).  A budget
 * relative to the window (the "top 10%" of Sec. I): with hot_den > 0 the
 * budget is ceil(U * hot_num / hot_den), U = the number of distinct remote
 * nodes of the window, decided on the device (needs n_hot = -1 and
 * 0 <= hot_num <= hot_den <= 2^31).  hot_ids_d
 * receives the chosen ids ascending, hot_freq_d (may be NULL) their freq;
 * hot_count_d[0] = entries written (<= cap), hot_count_d[1] = entries
 * required. */
int gg_build_hotset(const uint32_t* frontier_bits_d, int32_t W, const gg_part_t* part,
                    int64_t n_hot, int64_t hot_num, int64_t hot_den, int32_t* hot_ids_d,
                    int32_t* hot_freq_d, int64_t cap, int64_t* hot_count_d,
                    const gg_tuning_t* tuning, int32_t* status_d, void* ws, size_t ws_bytes,
                    hipStream_t stream);

/* Groups the hot set by owner, one bucket per owner (Sec. IV-A: one bulk
 * request per partition owner): bucket_ids_d receives the hot_count_d[0]
 * (<= cap) ids owner-major, input order kept inside each owner;
 * owner_off_d[m] .. owner_off_d[m+1] is owner m's bucket (P+1 entries).
 * flags: 0, or GG_BUCKET_OWNER_ORDERED when the caller knows the owners of
 * hot_ids_d never decrease along the list (true of gg_build_hotset's
 * ascending output under a GG_PART_RANGE book).  Under a range book that
 * list is its own bucketing, so the call is then a single copy pass; if the
 * order does not hold after all, GG_DEV_ORDER is raised and bucket_ids_d /
 * owner_off_d are not valid.  Under a GG_PART_MOD book the flag changes
 * nothing.  Any other flag bit is GG_ERR_ARG. */
#define GG_BUCKET_OWNER_ORDERED 1
int gg_bucket_by_owner(const int32_t* hot_ids_d, const int64_t* hot_count_d, int64_t cap,
                       const gg_part_t* part, int32_t flags, int32_t* bucket_ids_d,
                       int64_t* owner_off_d, int32_t* status_d, void* ws, size_t ws_bytes,
                       hipStream_t stream);

/* Stages the window cache (Sec. IV-C; Algorithm 1 WarmCache).  The rows of
 * the bucketed hot set (owner_off_d[P] <= cap entries of bucket_ids_d) go
 * to cache slots in bucket order (slot s at cache_d + s * cache_stride,
 * at most cache_rows) and slot_of_d[u] = s.  slot_of_d has num_nodes
 * entries, -1 where a node is not cached; the caller sets it to -1 once,
 * and every call first clears the entries clear_ids_d[0 .. clear_count_d[0])
 * (both may be NULL), normally the ids the previous call staged.
 * Without a source cache (src_cache_d == NULL) every row is requested from
 * its owner: one bulk copy per owner with a non-empty bucket.  With one
 * (same stride, at least cache_rows rows; its remap src_slot_of_d may be
 * slot_of_d itself, read before the clearing), a row whose node the source
 * remap holds is copied from the source cache in device memory and only
 * the rebuild delta Delta_{k,m} = (H_k in owner m) \ C_{k-1} of Sec. IV-A is
 * requested from the owners, one request per owner whose delta is
 * non-empty (the indicator of Eq. (1)).  stats_d->delta_rows counts the
 * rows of each bucket absent from the source (else the current) remap. */
int gg_stage_bulk(const int32_t* bucket_ids_d, const int64_t* owner_off_d, int64_t cap,
                  const gg_part_t* part, const gg_feat_t* feat, void* cache_d,
                  int64_t cache_stride, int64_t cache_rows, int32_t* slot_of_d,
                  const int32_t* clear_ids_d, const int64_t* clear_count_d,
                  const void* src_cache_d, const int32_t* src_slot_of_d,
                  gg_stage_stats_t* stats_d, const gg_tuning_t* tuning, int32_t* status_d,
                  void* ws, size_t ws_bytes, hipStream_t stream);

/* Delta staging into one persistent cache (Sec. IV-A rebuild events,
 * Eq. (1); Algorithm 1 WarmCache(H_{k+1} \ C)): rows the previous window
 * cached stay where they are, and only the rebuild delta is requested.
 * First the entries clear_ids_d[0 .. clear_count_d[0]) of slot_of_d (this
 * window's remap, num_nodes entries) are set to -1; both may be NULL.  A
 * node of the bucketed hot set (owner_off_d[P] <= cap entries of
 * bucket_ids_d) that prev_slot_of_d (the previous window's remap, another
 * buffer) holds keeps that slot in slot_of_d, and its cache row is not
 * touched.  Every other node is the delta Delta_{k,m}: it is requested from
 * its owner m (one request per owner with a non-empty delta, the indicator
 * of Eq. (1)) and takes, in bucket order, the lowest slot below cache_rows
 * that the previous window does not occupy.  occ_prev_d is that occupancy
 * as the previous call wrote it to its occ_d; occ_d (another buffer of the
 * same size) receives this window's.  An occupancy buffer is 16-byte
 * aligned and holds 16 + cache_rows rounded up to a multiple of 32 bytes:
 * an int64 extent (one past the highest slot any window has used; slots
 * from there on are free), 8 bytes of padding and one byte per slot
 * (non-zero = in use), valid below the extent.  With prev_slot_of_d and
 * occ_prev_d
 * both NULL (a first window) every row is requested and takes slot = its
 * bucket position.  Only free slots are written, so the previous window's
 * gathers may run concurrently; the window before it must be finished.
 * The cache must hold both windows: when the free slots run out,
 * GG_DEV_CAPACITY is raised and the delta rows past the last free slot
 * are not staged (their remap entries stay -1, so a gather serves them as
 * misses); the extent then covers the whole cache, so the next call treats
 * every slot this one filled as taken.  Statistics as gg_stage_bulk's with
 * a source cache: rows, bytes and requests count the delta rows copied,
 * delta_rows the whole delta, retained the rows kept in place. */
int gg_stage_inplace(const int32_t* bucket_ids_d, const int64_t* owner_off_d, int64_t cap,
                     const gg_part_t* part, const gg_feat_t* feat, void* cache_d,
                     int64_t cache_stride, int64_t cache_rows, int32_t* slot_of_d,
                     const int32_t* clear_ids_d, const int64_t* clear_count_d,
                     const int32_t* prev_slot_of_d, const uint8_t* occ_prev_d, uint8_t* occ_d,
                     gg_stage_stats_t* stats_d, const gg_tuning_t* tuning, int32_t* status_d,
                     void* ws, size_t ws_bytes, hipStream_t stream);

/* Assembles the input features of nseg consecutive batches (Algorithm 1
 * inner loop) in one launch.  Segment s (s < nseg) is batch s: its ids are
 * in_ids_d[bounds_d[s] .. bounds_d[s+1]) (bounds_d has nseg + 1 entries, on
 * the device) and they land in order at output rows bounds_d[s] - bounds_d[0]
 * onwards (row i at out_d + i * out_stride); out_d holds n_cap rows.  Row
 * i receives the feature row of its node u: from the local shard when u's
 * owner is part->local_owner, from cache slot slot_of_d[u] when that is
 * >= 0 (a hit), and otherwise through the miss path: u is one of the
 * residual misses M_{b,m} = (N_b in owner m) minus H_k (Sec. IV-A), served
 * on demand straight from owner m's shard.  stats_d[s] receives batch s's
 * counts; miss_requests[m] = 1 for every owner with a non-empty miss set,
 * the request indicator of Eq. (2).  Passing in_ids_d = frontier_ids and
 * bounds_d = frontier_off + L*W + b with nseg = 1 gathers N_b; with
 * bounds_d = frontier_off + L*W and nseg = W it gathers the whole window.
 * No host synchronisation is needed.  Rows past n_cap are dropped and set
 * GG_DEV_CAPACITY.  flags: 0, or GG_GATHER_SHARED when other streams run
 * latency-bound work (sampling) on the device at the same time: each lane
 * then keeps half as many row loads in flight, which costs the gather a few
 * percent alone and leaves the memory system's queues short enough for the
 * concurrent work, and a wavefront's tile of rows holds as many rows as fit
 * in 8 KB rather than a power of two.  Results are identical either way;
 * any other flag bit is GG_ERR_ARG. */
#define GG_GATHER_SHARED 1
int gg_gather_batch(const int32_t* in_ids_d, const int64_t* bounds_d, int32_t nseg,
                    int64_t n_cap, const gg_part_t* part, const gg_feat_t* feat,
                    const void* cache_d, int64_t cache_stride, int64_t cache_rows,
                    const int32_t* slot_of_d, void* out_d, int64_t out_stride, int32_t flags,
                    gg_gather_stats_t* stats_d, const gg_tuning_t* tuning, int32_t* status_d,
                    void* ws, size_t ws_bytes, hipStream_t stream);

/* gg_gather_batch for callers that cannot allocate: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  The
 * same arguments and results, without the workspace: the call's scratch
 * (the per-block statistics, 4 * (2 + P) bytes per gather block) lives in
 * a device array of GG_GATHER_SCRATCH_BYTES that the library holds on each
 * GPU it runs on until the process ends.  A call whose scratch would not
 * fit returns GG_ERR_CAPACITY and enqueues nothing; with the default 1024
 * gather blocks every call fits (at most 270 KB, at 64 segments and 64
 * owners).  The call never allocates; the first call on a device looks up
 * the array's address there.  Nothing in the array needs clearing (every
 * call writes the statistics it reads), but all calls on one GPU share it:
 * calls that overlap on one GPU (different streams or host threads) race,
 * so order them, e.g. on one stream. */
#define GG_GATHER_SCRATCH_BYTES (1 << 20)
int gg_gather_batch_noalloc(const int32_t* in_ids_d, const int64_t* bounds_d, int32_t nseg,
                            int64_t n_cap, const gg_part_t* part, const gg_feat_t* feat,
                            const void* cache_d, int64_t cache_stride, int64_t cache_rows,
                            const int32_t* slot_of_d, void* out_d, int64_t out_stride,
                            int32_t flags, gg_gather_stats_t* stats_d,
                            const gg_tuning_t* tuning, int32_t* status_d, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Window-size simulator counts.  The paper scores a candidate window size W
 * by replaying one epoch's trace: per window k it counts the rebuild delta
 * Delta_{k,m} = (H_k in owner m) minus C_{k-1} with C_{k-1} = H_{k-1}
 * (C_0 empty), per batch the residual misses M_{b,m} = (N_b in owner m)
 * minus H_k, over remote owners m (Sec. IV-A), and prices them with the
 * analytical model of Sec. IV-B: Eq. (1) rebuild energy, Eq. (2) miss
 * energy, Eq. (3) stall energy, E_phy = their sum.  Here the counts are the
 * fetch path's own: one window's gg_stage_stats_t.delta_rows and its
 * batches' gg_gather_stats_t.miss_rows, added to a running total.
 * ------------------------------------------------------------------------- */

/* Coefficients of the analytical model, per owner m.  A "row" is one
 * node's feature row (the paper's x features of a transfer).  Payload terms
 * are linear in the rows moved: eps_payload(m, x) = eps_row[m] * x and
 * lam_payload(m, x) = lam_row[m] * x.  An event (one window's rebuild, or
 * one batch's misses) lasts max(max over owners with x_m > 0 of
 * lam_init[m] + lam_row[m] * x_m, (sum_m x_m) * row_bytes / bw_bytes_per_s):
 * the slowest single-owner transfer or the aggregate bandwidth ceiling.
 * Units are the caller's (e.g. J, s, B/s, W); bw_bytes_per_s must be > 0. */
typedef struct gg_sim_coeffs {
  double eps_init[GG_MAX_PARTS];
  double eps_row[GG_MAX_PARTS];
  double lam_init[GG_MAX_PARTS];
  double lam_row[GG_MAX_PARTS];
  double bw_bytes_per_s;
  double row_bytes;
  double p_idle;
} gg_sim_coeffs_t;

/* Running totals for one candidate W (device; the caller zeroes it before
 * the first window).  z(W) of the paper's rank correction is (rebuild_events,
 * miss_events, t_stall, hits / remote_rows). */
typedef struct gg_sim_acc {
  int64_t windows;
  int64_t batches;
  int64_t rebuild_events;  /* sum over k, m of I[Delta_{k,m} != empty] */
  int64_t rebuild_rows;    /* sum over k, m of |Delta_{k,m}| */
  int64_t miss_events;     /* sum over b, m of I[M_{b,m} != empty] */
  int64_t miss_rows;       /* sum over b, m of |M_{b,m}| */
  int64_t remote_rows;     /* remote members of the N_b, over all batches */
  int64_t hits;            /* of those, served from the cache */
  double e_rebuild;        /* Eq. (1) */
  double e_miss;           /* Eq. (2) */
  double t_stall;          /* summed event durations */
  double e_stall;          /* Eq. (3): p_idle * t_stall */
  double e_phy;            /* e_rebuild + e_miss + e_stall */
} gg_sim_acc_t;

/* Adds one window to acc_d: stage_d is the window's staging statistics,
 * gather_d[0 .. nseg) its batches' gather statistics (one per batch, as a
 * whole-window gg_gather_batch writes them).  Owners equal to
 * part->local_owner are skipped.  The arithmetic is fp64 without fused
 * multiply-adds, in a fixed order (owners ascending; the rebuild, then the
 * batches in order), so totals are reproducible bit for bit.  One tiny
 * launch on `stream`; no host synchronisation. */
int gg_sim_accumulate(const gg_stage_stats_t* stage_d, const gg_gather_stats_t* gather_d,
                      int32_t nseg, const gg_part_t* part, const gg_sim_coeffs_t* coeffs,
                      gg_sim_acc_t* acc_d, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * The consumer of X_b: GraphSAGE with the mean aggregator (Algorithm 1's
 * forward pass on the assembled tensor; Sec. VI-A trains GraphSAGE).
 * ------------------------------------------------------------------------- */

#define GG_F32 0
#define GG_F16 1
#define GG_SAGE_MAX_DIM 128   /* d_out of every layer, and d_in of layers after the first */
#define GG_SAGE_MAX_IN 4096   /* d_in of the first layer */

/* One layer: for a node v with sampled neighbours S(v),
 * out = act(W_self^T h_v + W_neigh^T mean_{u in S(v)} h_u + bias), the mean
 * of an empty S(v) being 0, act = ReLU when relu != 0.  Weights are fp32,
 * row-major [d_in][d_out], on the device; bias [d_out] may be NULL. */
typedef struct gg_sage_layer {
  int32_t d_in;
  int32_t d_out;
  int32_t relu;
  const float* w_self;
  const float* w_neigh;
  const float* bias;
} gg_sage_layer_t;

/* Workspace bytes of gg_sage_forward for graphs of num_nodes nodes, windows
 * of at most W batches and at most rows_cap rows per level (all batches
 * together; the frontier capacity of N_b bounds it). */
size_t gg_ws_sage(int64_t num_nodes, int32_t W, int64_t rows_cap, int32_t L,
                  const gg_sage_layer_t* layers_h);

/* Runs L = the sampling depth GraphSAGE layers over the W batches of a
 * window sampled by gg_sample_window (smp) in one pass per layer.  Layer j
 * (1..L) computes h^j for the nodes of F_{L-j} from h^{j-1} over F_{L-j+1},
 * S(v) being v's neighbours drawn at hop L-j; h^0 = x_d, the rows of the
 * window's N_b back to back as gg_gather_batch writes them for the whole
 * window (layers_h[0].d_in elements of x_dtype per row at x_stride bytes;
 * at least min(rows_cap, |N_b| summed over the window) rows).  The first
 * layer finds rows of N_b by rank in smp->frontier_bits, which must still
 * hold the window's N_b (num_nodes is the graph's node count).
 * out_d receives the rows of F_0 (each batch's distinct seeds) of all
 * batches back to back, layers_h[L-1].d_out fp32 per row; out_rows_cap
 * bounds them.  The dense products run on MFMA in fp32 (each layer first
 * projects its input by [W_self | W_neigh], then averages the projected
 * neighbour rows: the same linear map in the other order).  A level with
 * more rows than rows_cap, or seeds beyond out_rows_cap, set
 * GG_DEV_CAPACITY and the excess is skipped. */
int gg_sage_forward(const gg_wsample_t* smp, int64_t num_nodes, int32_t W, int32_t L,
                    const int32_t* fanout_h,
                    const void* x_d, int32_t x_dtype, int64_t x_stride, int64_t rows_cap,
                    const gg_sage_layer_t* layers_h, float* out_d, int64_t out_rows_cap,
                    int32_t* status_d, void* ws, size_t ws_bytes, hipStream_t stream);

/* Helpers. */

/* Reads the sticky device status word once the work queued so far on
 * `stream` has finished: the one call of the library that waits, meant for
 * the once-per-window check of data-dependent failures (the caller's side
 * of the per-window barrier of Algorithm 1).  status_d: the int32 word
 * passed to the other calls; *out_h receives its GG_DEV_* bits.  The word
 * is not cleared.  Returns GG_ERR_ARG for a null pointer, GG_ERR_HIP when
 * the copy or the wait fails (a fault of earlier work on the stream is
 * reported here). */
int gg_read_status(const int32_t* status_d, int32_t* out_h, hipStream_t stream);

const char* gg_status_string(int32_t code);
const char* gg_last_error(void);
int gg_version(void);

#ifdef __cplusplus
}
#endif
#endif /* GG_H */
