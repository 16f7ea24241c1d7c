// libgg: status strings, error reporting, argument packing, sizes.
#include <string.h>

#include "gg_host.hpp"

namespace gg {

static thread_local char g_err[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

int pack_part(const gg_part_t* part, KPart* out) {
  GG_REQUIRE(part != nullptr, "partition book is NULL");
  const int32_t P = part->num_parts;
  GG_REQUIRE(P >= 1 && P <= GG_MAX_PARTS, "num_parts %d outside 1..%d", P, GG_MAX_PARTS);
  GG_REQUIRE(part->local_owner >= -1 && part->local_owner < P, "local_owner %d outside -1..%d",
             part->local_owner, P - 1);
  GG_REQUIRE(part->num_nodes >= 0 && part->num_nodes < (1LL << 31), "num_nodes %lld unsupported",
             (long long)part->num_nodes);
  out->P = P;
  out->kind = part->kind;
  out->local = part->local_owner;
  out->step0 = 1;
  while (out->step0 * 2 <= P - 1) out->step0 *= 2;
  out->N = part->num_nodes;
  out->div_magic = ((1ULL << 40) + (uint64_t)P - 1) / (uint64_t)P;
  if (part->kind == GG_PART_RANGE) {
    GG_REQUIRE(part->range_start[0] == 0, "range_start[0] must be 0");
    GG_REQUIRE(part->range_start[P] == part->num_nodes, "range_start[P] must equal num_nodes");
    for (int m = 0; m < P; ++m)
      GG_REQUIRE(part->range_start[m + 1] >= part->range_start[m], "range_start not ascending");
  } else {
    GG_REQUIRE(part->kind == GG_PART_MOD, "unknown partition kind %d", part->kind);
  }
  for (int m = 0; m <= GG_MAX_PARTS; ++m)
    out->start[m] = (part->kind == GG_PART_RANGE && m <= P) ? part->range_start[m] : part->num_nodes;
  return GG_OK;
}

int pack_feat(const gg_feat_t* feat, const gg_part_t* part, KFeat* out) {
  GG_REQUIRE(feat != nullptr, "feature description is NULL");
  GG_REQUIRE(feat->num_parts == part->num_parts, "feature shards (%d) != partitions (%d)",
             feat->num_parts, part->num_parts);
  GG_REQUIRE(feat->row_bytes > 0 && feat->row_bytes <= GG_MAX_ROW_BYTES && feat->row_bytes % 4 == 0,
             "row_bytes %d must be a positive multiple of 4 up to %d", feat->row_bytes,
             GG_MAX_ROW_BYTES);
  memset(out, 0, sizeof(*out));
  out->row_bytes = feat->row_bytes;
  out->P = feat->num_parts;
  for (int m = 0; m < feat->num_parts; ++m) {
    GG_REQUIRE(feat->shard_rows[m] >= 0, "shard_rows[%d] negative", m);
    GG_REQUIRE(feat->shard_rows[m] == 0 || feat->shard[m] != nullptr, "shard[%d] is NULL", m);
    GG_REQUIRE(feat->shard_rows[m] == 0 ||
                   (feat->row_stride[m] >= feat->row_bytes && feat->row_stride[m] % 4 == 0),
               "row_stride[%d] = %lld invalid", m, (long long)feat->row_stride[m]);
    GG_REQUIRE(((uintptr_t)feat->shard[m] & 3u) == 0, "shard[%d] not 4-byte aligned", m);
    out->shard[m] = (const char*)feat->shard[m];
    out->stride[m] = feat->row_stride[m];
    out->rows[m] = feat->shard_rows[m];
  }
  return GG_OK;
}

int resolve_tuning(const gg_tuning_t* t, Tune* out) {
  const gg_tuning_t z = {};
  if (!t) t = &z;
  GG_REQUIRE(t->tile_rows >= 0 && t->tile_rows <= kWave, "tuning: tile_rows %d outside 1..%d",
             t->tile_rows, kWave);
  GG_REQUIRE(t->gather_blocks == 0 || (t->gather_blocks >= 8 && t->gather_blocks <= 65536),
             "tuning: gather_blocks %d outside 8..65536", t->gather_blocks);
  GG_REQUIRE(t->gather_loads == 0 || t->gather_loads == 2 || t->gather_loads == 4 ||
                 t->gather_loads == 8,
             "tuning: gather_loads %d is not 2, 4 or 8", t->gather_loads);
  GG_REQUIRE(t->stage_blocks >= 0 && t->stage_blocks <= 65536,
             "tuning: stage_blocks %d outside 1..65536", t->stage_blocks);
  GG_REQUIRE(t->stage_host_blocks >= -1 && t->stage_host_blocks <= 65536,
             "tuning: stage_host_blocks %d outside 1..65536 (or -1)", t->stage_host_blocks);
  GG_REQUIRE(t->emit_blocks >= 0 && t->emit_blocks <= kEmitBlocksMax,
             "tuning: emit_blocks %d outside 1..%d", t->emit_blocks, kEmitBlocksMax);
  GG_REQUIRE(t->hot_max_chunks >= 0 && t->hot_max_chunks <= kHotMaxChunks,
             "tuning: hot_max_chunks %d outside 1..%d", t->hot_max_chunks, kHotMaxChunks);
  GG_REQUIRE(t->bytemap_max_mb >= -1 && t->bytemap_max_mb <= 65536,
             "tuning: bytemap_max_mb %d outside 1..65536 (or -1)", t->bytemap_max_mb);
  GG_REQUIRE(t->sample_order >= GG_SAMPLE_BATCH_ORDER && t->sample_order <= GG_SAMPLE_TILES_ALL,
             "tuning: sample_order %d unknown", t->sample_order);
  GG_REQUIRE(t->sample_tile_runs >= 0 && t->sample_tile_runs <= 64 &&
                 (t->sample_tile_runs & (t->sample_tile_runs - 1)) == 0,
             "tuning: sample_tile_runs %d is not a power of two up to 64", t->sample_tile_runs);
  GG_REQUIRE(t->mark_slices_max >= -1 && t->mark_slices_max <= 4096,
             "tuning: mark_slices_max %d outside 1..4096 (or -1)", t->mark_slices_max);
  GG_REQUIRE(t->mark_slice_chunks >= 0 && t->mark_slice_chunks <= 8,
             "tuning: mark_slice_chunks %d outside 1..8", t->mark_slice_chunks);
  GG_REQUIRE(t->mark_block == 0 || t->mark_block == 256 || t->mark_block == 1024,
             "tuning: mark_block %d is not 256 or 1024", t->mark_block);
  GG_REQUIRE(t->mark_min_slots >= -1, "tuning: mark_min_slots %d below -1", t->mark_min_slots);
  GG_REQUIRE(t->mark_min_batches >= -1 && t->mark_min_batches <= GG_MAX_W,
             "tuning: mark_min_batches %d outside 1..%d (or -1)", t->mark_min_batches, GG_MAX_W);
  out->tile_rows = t->tile_rows;
  out->gather_blocks = t->gather_blocks ? t->gather_blocks : kGatherBlocksDefault;
  out->gather_loads = t->gather_loads;
  out->stage_blocks = t->stage_blocks ? t->stage_blocks : kStageBlocksDefault;
  out->stage_host_blocks = t->stage_host_blocks == 0 ? kStageHostBlocksDefault
                           : t->stage_host_blocks < 0 ? out->stage_blocks
                                                      : t->stage_host_blocks;
  out->emit_blocks = t->emit_blocks ? t->emit_blocks : kEmitBlocksMax;
  out->hot_max_chunks = t->hot_max_chunks ? t->hot_max_chunks : kHotMaxChunks;
  out->bytemap_max_bytes = t->bytemap_max_mb == 0 ? kByteMapMaxBytes
                           : t->bytemap_max_mb < 0 ? -1
                                                   : (int64_t)t->bytemap_max_mb << 20;
  out->sample_order = t->sample_order;
  out->sample_tile_runs = t->sample_tile_runs;
  out->mark_slices_max = t->mark_slices_max ? t->mark_slices_max : kMarkSlicesDefault;
  out->mark_slice_chunks = t->mark_slice_chunks ? t->mark_slice_chunks : kMarkSliceChunksDefault;
  out->mark_block = t->mark_block ? t->mark_block : kMarkBlockLanes;
  // default: a slice's words (a smaller hop does not pay for a pass over the slices)
  out->mark_min_batches = t->mark_min_batches;
  out->mark_min_slots = t->mark_min_slots == 0 ? (int64_t)out->mark_slice_chunks * 2048
                        : t->mark_min_slots < 0 ? 0
                                                : t->mark_min_slots;
  return GG_OK;
}

int32_t copy_tile(const Tune& tune, int32_t row_bytes, int32_t max_bytes, bool pow2) {
  if (tune.tile_rows > 0) return tune.tile_rows;
  return pow2 ? tile_rows(row_bytes, max_bytes) : fill_rows(row_bytes, max_bytes);
}

int host_shards(const KFeat& f) {
  int n = 0;
  for (int m = 0; m < f.P; ++m) {
    if (f.rows[m] == 0) continue;
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, f.shard[m]) != hipSuccess) {
      (void)hipGetLastError();   // not known to the runtime: plain host memory
      continue;
    }
    if (at.type == hipMemoryTypeHost) ++n;
  }
  return n;
}

}  // namespace gg

extern "C" {

const char* gg_last_error(void) { return gg::g_err; }

int gg_version(void) { return GG_VERSION; }

int gg_read_status(const int32_t* status_d, int32_t* out_h, hipStream_t stream) {
  GG_REQUIRE(status_d && out_h, "gg_read_status: null pointer");
  int32_t v = 0;
  hipError_t e = hipMemcpyAsync(&v, status_d, sizeof(v), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    gg::set_error("gg_read_status: %s", hipGetErrorString(e));
    return GG_ERR_HIP;
  }
  *out_h = v;
  return GG_OK;
}

const char* gg_status_string(int32_t code) {
  switch (code) {
    case GG_OK: return "ok";
    case GG_ERR_ARG: return "invalid argument";
    case GG_ERR_CAPACITY: return "capacity too small";
    case GG_ERR_HIP: return "HIP runtime error";
    case GG_ERR_UNSUPPORTED: return "unsupported";
    default: return "unknown status";
  }
}

int64_t gg_bits_words(int64_t num_nodes) {
  const int64_t words = (num_nodes + 31) / 32;
  const int64_t w = gg::cdiv(words > 0 ? words : 1, gg::kChunkWords) * gg::kChunkWords;
  return w;
}

int gg_sample_caps(int64_t num_nodes, int32_t W, int64_t max_batch, const int32_t* fanout_h,
                   int32_t L, int64_t* frontier_cap, int64_t* nbr_cap) {
  GG_REQUIRE(W >= 1 && W <= GG_MAX_W && L >= 1 && L <= GG_MAX_LAYERS && fanout_h && max_batch >= 0,
             "bad arguments to gg_sample_caps");
  int64_t f = 0, n = 0;
  int64_t level = max_batch < num_nodes ? max_batch : num_nodes;
  for (int32_t l = 0; l <= L; ++l) {
    f += level;
    if (l < L) {
      n += level * fanout_h[l];
      const int64_t grow = level * (int64_t)(fanout_h[l] + 1);
      level = grow < num_nodes ? grow : num_nodes;
    }
  }
  *frontier_cap = f * W;
  *nbr_cap = n * W;
  return GG_OK;
}

}  // extern "C"
