// Window-size simulator counts (Sec. IV-A simulation; Sec. IV-B, Eqs.
// (1)-(3)): one window's rebuild-delta and miss counters, taken from the
// staging and gather statistics the fetch path already writes, priced with
// the analytical energy model and added to a running total.
#include "gg_host.hpp"

namespace gg {
namespace {

// One transfer event: owners' row counts x_m.  Returns the event's energy
// (initiation for every owner with rows, plus the linear payload) and
// accumulates its duration into *t (zero when no owner has rows).
__device__ double price_event(const int64_t* x, int P, int local, const gg_sim_coeffs_t& c,
                              int64_t* events, int64_t* rows, double* t) {
#pragma clang fp contract(off)
  double e = 0.0, tmax = 0.0;
  int64_t sum = 0;
  for (int m = 0; m < P; ++m) {
    if (m == local) continue;
    const int64_t xm = x[m];
    if (xm <= 0) continue;
    const double xd = (double)xm;
    e = e + (c.eps_init[m] + c.eps_row[m] * xd);
    const double tm = c.lam_init[m] + c.lam_row[m] * xd;
    tmax = tm > tmax ? tm : tmax;
    sum += xm;
    *events += 1;
  }
  *rows += sum;
  if (sum > 0) {
    const double tbw = (double)sum * c.row_bytes / c.bw_bytes_per_s;
    *t = *t + (tmax > tbw ? tmax : tbw);
  }
  return e;
}

// A single lane does the window's few hundred operations in a fixed order.
__global__ void k_sim_accumulate(const gg_stage_stats_t* st, const gg_gather_stats_t* gs,
                                 int32_t nseg, int32_t P, int32_t local, gg_sim_coeffs_t c,
                                 gg_sim_acc_t* acc) {
#pragma clang fp contract(off)
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  gg_sim_acc_t a = *acc;
  double t = a.t_stall;
  a.e_rebuild = a.e_rebuild + price_event(st->delta_rows, P, local, c, &a.rebuild_events,
                                          &a.rebuild_rows, &t);
  for (int32_t b = 0; b < nseg; ++b) {
    a.e_miss = a.e_miss + price_event(gs[b].miss_rows, P, local, c, &a.miss_events,
                                      &a.miss_rows, &t);
    a.hits += gs[b].hits;
    a.remote_rows += gs[b].hits + gs[b].misses;
  }
  a.t_stall = t;
  a.windows += 1;
  a.batches += nseg;
  a.e_stall = c.p_idle * a.t_stall;
  a.e_phy = (a.e_rebuild + a.e_miss) + a.e_stall;
  *acc = a;
}

}  // namespace
}  // namespace gg

using namespace gg;

extern "C" int gg_sim_accumulate(const gg_stage_stats_t* stage_d, const gg_gather_stats_t* gather_d,
                                 int32_t nseg, const gg_part_t* part, const gg_sim_coeffs_t* coeffs,
                                 gg_sim_acc_t* acc_d, hipStream_t stream) {
  GG_REQUIRE(stage_d && acc_d && coeffs && part, "NULL argument");
  GG_REQUIRE(nseg >= 0 && nseg <= GG_MAX_W, "nseg %d out of range [0, %d]", nseg, GG_MAX_W);
  GG_REQUIRE(nseg == 0 || gather_d, "gather statistics are NULL");
  GG_REQUIRE(part->num_parts >= 1 && part->num_parts <= GG_MAX_PARTS, "num_parts %d invalid",
             part->num_parts);
  GG_REQUIRE(coeffs->bw_bytes_per_s > 0.0, "bw_bytes_per_s must be positive");
  hipLaunchKernelGGL(k_sim_accumulate, dim3(1), dim3(kWave), 0, stream, stage_d, gather_d, nseg,
                     part->num_parts, part->local_owner, *coeffs, acc_d);
  GG_LAUNCH_CHECK("k_sim_accumulate");
  return GG_OK;
}
