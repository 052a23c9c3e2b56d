// Filler Packing (Sec. IV-C of arXiv 2608.01150, Eq. 8): the planner's second
// stage, which keeps lightweight sequences whole and places them, most
// expensive first, into the compute and memory headroom that the anchors'
// placement leaves on each rank.  Host-only C++; the prices it consumes are
// the per-rank times the price table measures with this library's kernels.

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <numeric>
#include <vector>

#include "zl_attn.h"
#include "zl_internal.h"

namespace {

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

zl_status invalid(const char* what, long idx = -1) {
  char buf[160];
  if (idx >= 0)
    snprintf(buf, sizeof(buf), "zl_fill_pack: %s (index %ld)", what, idx);
  else
    snprintf(buf, sizeof(buf), "zl_fill_pack: %s", what);
  return zl::host_status(ZL_ERR_INVALID_ARG, buf);
}

}  // namespace

extern "C" zl_status zl_fill_pack(int32_t num_ranks, int32_t num_fillers, const double* price, const double* mem,
                                  double load_floor, double mem_cap, double* load, double* mem_used,
                                  int32_t* rank_of, int32_t* failed) {
  if (num_ranks < 1) return invalid("num_ranks must be >= 1");
  if (num_fillers < 0) return invalid("num_fillers must be >= 0");
  if (!load || !mem_used) return invalid("load and mem_used must not be NULL");
  if (num_fillers > 0 && (!price || !mem || !rank_of)) return invalid("price, mem and rank_of must not be NULL");
  if (!(std::isfinite(load_floor) && load_floor > 0.0)) return invalid("load_floor must be finite and positive");
  if (!(std::isfinite(mem_cap) && mem_cap > 0.0)) return invalid("mem_cap must be finite and positive");
  const size_t N = (size_t)num_ranks, n = (size_t)num_fillers;
  for (size_t r = 0; r < N; ++r) {
    if (!std::isfinite(load[r])) return invalid("load must be finite", (long)r);
    if (!finite_nonneg(mem_used[r])) return invalid("mem_used must be finite and >= 0", (long)r);
  }
  for (size_t s = 0; s < n; ++s) {
    if (!finite_nonneg(price[s])) return invalid("price must be finite and >= 0", (long)s);
    for (size_t r = 0; r < N; ++r)
      if (!finite_nonneg(mem[s * N + r])) return invalid("mem must be finite and >= 0", (long)(s * N + r));
  }

  // Fillers in decreasing price; equal prices keep their input order.
  std::vector<int32_t> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return price[a] > price[b]; });

  std::fill(rank_of, rank_of + n, -1);
  if (failed) *failed = -1;
  for (const int32_t s : order) {
    const double p = price[s];
    const double* need_row = mem + (size_t)s * N;
    int32_t best_r = -1;
    double best = 0.0;
    for (size_t r = 0; r < N; ++r) {
      const double need = need_row[r];
      const double h_m = mem_cap - mem_used[r];
      if (!(h_m >= need)) continue;  // r is not in R_s
      const double h_c = load_floor - load[r];
      const double rho_c = (h_c - p) / load_floor;
      const double rho_m = (h_m - need) / mem_cap;
      const double score = std::min(rho_c, rho_m);
      if (best_r < 0 || score > best) {  // strict: a tie keeps the lower rank
        best_r = (int32_t)r;
        best = score;
      }
    }
    if (best_r < 0) {
      if (failed) *failed = s;
      char buf[128];
      snprintf(buf, sizeof(buf), "zl_fill_pack: filler %d (price %g) fits on no rank", s, p);
      return zl::host_status(ZL_ERR_INFEASIBLE, buf);
    }
    rank_of[s] = best_r;
    load[best_r] += p;
    mem_used[best_r] += need_row[best_r];
  }
  return zl::host_status(ZL_OK, "");
}
