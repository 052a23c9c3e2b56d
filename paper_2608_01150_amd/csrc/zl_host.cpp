// Host side of the C ABI: argument validation, the segment scheduler, the
// device work-table cache and kernel launches.
//
// The scheduler lowers a rank-local segment list (Sec. IV-D of arXiv
// 2608.01150: the placement materialised as the rank's own token ranges) into
// work items and orders them longest-processing-time first: cost = rows x keys,
// the quadratic attention work of Sec. II-A.  Ties follow segment order, as
// Sec. IV-D sorts a rank's segments by split degree with a fixed placement
// order settling ties.  With each free compute unit taking the next item in
// this order (from the kernels' work queues), the launch runs as greedy list
// scheduling of the items in LPT order: each item goes, largest first, to the
// least-loaded place, as the paper's Filler Packing (Eq. 8) places fillers
// across ranks.

#include "zl_attn.h"
#include "zl_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

namespace {

thread_local std::string g_last_error;

zl_status fail(zl_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
zl_status fail(zl_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

zl_status ok() {
  g_last_error.clear();
  return ZL_OK;
}

}  // namespace

namespace zl {
zl_status host_status(zl_status st, const char* msg) {
  if (st == ZL_OK) return ok();
  return fail(st, "%s", msg);
}
}  // namespace zl

namespace {

// Which buffers a validated descriptor touches.
struct Shape {
  int64_t total_q = 0, total_k = 0;
  bool any_whole_rows = false, any_shard_rows = false;
  bool multi_block_shard = false;  // a SHARD segment with query rows uses several ranges
  bool ranges_single_owner = true;
};

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// step_mode (zl_attn_fwd_step): every SHARD segment has exactly one range and
// block slots are not used (block_index may be NULL, num_slots is ignored).
zl_status validate_desc(const zl_seg_desc* d, int32_t num_slots_arg, bool check_slots, Shape* out,
                        bool step_mode = false) {
  if (!d) return fail(ZL_ERR_INVALID_ARG, "descriptor is NULL");
  const int32_t nq = d->num_q_segs, nk = d->num_kv_ranges;
  if (nq < 0 || nk < 0) return fail(ZL_ERR_INVALID_ARG, "negative segment or range count");
  if (!d->cu_seqlens_q || !d->cu_seqlens_k)
    return fail(ZL_ERR_INVALID_ARG, "cu_seqlens_q / cu_seqlens_k must not be NULL");
  if (nq > 0 && (!d->kind || !d->kv_first || !d->kv_count))
    return fail(ZL_ERR_INVALID_ARG, "kind / kv_first / kv_count must not be NULL");
  if (nk > 0 && !d->block_index && !step_mode) return fail(ZL_ERR_INVALID_ARG, "block_index must not be NULL");
  if (d->cu_seqlens_q[0] != 0) return fail(ZL_ERR_INVALID_ARG, "cu_seqlens_q[0] must be 0");
  if (d->cu_seqlens_k[0] != 0) return fail(ZL_ERR_INVALID_ARG, "cu_seqlens_k[0] must be 0");
  for (int32_t s = 0; s < nq; ++s)
    if (d->cu_seqlens_q[s + 1] < d->cu_seqlens_q[s])
      return fail(ZL_ERR_INVALID_ARG, "cu_seqlens_q decreases at segment %d", s);
  for (int32_t j = 0; j < nk; ++j)
    if (d->cu_seqlens_k[j + 1] < d->cu_seqlens_k[j])
      return fail(ZL_ERR_INVALID_ARG, "cu_seqlens_k decreases at range %d", j);
  const int32_t nslots = d->num_slots;
  if (nslots < 0) return fail(ZL_ERR_INVALID_ARG, "num_slots is negative");
  if (check_slots && !step_mode && num_slots_arg != nslots)
    return fail(ZL_ERR_INVALID_ARG, "num_slots argument (%d) differs from the descriptor's (%d)",
                num_slots_arg, nslots);
  // Offsets, when given: non-negative, and offset + length within int64.
  constexpr int64_t kOffMax = INT64_MAX - ((int64_t)1 << 31);
  if (d->k_offset)
    for (int32_t j = 0; j < nk; ++j)
      if (d->k_offset[j] < 0 || d->k_offset[j] > kOffMax)
        return fail(ZL_ERR_INVALID_ARG, "range %d has k_offset %lld outside [0, 2^63 - 2^31]", j,
                    (long long)d->k_offset[j]);
  std::vector<int32_t> owners(nk, 0);
  Shape sh;
  sh.total_q = d->cu_seqlens_q[nq];
  sh.total_k = d->cu_seqlens_k[nk];
  for (int32_t s = 0; s < nq; ++s) {
    const int32_t lq = d->cu_seqlens_q[s + 1] - d->cu_seqlens_q[s];
    const int kind = d->kind[s];
    const int32_t f = d->kv_first[s], c = d->kv_count[s];
    if (kind != ZL_WHOLE && kind != ZL_SHARD)
      return fail(ZL_ERR_INVALID_ARG, "segment %d has unknown kind %d", s, kind);
    if (c < 1) return fail(ZL_ERR_INVALID_ARG, "segment %d has kv_count %d < 1", s, c);
    if (f < 0 || f > nk - c)
      return fail(ZL_ERR_INVALID_ARG, "segment %d uses ranges [%d, %d) outside [0, %d)", s, f, f + c, nk);
    if (d->q_offset && (d->q_offset[s] < 0 || d->q_offset[s] > kOffMax))
      return fail(ZL_ERR_INVALID_ARG, "segment %d has q_offset %lld outside [0, 2^63 - 2^31]", s,
                  (long long)d->q_offset[s]);
    for (int32_t j = f; j < f + c; ++j) owners[j]++;
    if (kind == ZL_WHOLE) {
      if (c != 1) return fail(ZL_ERR_INVALID_ARG, "WHOLE segment %d must use exactly one range", s);
      const int32_t lk = d->cu_seqlens_k[f + 1] - d->cu_seqlens_k[f];
      if (lk != lq)
        return fail(ZL_ERR_INVALID_ARG, "WHOLE segment %d has %d queries but range %d has %d keys", s, lq, f, lk);
      if (d->q_offset && d->k_offset && d->q_offset[s] != d->k_offset[f])
        return fail(ZL_ERR_INVALID_ARG, "WHOLE segment %d: q_offset differs from its range's k_offset", s);
      if (lq > 0) sh.any_whole_rows = true;
    } else {
      if (lq > 0) sh.any_shard_rows = true;
      if (lq > 0 && c > 1) sh.multi_block_shard = true;
      if (step_mode) {
        if (c != 1)
          return fail(ZL_ERR_INVALID_ARG, "ring step: SHARD segment %d must use exactly one range (has %d)", s, c);
        continue;
      }
      for (int32_t j = f; j < f + c; ++j) {
        const int32_t b = d->block_index[j];
        if (b < 0 || b >= nslots)
          return fail(ZL_ERR_INVALID_ARG, "SHARD segment %d: range %d has block_index %d outside [0, %d)",
                      s, j, b, nslots);
        for (int32_t i = f; i < j; ++i)
          if (d->block_index[i] == b)
            return fail(ZL_ERR_INVALID_ARG, "SHARD segment %d: ranges %d and %d write the same slot %d",
                        s, i, j, b);
        if (d->k_offset) {
          const int64_t a0 = d->k_offset[j], a1 = a0 + (d->cu_seqlens_k[j + 1] - d->cu_seqlens_k[j]);
          for (int32_t i = f; i < j; ++i) {
            const int64_t b0 = d->k_offset[i], b1 = b0 + (d->cu_seqlens_k[i + 1] - d->cu_seqlens_k[i]);
            if (a1 > a0 && b1 > b0 && a0 < b1 && b0 < a1)  // empty blocks cover no token
              return fail(ZL_ERR_INVALID_ARG,
                          "SHARD segment %d: blocks %d and %d overlap in global token positions", s, i, j);
          }
        }
      }
    }
  }
  for (int32_t j = 0; j < nk; ++j)
    if (owners[j] > 1) sh.ranges_single_owner = false;
  if (sh.any_shard_rows && nslots < 1 && !step_mode)
    return fail(ZL_ERR_INVALID_ARG, "SHARD rows need num_slots >= 1");
  *out = sh;
  return ZL_OK;
}

zl_status validate_common(int32_t H, int32_t hd, zl_dtype dt, float scale, bool need_scale) {
  if (H < 1) return fail(ZL_ERR_INVALID_ARG, "num_heads must be >= 1 (got %d)", H);
  if (H > ZL_MAX_HEADS)
    return fail(ZL_ERR_UNSUPPORTED, "num_heads %d exceeds %d (tile rows are addressed with 32-bit offsets)", H,
                ZL_MAX_HEADS);
  if (hd != 64 && hd != 128) return fail(ZL_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", hd);
  if (dt != ZL_BF16 && dt != ZL_FP32) return fail(ZL_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
  if (need_scale && !(std::isfinite(scale) && scale > 0.f))
    return fail(ZL_ERR_INVALID_ARG, "softmax_scale must be finite and > 0");
  return ZL_OK;
}

zl_status check_sizes(const Shape& sh, int32_t H, int32_t hd, int32_t nslots) {
  // Row indices are int32 in the work tables; element offsets are int64.
  const int64_t lim = (int64_t)1 << 31;
  if (sh.total_q >= lim || sh.total_k >= lim) return fail(ZL_ERR_UNSUPPORTED, "more than 2^31-1 rows");
  if ((double)nslots * sh.total_q * H * hd > 9.0e18) return fail(ZL_ERR_UNSUPPORTED, "partial buffer too large");
  return ZL_OK;
}

// ---------------------------------------------------------------- scheduler

struct TileCfg {
  int m, n;
};

TileCfg tile_cfg(zl_dtype dt, int op) {
  if (op == ZL_OP_FWD) return dt == ZL_BF16 ? TileCfg{zl::kFwdTileM, zl::kFwdTileN}
                                            : TileCfg{zl::kFwd32TileM, zl::kFwd32TileN};
  if (op == ZL_OP_BWD_DQ) return TileCfg{zl::kDqTileM, zl::kDqTileN};
  return TileCfg{zl::kBwdTileM, zl::kBwdTileN};
}

// Internal plan kinds beside the public ZL_OP_* codes: the merge table, and
// the forward and backward of a ring step.  Step plans ignore block_index:
// their SHARD items carry slot 0, which only marks them as SHARD.
constexpr int kPlanMerge = 2;
constexpr int kPlanBwdStep = 5;
constexpr int kPlanFwdStep = 6;

bool is_step_plan(int op) { return op == kPlanFwdStep || op == kPlanBwdStep; }

// step: SHARD items carry slot 0 instead of their block's slot (dQ items:
// instead of -1).  dK/dV items also cover the ranges of a SHARD segment with
// no query rows: their gradient is zero, and the kernel stores it.
std::vector<zl::Item> build_items(const zl_seg_desc* d, int32_t H, int op, TileCfg t, bool step = false) {
  std::vector<zl::Item> items;
  for (int32_t s = 0; s < d->num_q_segs; ++s) {
    const int32_t q0 = d->cu_seqlens_q[s], q1 = d->cu_seqlens_q[s + 1];
    if (q1 == q0 && op != ZL_OP_BWD) continue;
    const bool shard = d->kind[s] == ZL_SHARD;
    if (op == ZL_OP_BWD_DQ) {
      const int32_t j0 = d->kv_first[s], j1 = j0 + d->kv_count[s];
      // consecutive ranges are contiguous rows of K/V: the dQ item streams rows [cu_k[j0], cu_k[j1])
      const int32_t total = d->cu_seqlens_k[j1] - d->cu_seqlens_k[j0];
      for (int32_t h = 0; h < H; ++h)
        for (int32_t t0 = q0; t0 < q1; t0 += t.m)
          items.push_back({t0, std::min(t.m, q1 - t0), d->cu_seqlens_k[j0], total, h, step && shard ? 0 : -1, s, j0});
      continue;
    }
    for (int32_t j = d->kv_first[s]; j < d->kv_first[s] + d->kv_count[s]; ++j) {
      const int32_t k0 = d->cu_seqlens_k[j], k1 = d->cu_seqlens_k[j + 1];
      const int32_t slot = shard ? (step ? 0 : d->block_index[j]) : -1;
      for (int32_t h = 0; h < H; ++h) {
        if (op == ZL_OP_FWD) {
          for (int32_t t0 = q0; t0 < q1; t0 += t.m)
            items.push_back({t0, std::min(t.m, q1 - t0), k0, k1 - k0, h, slot, s, j});
        } else {
          for (int32_t t0 = k0; t0 < k1; t0 += t.n)
            items.push_back({q0, q1 - q0, t0, std::min(t.n, k1 - t0), h, slot, s, j});
        }
      }
    }
  }
  std::stable_sort(items.begin(), items.end(), [](const zl::Item& a, const zl::Item& b) {
    const int64_t ca = (int64_t)a.q_len * a.k_len, cb = (int64_t)b.q_len * b.k_len;
    if (ca != cb) return ca > cb;
    if (a.seg != b.seg) return a.seg < b.seg;
    if (a.head != b.head) return a.head < b.head;
    if (a.q_start != b.q_start) return a.q_start < b.q_start;
    if (a.k_start != b.k_start) return a.k_start < b.k_start;
    return a.range < b.range;
  });
  return items;
}

struct MergeTable {
  std::vector<zl::MergeSeg> segs;
  std::vector<int32_t> slots;
  int64_t units = 0;
};

MergeTable build_merge(const zl_seg_desc* d, int32_t H) {
  MergeTable t;
  for (int32_t s = 0; s < d->num_q_segs; ++s) {
    if (d->kind[s] != ZL_SHARD) continue;
    const int32_t q0 = d->cu_seqlens_q[s], lq = d->cu_seqlens_q[s + 1] - q0;
    if (lq == 0) continue;
    zl::MergeSeg m{q0, lq, (int32_t)t.slots.size(), d->kv_count[s], t.units};
    for (int32_t j = d->kv_first[s]; j < d->kv_first[s] + d->kv_count[s]; ++j) t.slots.push_back(d->block_index[j]);
    t.segs.push_back(m);
    t.units += (int64_t)lq * H;
  }
  return t;
}

// ------------------------------------------------------------- plan cache

struct Plan {
  int device = -1;
  void* dev = nullptr;          // device copy of the table(s)
  std::vector<char> host;       // host copy (source of the upload)
  int32_t n_items = 0;          // forward items, or backward dK/dV items
  int32_t n_items2 = 0;         // backward dQ items
  int32_t n_segs = 0;
  int64_t n_units = 0;
  size_t slots_offset = 0;      // merge: slot list; backward: dQ items
};

size_t align256(size_t n) { return (n + 255) / 256 * 256; }

// Bytes of the backward's D and LSE*log2(e) workspace: two fp32 [Tq, H] arrays.
size_t bwd_workspace_bytes(const Shape& sh, int32_t H) { return 2 * align256((size_t)sh.total_q * H * sizeof(float)); }

struct KeyHash {
  size_t operator()(const std::vector<int64_t>& k) const noexcept {
    uint64_t h = 1469598103934665603ull;  // FNV-1a over the 64-bit words
    for (int64_t x : k) {
      h ^= (uint64_t)x;
      h *= 1099511628211ull;
    }
    return (size_t)h;
  }
};

// Every table stays cached until zl_shutdown: a call never frees one, so a
// HIP graph captured after a descriptor's first call keeps valid table
// addresses, and no call has to synchronise the device to retire a table.
// A table is 32 bytes per work item (under 6 MB for the largest batches
// here).  Node-based, so Plan pointers stay valid as the map grows.
std::mutex g_mu;
std::unordered_map<std::vector<int64_t>, Plan, KeyHash> g_plans;

std::vector<int64_t> plan_key(const zl_seg_desc* d, int32_t H, int32_t hd, zl_dtype dt, int op, int dev) {
  std::vector<int64_t> k = {op, (int64_t)dt, H, hd, dev, d->num_q_segs, d->num_kv_ranges, d->num_slots};
  for (int32_t s = 0; s <= d->num_q_segs; ++s) k.push_back(d->cu_seqlens_q[s]);
  for (int32_t s = 0; s < d->num_q_segs; ++s) {
    k.push_back(d->kind[s]);
    k.push_back(d->kv_first[s]);
    k.push_back(d->kv_count[s]);
  }
  for (int32_t j = 0; j <= d->num_kv_ranges; ++j) k.push_back(d->cu_seqlens_k[j]);
  const bool slots = !is_step_plan(op) && d->block_index;  // step plans do not read block_index
  for (int32_t j = 0; j < d->num_kv_ranges; ++j) k.push_back(slots ? d->block_index[j] : 0);
  return k;
}

zl_status insert_plan(std::vector<int64_t>&& key, Plan&& p, hipStream_t stream, Plan** out);

// Builds the host copy of a plan's table(s) into p.
zl_status build_plan_host(const zl_seg_desc* d, int32_t H, zl_dtype dt, int op, Plan& p) {
  if (op == kPlanMerge) {
    MergeTable t = build_merge(d, H);
    p.n_segs = (int32_t)t.segs.size();
    p.n_units = t.units;
    const size_t seg_bytes = t.segs.size() * sizeof(zl::MergeSeg);
    p.slots_offset = (seg_bytes + 255) / 256 * 256;
    p.host.resize(p.slots_offset + t.slots.size() * sizeof(int32_t));
    if (seg_bytes) std::memcpy(p.host.data(), t.segs.data(), seg_bytes);
    if (!t.slots.empty()) std::memcpy(p.host.data() + p.slots_offset, t.slots.data(), t.slots.size() * 4);
  } else if (op == ZL_OP_BWD || op == kPlanBwdStep) {
    const bool step = op == kPlanBwdStep;
    std::vector<zl::Item> kv = build_items(d, H, ZL_OP_BWD, tile_cfg(dt, ZL_OP_BWD), step);
    std::vector<zl::Item> qi = build_items(d, H, ZL_OP_BWD_DQ, tile_cfg(dt, ZL_OP_BWD_DQ), step);
    if (kv.size() > (size_t)INT32_MAX || qi.size() > (size_t)INT32_MAX)
      return fail(ZL_ERR_UNSUPPORTED, "too many work items");
    p.n_items = (int32_t)kv.size();
    p.n_items2 = (int32_t)qi.size();
    p.slots_offset = align256(kv.size() * sizeof(zl::Item));
    p.host.assign(p.slots_offset + qi.size() * sizeof(zl::Item), 0);
    if (!kv.empty()) std::memcpy(p.host.data(), kv.data(), kv.size() * sizeof(zl::Item));
    if (!qi.empty()) std::memcpy(p.host.data() + p.slots_offset, qi.data(), qi.size() * sizeof(zl::Item));
  } else {
    const bool step = op == kPlanFwdStep;
    const int base_op = step ? ZL_OP_FWD : op;
    std::vector<zl::Item> items = build_items(d, H, base_op, tile_cfg(dt, base_op), step);
    if (items.size() > (size_t)INT32_MAX) return fail(ZL_ERR_UNSUPPORTED, "too many work items");
    p.n_items = (int32_t)items.size();
    p.host.resize(items.size() * sizeof(zl::Item));
    if (!items.empty()) std::memcpy(p.host.data(), items.data(), p.host.size());
  }
  return ZL_OK;
}

// Returns the cached plan for this descriptor, building and uploading it on a
// miss.  Caller holds g_mu.
zl_status get_plan(const zl_seg_desc* d, int32_t H, int32_t hd, zl_dtype dt, int op, hipStream_t stream,
                   Plan** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(ZL_ERR_HIP, "hipGetDevice failed: no usable GPU");
  std::vector<int64_t> key = plan_key(d, H, hd, dt, op, dev);
  auto hit = g_plans.find(key);
  if (hit != g_plans.end()) {
    *out = &hit->second;
    return ZL_OK;
  }
  Plan p;
  p.device = dev;
  zl_status st = build_plan_host(d, H, dt, op, p);
  if (st != ZL_OK) return st;
  return insert_plan(std::move(key), std::move(p), stream, out);
}

// Host-only plans (no device copy) for callers that bring their own device
// memory for the tables: built once per descriptor and kept until
// zl_shutdown, like the device tables.  Caller holds g_mu.
std::unordered_map<std::vector<int64_t>, Plan, KeyHash> g_host_plans;

zl_status get_host_plan(const zl_seg_desc* d, int32_t H, int32_t hd, zl_dtype dt, int op, const Plan** out) {
  std::vector<int64_t> key = plan_key(d, H, hd, dt, op, -1);
  auto hit = g_host_plans.find(key);
  if (hit == g_host_plans.end()) {
    Plan p;
    zl_status st = build_plan_host(d, H, dt, op, p);
    if (st != ZL_OK) return st;
    hit = g_host_plans.emplace(std::move(key), std::move(p)).first;
  }
  *out = &hit->second;
  return ZL_OK;
}

// Uploads a built plan (stream-ordered, from its own host copy, which the
// cache keeps alive) and caches it.  Caller holds g_mu.
zl_status insert_plan(std::vector<int64_t>&& key, Plan&& p, hipStream_t stream, Plan** out) {
  if (!p.host.empty()) {
    if (hipMalloc(&p.dev, p.host.size()) != hipSuccess)
      return fail(ZL_ERR_HIP, "hipMalloc of a %zu-byte work table failed", p.host.size());
    if (hipMemcpyAsync(p.dev, p.host.data(), p.host.size(), hipMemcpyHostToDevice, stream) != hipSuccess) {
      (void)hipFree(p.dev);
      return fail(ZL_ERR_HIP, "upload of the work table failed");
    }
  }
  auto ins = g_plans.emplace(std::move(key), std::move(p));
  *out = &ins.first->second;
  return ZL_OK;
}

// ------------------------------------------------------------- Ulysses row map

// Row map of a Ulysses group: rank-major row (rank j's rows, then j+1's, each
// in sequence order) -> row of the full-sequence layout.  cu_rank[j*(n+1)+s]
// is where sequence s starts among rank j's local rows.  Caller holds g_mu.
zl_status get_rowmap(int32_t group, int32_t nseq, const int32_t* cu_rank, hipStream_t stream, Plan** out,
                     int64_t* total_rows) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(ZL_ERR_HIP, "hipGetDevice failed: no usable GPU");
  std::vector<int64_t> key = {100, dev, group, nseq};
  for (int64_t i = 0; i < (int64_t)group * (nseq + 1); ++i) key.push_back(cu_rank[i]);
  const int64_t w = nseq + 1;
  int64_t total = 0;
  for (int32_t j = 0; j < group; ++j) total += cu_rank[j * w + nseq];
  *total_rows = total;
  auto hit = g_plans.find(key);
  if (hit != g_plans.end()) {
    *out = &hit->second;
    return ZL_OK;
  }
  // full-layout start of each sequence and of each rank's shard inside it
  std::vector<int64_t> seq_start(nseq + 1, 0);
  for (int32_t s = 0; s < nseq; ++s) {
    int64_t len = 0;
    for (int32_t j = 0; j < group; ++j) len += cu_rank[j * w + s + 1] - cu_rank[j * w + s];
    seq_start[s + 1] = seq_start[s] + len;
  }
  Plan p;
  p.device = dev;
  p.host.resize((size_t)total * sizeof(int32_t));
  int32_t* map = reinterpret_cast<int32_t*>(p.host.data());
  std::vector<int64_t> before(nseq, 0);  // rows of sequence s on ranks < j
  int64_t r = 0;
  for (int32_t j = 0; j < group; ++j) {
    for (int32_t s = 0; s < nseq; ++s) {
      const int32_t n = cu_rank[j * w + s + 1] - cu_rank[j * w + s];
      for (int32_t o = 0; o < n; ++o) map[r++] = (int32_t)(seq_start[s] + before[s] + o);
      before[s] += n;
    }
  }
  return insert_plan(std::move(key), std::move(p), stream, out);
}

zl_status validate_ulysses(int32_t group, int32_t H, int32_t hd, zl_dtype dt) {
  if (group < 1) return fail(ZL_ERR_INVALID_ARG, "group must be >= 1 (got %d)", group);
  if (H < 1 || H % group != 0)
    return fail(ZL_ERR_INVALID_ARG, "num_heads %d must be a positive multiple of the group size %d", H, group);
  if (hd != 64 && hd != 128) return fail(ZL_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", hd);
  if (dt != ZL_BF16) return fail(ZL_ERR_UNSUPPORTED, "Ulysses staging is bf16 only");
  return ZL_OK;
}

zl_status validate_cu_rank(int32_t group, int32_t nseq, const int32_t* cu_rank, int64_t* total_rows) {
  if (nseq < 0) return fail(ZL_ERR_INVALID_ARG, "negative sequence count");
  if (!cu_rank) return fail(ZL_ERR_INVALID_ARG, "cu_rank is NULL");
  int64_t total = 0;
  for (int32_t j = 0; j < group; ++j) {
    const int32_t* c = cu_rank + (int64_t)j * (nseq + 1);
    if (c[0] != 0) return fail(ZL_ERR_INVALID_ARG, "cu_rank of rank %d must start at 0", j);
    for (int32_t s = 0; s < nseq; ++s)
      if (c[s + 1] < c[s]) return fail(ZL_ERR_INVALID_ARG, "cu_rank of rank %d decreases at sequence %d", j, s);
    total += c[nseq];
  }
  if (total >= ((int64_t)1 << 31)) return fail(ZL_ERR_UNSUPPORTED, "more than 2^31-1 rows");
  *total_rows = total;
  return ZL_OK;
}

// ------------------------------------------------------------- profiler

struct ProfSlot {
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pending;
  double total_ms = 0.0;
  int64_t launches = 0;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
ProfSlot g_prof[ZL_K_COUNT];

// Runs `launch` (which enqueues one kernel on `s`), bracketed by events when
// profiling is on.
template <class F>
hipError_t timed(int kid, hipStream_t s, F&& launch) {
  bool on;
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    on = g_prof_on;
  }
  if (!on) return launch();
  hipEvent_t a = nullptr, b = nullptr;
  if (hipEventCreate(&a) != hipSuccess) return hipErrorOutOfMemory;
  if (hipEventCreate(&b) != hipSuccess) {
    (void)hipEventDestroy(a);
    return hipErrorOutOfMemory;
  }
  (void)hipEventRecord(a, s);
  const hipError_t e = launch();
  (void)hipEventRecord(b, s);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof[kid].pending.emplace_back(a, b);
  return e;
}

// Work items per XCD run of the dispatch order (see dispatch_item).  The
// hardware hands consecutive workgroups to the 8 XCDs in turn, and each XCD
// has its own L2.  When every segment brings one K/V range (WHOLE segments,
// and SHARD segments in a ring step or against gathered blocks), a segment's
// tiles of one head are consecutive in the work table (equal cost, ties by
// query or key tile) and read the same K/V (or Q/dO) tiles, so runs of 16
// keep them on one XCD, where they share that data through its L2.  When a
// SHARD brings several blocks, the tie-break orders its items by query tile,
// then block, so plain order (1) already sends block j of every query tile to
// XCD j mod 8 and the block's K/V stays in one L2; longer runs would mix
// blocks there.  ZL_XCD_CHUNK (read once, 1..4096) overrides the choice for
// every launch.
int32_t xcd_chunk(const Shape& sh) {
  static const int32_t env = [] {
    const char* e = std::getenv("ZL_XCD_CHUNK");
    const long x = e ? std::strtol(e, nullptr, 10) : 0;
    return (int32_t)(x >= 1 && x <= 4096 ? x : 0);
  }();
  if (env) return env;
  return sh.multi_block_shard ? 1 : 16;
}

zl_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(ZL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

extern "C" {

int32_t zl_abi_version(void) { return ZL_ABI_VERSION; }

const char* zl_last_error(void) { return g_last_error.c_str(); }

zl_status zl_workspace_size(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype dt, int32_t op,
                            size_t* bytes) {
  if (!bytes) return fail(ZL_ERR_INVALID_ARG, "bytes is NULL");
  zl_status st = validate_common(H, hd, dt, 1.f, false);
  if (st != ZL_OK) return st;
  Shape sh;
  if ((st = validate_desc(desc, 0, false, &sh)) != ZL_OK) return st;
  if (op == ZL_OP_FWD) {
    *bytes = 0;
    return ok();
  }
  if (op != ZL_OP_BWD) return fail(ZL_ERR_INVALID_ARG, "op must be ZL_OP_FWD or ZL_OP_BWD");
  *bytes = bwd_workspace_bytes(sh, H);
  return ok();
}

zl_status zl_attn_fwd(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype dt, float scale, const void* q,
                      const void* k, const void* v, void* out, float* lse, float* o_part, float* lse_part,
                      int32_t num_slots, void* stream) {
  return zl_attn_fwd_ex(desc, H, hd, dt, scale, q, k, v, out, lse, o_part, ZL_FP32, lse_part, num_slots, stream);
}

zl_status zl_attn_fwd_ex(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype dt, float scale, const void* q,
                         const void* k, const void* v, void* out, float* lse, void* o_part, zl_dtype part_dt,
                         float* lse_part, int32_t num_slots, void* stream) {
  zl_status st = validate_common(H, hd, dt, scale, true);
  if (st != ZL_OK) return st;
  if (part_dt != ZL_FP32 && part_dt != ZL_BF16) return fail(ZL_ERR_INVALID_ARG, "unknown partial dtype %d", (int)part_dt);
  if (part_dt == ZL_BF16 && dt != ZL_BF16)
    return fail(ZL_ERR_UNSUPPORTED, "bf16 partials need a bf16 forward");
  Shape sh;
  if ((st = validate_desc(desc, num_slots, true, &sh)) != ZL_OK) return st;
  if ((st = check_sizes(sh, H, hd, num_slots)) != ZL_OK) return st;
  if (sh.total_q > 0 && !q) return fail(ZL_ERR_INVALID_ARG, "q is NULL");
  if (sh.total_k > 0 && (!k || !v)) return fail(ZL_ERR_INVALID_ARG, "k or v is NULL");
  if (sh.any_whole_rows && (!out || !lse)) return fail(ZL_ERR_INVALID_ARG, "WHOLE rows need out and lse");
  if (sh.any_shard_rows && (!o_part || !lse_part))
    return fail(ZL_ERR_INVALID_ARG, "SHARD rows need o_part and lse_part");
  for (const void* p : {q, k, v, (const void*)out, (const void*)o_part})
    if (p && !aligned(p, 16)) return fail(ZL_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  for (const void* p : {(const void*)lse, (const void*)lse_part})
    if (p && !aligned(p, 4)) return fail(ZL_ERR_INVALID_ARG, "LSE pointers must be 4-byte aligned");
  std::lock_guard<std::mutex> lock(g_mu);
  Plan* plan = nullptr;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = get_plan(desc, H, hd, dt, ZL_OP_FWD, s, &plan)) != ZL_OK) return st;
  if (plan->n_items == 0) return ok();
  zl::FwdParams p{};
  p.q = q;
  p.k = k;
  p.v = v;
  p.out = out;
  p.lse = lse;
  p.o_part = o_part;
  p.part_bf16 = part_dt == ZL_BF16 ? 1 : 0;
  p.lse_part = lse_part;
  p.items = static_cast<const zl::Item*>(plan->dev);
  p.n_items = plan->n_items;
  p.num_heads = H;
  p.slot_stride = (int64_t)sh.total_q * H * hd;
  p.lse_slot_stride = (int64_t)sh.total_q * H;
  p.scale = scale;
  p.scale_log2 = scale * 1.4426950408889634f;
  p.xcd_chunk = xcd_chunk(sh);
  if ((st = zl::stream_counters(s, &p.wq)) != ZL_OK) return st;
  hipError_t e = timed(ZL_K_FWD, s, [&] {
    return dt == ZL_BF16 ? zl::launch_fwd_bf16(p, hd, s) : zl::launch_fwd_fp32(p, hd, s);
  });
  return hip_status(e, "forward launch");
}

zl_status zl_attn_fwd_step(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype dt, float scale, const void* q,
                           const void* k, const void* v, void* out, float* lse, float* o_acc, float* lse_acc,
                           uint32_t flags, void* stream) {
  zl_status st = validate_common(H, hd, dt, scale, true);
  if (st != ZL_OK) return st;
  if (flags & ~(ZL_STEP_FIRST | ZL_STEP_LAST)) return fail(ZL_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
  Shape sh;
  if ((st = validate_desc(desc, 0, false, &sh, true)) != ZL_OK) return st;
  if ((st = check_sizes(sh, H, hd, 1)) != ZL_OK) return st;
  const bool first = flags & ZL_STEP_FIRST, last = flags & ZL_STEP_LAST;
  if (sh.total_q > 0 && !q) return fail(ZL_ERR_INVALID_ARG, "q is NULL");
  if (sh.total_k > 0 && (!k || !v)) return fail(ZL_ERR_INVALID_ARG, "k or v is NULL");
  if ((sh.any_whole_rows || (sh.any_shard_rows && last)) && (!out || !lse))
    return fail(ZL_ERR_INVALID_ARG, "WHOLE rows and the last ring step need out and lse");
  if (sh.any_shard_rows && !(first && last) && (!o_acc || !lse_acc))
    return fail(ZL_ERR_INVALID_ARG, "SHARD rows need o_acc and lse_acc unless the call is both first and last");
  for (const void* p : {q, k, v, (const void*)out, (const void*)o_acc})
    if (p && !aligned(p, 16)) return fail(ZL_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  for (const void* p : {(const void*)lse, (const void*)lse_acc})
    if (p && !aligned(p, 4)) return fail(ZL_ERR_INVALID_ARG, "LSE pointers must be 4-byte aligned");
  std::lock_guard<std::mutex> lock(g_mu);
  Plan* plan = nullptr;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = get_plan(desc, H, hd, dt, kPlanFwdStep, s, &plan)) != ZL_OK) return st;
  if (plan->n_items == 0) return ok();
  zl::FwdParams p{};
  p.q = q;
  p.k = k;
  p.v = v;
  p.out = out;
  p.lse = lse;
  p.items = static_cast<const zl::Item*>(plan->dev);
  p.n_items = plan->n_items;
  p.num_heads = H;
  p.scale = scale;
  p.scale_log2 = scale * 1.4426950408889634f;
  p.xcd_chunk = xcd_chunk(sh);
  p.step_mode = 1;
  p.step_first = first;
  p.step_last = last;
  p.o_acc = o_acc;
  p.lse_acc = lse_acc;
  if ((st = zl::stream_counters(s, &p.wq)) != ZL_OK) return st;
  hipError_t e = timed(ZL_K_FWD, s, [&] {
    return dt == ZL_BF16 ? zl::launch_fwd_bf16(p, hd, s) : zl::launch_fwd_fp32(p, hd, s);
  });
  return hip_status(e, "ring-step forward launch");
}

zl_status zl_ulysses_pack_qkv(int32_t group, int32_t t_local, int32_t H, int32_t hd, zl_dtype dt, const void* q,
                              const void* k, const void* v, void* send, void* stream) {
  zl_status st = validate_ulysses(group, H, hd, dt);
  if (st != ZL_OK) return st;
  if (t_local < 0) return fail(ZL_ERR_INVALID_ARG, "negative t_local");
  if (t_local == 0) return ok();
  if (!q || !k || !v || !send) return fail(ZL_ERR_INVALID_ARG, "q, k, v and send must not be NULL");
  for (const void* p : {q, k, v, (const void*)send})
    if (!aligned(p, 16)) return fail(ZL_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  zl::UlyssesParams p{};
  p.a = q;
  p.b = k;
  p.c = v;
  p.dst = send;
  p.rows = t_local;
  p.heads = H;
  p.heads_local = H / group;
  p.group = group;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return hip_status(timed(ZL_K_ULYSSES, s, [&] { return zl::launch_ulysses(p, 0, hd, s); }), "Ulysses pack_qkv launch");
}

zl_status zl_ulysses_unpack_qkv(int32_t group, int32_t num_seqs, const int32_t* cu_rank, int32_t H, int32_t hd,
                                zl_dtype dt, const void* recv, void* q, void* k, void* v, void* stream) {
  zl_status st = validate_ulysses(group, H, hd, dt);
  if (st != ZL_OK) return st;
  int64_t total = 0;
  if ((st = validate_cu_rank(group, num_seqs, cu_rank, &total)) != ZL_OK) return st;
  if (total == 0) return ok();
  if (!recv || !q || !k || !v) return fail(ZL_ERR_INVALID_ARG, "recv, q, k and v must not be NULL");
  for (const void* p : {recv, (const void*)q, (const void*)k, (const void*)v})
    if (!aligned(p, 16)) return fail(ZL_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  std::lock_guard<std::mutex> lock(g_mu);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Plan* plan = nullptr;
  if ((st = get_rowmap(group, num_seqs, cu_rank, s, &plan, &total)) != ZL_OK) return st;
  zl::UlyssesParams p{};
  p.a = recv;
  p.dst = q;
  p.dst2 = k;
  p.dst3 = v;
  p.row_map = static_cast<const int32_t*>(plan->dev);
  p.rows = total;
  p.heads = H;
  p.heads_local = H / group;
  p.group = group;
  return hip_status(timed(ZL_K_ULYSSES, s, [&] { return zl::launch_ulysses(p, 1, hd, s); }), "Ulysses unpack_qkv launch");
}

zl_status zl_ulysses_pack_out(int32_t group, int32_t num_seqs, const int32_t* cu_rank, int32_t H, int32_t hd,
                              zl_dtype dt, const void* out, void* send, void* stream) {
  zl_status st = validate_ulysses(group, H, hd, dt);
  if (st != ZL_OK) return st;
  int64_t total = 0;
  if ((st = validate_cu_rank(group, num_seqs, cu_rank, &total)) != ZL_OK) return st;
  if (total == 0) return ok();
  if (!out || !send) return fail(ZL_ERR_INVALID_ARG, "out and send must not be NULL");
  if (!aligned(out, 16) || !aligned(send, 16)) return fail(ZL_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  std::lock_guard<std::mutex> lock(g_mu);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Plan* plan = nullptr;
  if ((st = get_rowmap(group, num_seqs, cu_rank, s, &plan, &total)) != ZL_OK) return st;
  zl::UlyssesParams p{};
  p.a = out;
  p.dst = send;
  p.row_map = static_cast<const int32_t*>(plan->dev);
  p.rows = total;
  p.heads = H;
  p.heads_local = H / group;
  p.group = group;
  return hip_status(timed(ZL_K_ULYSSES, s, [&] { return zl::launch_ulysses(p, 2, hd, s); }), "Ulysses pack_out launch");
}

zl_status zl_ulysses_unpack_out(int32_t group, int32_t t_local, int32_t H, int32_t hd, zl_dtype dt, const void* recv,
                                void* out_local, void* stream) {
  zl_status st = validate_ulysses(group, H, hd, dt);
  if (st != ZL_OK) return st;
  if (t_local < 0) return fail(ZL_ERR_INVALID_ARG, "negative t_local");
  if (t_local == 0) return ok();
  if (!recv || !out_local) return fail(ZL_ERR_INVALID_ARG, "recv and out_local must not be NULL");
  if (!aligned(recv, 16) || !aligned(out_local, 16))
    return fail(ZL_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  zl::UlyssesParams p{};
  p.a = recv;
  p.dst = out_local;
  p.rows = t_local;
  p.heads = H;
  p.heads_local = H / group;
  p.group = group;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return hip_status(timed(ZL_K_ULYSSES, s, [&] { return zl::launch_ulysses(p, 3, hd, s); }), "Ulysses unpack_out launch");
}

zl_status zl_lse_merge(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype out_dt, const float* o_part,
                       const float* lse_part, int32_t num_slots, void* out, float* lse, void* stream) {
  return zl_lse_merge_ex(desc, H, hd, out_dt, o_part, ZL_FP32, lse_part, num_slots, out, lse, stream);
}

zl_status zl_lse_merge_ex(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype out_dt, const void* o_part,
                          zl_dtype part_dt, const float* lse_part, int32_t num_slots, void* out, float* lse,
                          void* stream) {
  zl_status st = validate_common(H, hd, out_dt, 1.f, false);
  if (st != ZL_OK) return st;
  if (part_dt != ZL_FP32 && part_dt != ZL_BF16) return fail(ZL_ERR_INVALID_ARG, "unknown partial dtype %d", (int)part_dt);
  Shape sh;
  if ((st = validate_desc(desc, num_slots, true, &sh)) != ZL_OK) return st;
  if ((st = check_sizes(sh, H, hd, num_slots)) != ZL_OK) return st;
  if (!sh.any_shard_rows) return ok();
  if (!o_part || !lse_part || !out || !lse) return fail(ZL_ERR_INVALID_ARG, "merge needs o_part, lse_part, out, lse");
  if (!aligned(o_part, 16) || !aligned(out, 16)) return fail(ZL_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  if (!aligned(lse_part, 4) || !aligned(lse, 4)) return fail(ZL_ERR_INVALID_ARG, "LSE pointers must be 4-byte aligned");
  std::lock_guard<std::mutex> lock(g_mu);
  Plan* plan = nullptr;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = get_plan(desc, H, hd, out_dt, kPlanMerge, s, &plan)) != ZL_OK) return st;
  if (plan->n_units == 0) return ok();
  zl::MergeParams p{};
  p.o_part = o_part;
  p.lse_part = lse_part;
  p.out = out;
  p.lse = lse;
  p.segs = static_cast<const zl::MergeSeg*>(plan->dev);
  p.slots = reinterpret_cast<const int32_t*>(static_cast<const char*>(plan->dev) + plan->slots_offset);
  p.n_segs = plan->n_segs;
  p.num_heads = H;
  p.n_units = plan->n_units;
  p.slot_stride = (int64_t)sh.total_q * H * hd;
  p.lse_slot_stride = (int64_t)sh.total_q * H;
  return hip_status(
      timed(ZL_K_MERGE, s, [&] { return zl::launch_merge(p, hd, out_dt == ZL_BF16, part_dt == ZL_BF16, s); }),
      "merge launch");
}

}  // extern "C"

namespace {

// Arguments of one backward call.
struct BwdCall {
  const zl_seg_desc* desc;
  int32_t H, hd;
  zl_dtype dt;
  float scale;
  const void *q, *k, *v, *out;
  const float* lse;
  const void* dout;
  void *dq, *dk, *dv;
  bool step;        // zl_attn_bwd_step
  float* dq_acc;
  uint32_t flags;
};

// Everything about a backward call except its workspace; fills *sh.
zl_status validate_bwd(const BwdCall& c, Shape* sh) {
  zl_status st = validate_common(c.H, c.hd, c.dt, c.scale, true);
  if (st != ZL_OK) return st;
  if (c.dt != ZL_BF16) return fail(ZL_ERR_UNSUPPORTED, "backward supports ZL_BF16 only");
  if (!c.step && c.flags != 0) return fail(ZL_ERR_INVALID_ARG, "flags must be 0");
  if (c.step && (c.flags & ~(uint32_t)(ZL_STEP_FIRST | ZL_STEP_LAST)))
    return fail(ZL_ERR_INVALID_ARG, "flags may only hold ZL_STEP_FIRST and ZL_STEP_LAST");
  const bool first = !c.step || (c.flags & ZL_STEP_FIRST), last = !c.step || (c.flags & ZL_STEP_LAST);
  if ((st = validate_desc(c.desc, 0, false, sh, c.step)) != ZL_OK) return st;
  if ((st = check_sizes(*sh, c.H, c.hd, 0)) != ZL_OK) return st;
  if (!sh->ranges_single_owner)
    return fail(ZL_ERR_INVALID_ARG, "backward needs every K/V range used by at most one segment");
  if (sh->total_q > 0 && (!c.q || !c.out || !c.lse || !c.dout || !c.dq))
    return fail(ZL_ERR_INVALID_ARG, "q, out, lse, dout and dq must not be NULL");
  if (sh->total_k > 0 && (!c.k || !c.v || !c.dk || !c.dv))
    return fail(ZL_ERR_INVALID_ARG, "k, v, dk and dv must not be NULL");
  if (c.step && sh->any_shard_rows && !(first && last) && !c.dq_acc)
    return fail(ZL_ERR_INVALID_ARG, "dq_acc is needed unless flags = ZL_STEP_FIRST | ZL_STEP_LAST");
  for (const void* p : {c.q, c.k, c.v, c.out, c.dout, (const void*)c.dq, (const void*)c.dk, (const void*)c.dv})
    if (p && !aligned(p, 16)) return fail(ZL_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  if (c.dq_acc && !aligned(c.dq_acc, 16)) return fail(ZL_ERR_INVALID_ARG, "dq_acc must be 16-byte aligned");
  if (c.lse && !aligned(c.lse, 4)) return fail(ZL_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  return ZL_OK;
}


// Enqueues the three backward kernels.  tables: the dK/dV items, then (at
// q_offset bytes) the dQ items; workspace: bwd_workspace_bytes of device
// memory.  No early return for Tq = 0: the ranges of a SHARD without query
// rows still get their (zero) dK/dV.
zl_status launch_bwd(const BwdCall& c, const Shape& sh, const void* tables, size_t q_offset, int32_t n_kv,
                     int32_t n_q, void* workspace, hipStream_t s) {
  const bool first = !c.step || (c.flags & ZL_STEP_FIRST), last = !c.step || (c.flags & ZL_STEP_LAST);
  zl::BwdParams p{};
  p.q = c.q;
  p.k = c.k;
  p.v = c.v;
  p.out = c.out;
  p.lse = c.lse;
  p.dout = c.dout;
  p.dq = c.dq;
  p.dk = c.dk;
  p.dv = c.dv;
  p.dsum = static_cast<float*>(workspace);
  p.lse2 = reinterpret_cast<float*>(static_cast<char*>(workspace) + align256((size_t)sh.total_q * c.H * sizeof(float)));
  const char* base = static_cast<const char*>(tables);
  p.kv_items = reinterpret_cast<const zl::Item*>(base);
  p.n_kv_items = n_kv;
  p.q_items = reinterpret_cast<const zl::Item*>(base + q_offset);
  p.n_q_items = n_q;
  p.num_heads = c.H;
  p.total_q = sh.total_q;
  p.scale = c.scale;
  p.scale_log2 = c.scale * 1.4426950408889634f;
  p.xcd_chunk = xcd_chunk(sh);
  p.step_mode = c.step && !(first && last) ? 1 : 0;
  p.step_first = first ? 1 : 0;
  p.step_last = last ? 1 : 0;
  p.dq_acc = c.dq_acc;
  int* wq = nullptr;
  const zl_status wst = zl::stream_counters(s, &wq);
  if (wst != ZL_OK) return wst;
  p.wq_kv = wq ? wq + zl::kWqPerLaunch : nullptr;
  p.wq_q = wq ? wq + 2 * zl::kWqPerLaunch : nullptr;
  const int hd = c.hd;
  hipError_t e = timed(ZL_K_BWD_PRE, s, [&] { return zl::launch_bwd_bf16(p, hd, 0, s); });
  if (e == hipSuccess) e = timed(ZL_K_BWD_DKDV, s, [&] { return zl::launch_bwd_bf16(p, hd, 1, s); });
  if (e == hipSuccess) e = timed(ZL_K_BWD_DQ, s, [&] { return zl::launch_bwd_bf16(p, hd, 2, s); });
  return hip_status(e, "backward launch");
}

// Shared by zl_attn_bwd (step = false) and zl_attn_bwd_step.
zl_status attn_bwd_impl(const BwdCall& c, void* workspace, size_t ws_bytes, void* stream) {
  Shape sh;
  zl_status st = validate_bwd(c, &sh);
  if (st != ZL_OK) return st;
  const size_t need = bwd_workspace_bytes(sh, c.H);
  if (need > 0 && (!workspace || ws_bytes < need))
    return fail(ZL_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace ? ws_bytes : 0);
  if (workspace && !aligned(workspace, 256)) return fail(ZL_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  std::lock_guard<std::mutex> lock(g_mu);
  Plan* plan = nullptr;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = get_plan(c.desc, c.H, c.hd, c.dt, c.step ? kPlanBwdStep : ZL_OP_BWD, s, &plan)) != ZL_OK) return st;
  return launch_bwd(c, sh, plan->dev, plan->slots_offset, plan->n_items, plan->n_items2, workspace, s);
}

}  // namespace

namespace zl {

zl_status attn_bwd_scratch(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype dt, float scale, const void* q,
                           const void* k, const void* v, const void* out, const float* lse, const void* dout, void* dq,
                           void* dk, void* dv, size_t scratch_bytes, ScratchFn acquire, void* stream) {
  const BwdCall c{desc, H, hd, dt, scale, q, k, v, out, lse, dout, dq, dk, dv, false, nullptr, 0u};
  Shape sh;
  zl_status st = validate_bwd(c, &sh);
  if (st != ZL_OK) return st;
  std::lock_guard<std::mutex> lock(g_mu);
  const Plan* hp = nullptr;
  if ((st = get_host_plan(desc, H, hd, dt, ZL_OP_BWD, &hp)) != ZL_OK) return st;
  // layout: [dK/dV items | dQ items] (the plan's host bytes), then the workspace
  const size_t tables = align256(hp->host.size());
  const size_t need = tables + bwd_workspace_bytes(sh, H);
  if (need > scratch_bytes)
    return fail(ZL_ERR_WORKSPACE, "this batch needs %zu bytes of scratch (work tables %zu, workspace %zu); the "
                "static scratch holds %zu", need, tables, need - tables, scratch_bytes);
  void* base = nullptr;
  if ((st = acquire(&base)) != ZL_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!hp->host.empty() &&
      hipMemcpyAsync(base, hp->host.data(), hp->host.size(), hipMemcpyHostToDevice, s) != hipSuccess)
    return fail(ZL_ERR_HIP, "copy of the work tables into the scratch failed");
  return launch_bwd(c, sh, base, hp->slots_offset, hp->n_items, hp->n_items2, static_cast<char*>(base) + tables, s);
}

}  // namespace zl

extern "C" {

zl_status zl_attn_bwd(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype dt, float scale, const void* q,
                      const void* k, const void* v, const void* out, const float* lse, const void* dout, void* dq,
                      void* dk, void* dv, uint32_t flags, void* workspace, size_t ws_bytes, void* stream) {
  const BwdCall c{desc, H, hd, dt, scale, q, k, v, out, lse, dout, dq, dk, dv, false, nullptr, flags};
  return attn_bwd_impl(c, workspace, ws_bytes, stream);
}

zl_status zl_attn_bwd_step(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype dt, float scale, const void* q,
                           const void* k, const void* v, const void* out, const float* lse, const void* dout, void* dq,
                           void* dk, void* dv, float* dq_acc, uint32_t flags, void* workspace, size_t ws_bytes,
                           void* stream) {
  const BwdCall c{desc, H, hd, dt, scale, q, k, v, out, lse, dout, dq, dk, dv, true, dq_acc, flags};
  return attn_bwd_impl(c, workspace, ws_bytes, stream);
}

zl_status zl_plan_dump(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype dt, int32_t op, int32_t* items,
                       size_t cap, size_t* n, int32_t* tile_m, int32_t* tile_n) {
  zl_status st = validate_common(H, hd, dt, 1.f, false);
  if (st != ZL_OK) return st;
  if (op != ZL_OP_FWD && op != ZL_OP_BWD && op != ZL_OP_BWD_DQ)
    return fail(ZL_ERR_INVALID_ARG, "op must be ZL_OP_FWD, ZL_OP_BWD or ZL_OP_BWD_DQ");
  if (!n) return fail(ZL_ERR_INVALID_ARG, "n is NULL");
  if (cap > 0 && !items) return fail(ZL_ERR_INVALID_ARG, "items is NULL with cap > 0");
  Shape sh;
  if ((st = validate_desc(desc, 0, false, &sh)) != ZL_OK) return st;
  const TileCfg t = tile_cfg(dt, op);
  std::vector<zl::Item> v = build_items(desc, H, op, t);
  *n = v.size();
  const size_t m = std::min(cap, v.size());
  if (m) std::memcpy(items, v.data(), m * sizeof(zl::Item));
  if (tile_m) *tile_m = t.m;
  if (tile_n) *tile_n = t.n;
  return ok();
}

zl_status zl_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_on = on != 0;
  return ok();
}

zl_status zl_profile_read(int32_t kid, double* total_ms, int64_t* launches) {
  if (kid < 0 || kid >= ZL_K_COUNT) return fail(ZL_ERR_INVALID_ARG, "unknown kernel id %d", kid);
  std::vector<std::pair<hipEvent_t, hipEvent_t>> ev;
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    ev.swap(g_prof[kid].pending);
  }
  double add = 0.0;
  hipError_t err = hipSuccess;
  for (auto& pr : ev) {
    float ms = 0.f;
    if (err == hipSuccess) err = hipEventSynchronize(pr.second);
    if (err == hipSuccess) err = hipEventElapsedTime(&ms, pr.first, pr.second);
    add += ms;
    (void)hipEventDestroy(pr.first);
    (void)hipEventDestroy(pr.second);
  }
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof[kid].total_ms += add;
  g_prof[kid].launches += (int64_t)ev.size();
  if (total_ms) *total_ms = g_prof[kid].total_ms;
  if (launches) *launches = g_prof[kid].launches;
  if (err != hipSuccess) return fail(ZL_ERR_HIP, "event timing failed: %s", hipGetErrorString(err));
  return ok();
}

void zl_profile_reset(void) {
  for (int k = 0; k < ZL_K_COUNT; ++k) {
    double t;
    int64_t n;
    (void)zl_profile_read(k, &t, &n);
  }
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& sl : g_prof) {
    sl.total_ms = 0.0;
    sl.launches = 0;
  }
}

void zl_shutdown(void) {
  zl_profile_reset();  // retires and destroys any pending timing events
  std::lock_guard<std::mutex> lock(g_mu);
  int cur = 0;
  const bool have_dev = hipGetDevice(&cur) == hipSuccess;
  for (auto& kv : g_plans) {
    Plan& p = kv.second;
    if (p.dev) {
      (void)hipSetDevice(p.device);
      (void)hipDeviceSynchronize();
      (void)hipFree(p.dev);
    }
  }
  g_plans.clear();
  g_host_plans.clear();
  if (have_dev) (void)hipSetDevice(cur);
}

}  // extern "C"
