// Internal interface between the host library (validation, scheduling, plan
// cache) and the gfx950 kernels.  Not part of the C ABI.
#pragma once

#include <cstddef>
#include <cstdint>

#include <hip/hip_runtime_api.h>

#include "zl_attn.h"

namespace zl {

// Records `msg` as the calling thread's zl_last_error (clears it for ZL_OK)
// and returns st: the one error channel of every C ABI entry point.
zl_status host_status(zl_status st, const char* msg);

// One unit of work of a launch.  Forward: query rows [q_start, q_start+q_len)
// of one head against the keys [k_start, k_start+k_len) of one K/V range.
// Backward: keys [k_start, k_start+k_len) of one range against all of the
// owning segment's queries [q_start, q_start+q_len).
struct Item {
  int32_t q_start, q_len, k_start, k_len, head, slot, seg, range;
};
static_assert(sizeof(Item) == 32, "work item must stay 32 bytes");

// Tile shapes of each kernel family (rows of Q per forward item, keys per
// backward item, and the inner tile of the loop each one runs).
constexpr int kFwdTileM = 256;       // bf16 forward: 8 waves x 32 query rows
constexpr int kFwdTileN = 64;        // keys per inner step
constexpr int kFwd32TileM = 64;      // fp32 forward: one query row per lane
constexpr int kFwd32TileN = 32;
constexpr int kBwdTileN = 128;       // dK/dV kernel: 4 producer waves x 32 keys per item
constexpr int kBwdTileM = 64;        // queries per dK/dV inner step
constexpr int kDqTileM = 256;        // dQ kernel: 8 waves x 32 query rows per item
constexpr int kDqTileN = 64;         // keys per dQ inner step

// Work-item index of workgroup `b`.  Workgroups are dispatched round-robin
// over the 8 XCDs (b % 8); each run of 8*chunk consecutive workgroups is
// regrouped so that one XCD takes `chunk` consecutive items (neighbouring
// query tiles of one head share K/V tiles in that XCD's L2).  A trailing
// incomplete run keeps the identity order.  A bijection on [0, n).
__host__ __device__ inline int32_t dispatch_item(int32_t b, int32_t n, int32_t chunk) {
  const int32_t group = 8 * chunk;
  if (chunk <= 1) return b;
  const int32_t base = (b / group) * group;
  if (base + group > n) return b;
  const int32_t r = b - base;
  return base + (r % 8) * chunk + (r / 8);
}

struct FwdParams {
  const void* q;
  const void* k;
  const void* v;
  void* out;
  float* lse;
  void* o_part;          // [S, Tq, H, d] fp32, or bf16 when part_bf16
  float* lse_part;
  const Item* items;
  int32_t n_items;
  int32_t num_heads;
  int64_t slot_stride;   // elements between partial slots of o_part (Tq*H*d)
  int64_t lse_slot_stride;  // Tq*H
  float scale;           // softmax scale
  float scale_log2;      // softmax scale * log2(e)
  int32_t xcd_chunk;
  // Ring-step mode (zl_attn_fwd_step): SHARD items fold their block into the
  // running (o_acc, lse_acc) instead of writing a partial slot.
  int32_t step_mode;
  int32_t step_first;    // the accumulator starts from this block
  int32_t step_last;     // the combined result goes to out / lse
  float* o_acc;          // [Tq, H, d] fp32
  float* lse_acc;        // [Tq, H] fp32
  int32_t part_bf16;     // SHARD partials stored as bf16 (rounded once) instead of fp32
  // Work-queue counters of this launch (the stream's, see stream_counters),
  // or NULL for one item per workgroup in dispatch order (grid = n_items).
  int* wq;
};

struct MergeSeg {
  int32_t row_start, row_count, slot_first, slot_count;
  int64_t unit_start;    // first (row, head) unit of this segment in the flat unit space
};

struct MergeParams {
  const void* o_part;    // fp32, or bf16 (launch_merge's part_bf16)
  const float* lse_part;
  void* out;
  float* lse;
  const MergeSeg* segs;
  const int32_t* slots;
  int32_t n_segs;
  int32_t num_heads;
  int64_t n_units;
  int64_t slot_stride;
  int64_t lse_slot_stride;
};

struct BwdParams {
  const void* q;
  const void* k;
  const void* v;
  const void* out;
  const float* lse;
  const void* dout;
  void* dq;
  void* dk;
  void* dv;
  float* dsum;                 // [Tq, H] fp32 workspace: -D = -rowsum(dO * O)
  float* lse2;                 // [Tq, H] fp32 workspace: LSE * log2(e)
  const Item* kv_items;        // dK/dV items: one key tile against all of its segment's queries
  int32_t n_kv_items;
  const Item* q_items;         // dQ items: one query tile against every key of its segment
  int32_t n_q_items;
  int32_t num_heads;
  int64_t total_q;             // Tq
  float scale;
  float scale_log2;
  int32_t xcd_chunk;
  // Ring-step mode (zl_attn_bwd_step): dQ rows of SHARD items (slot >= 0)
  // accumulate this call's key block into dq_acc (raw, unscaled sums) and are
  // written to dq only by the last step.
  int32_t step_mode;
  int32_t step_first;    // the accumulator starts from this block
  int32_t step_last;     // the accumulated dQ (scaled, bf16) goes to dq
  float* dq_acc;         // [Tq, H, d] fp32
  int* wq_kv;            // work-queue counters of the dK/dV and dQ launches, or NULL (see FwdParams::wq)
  int* wq_q;
};

// Work-queue counters: each stream the library launches on gets one block of
// kWqInts ints in a static device array (zero at load; every launch leaves
// its counters at zero), kWqPerLaunch per kernel.  *out is NULL when the
// device's kWqSlots blocks are all taken by other streams: the kernels then
// run one item per workgroup.  Caller holds the library lock.
constexpr int kWqPerLaunch = 16;
constexpr int kWqInts = 4 * kWqPerLaunch;  // forward, dK/dV, dQ, spare
constexpr int kWqSlots = 64;
zl_status stream_counters(hipStream_t s, int** out);

// Grid of a launch of `kernel` (block threads, static LDS) over n_items with
// work queues: n_items when ctr is NULL, else min(n_items, resident
// workgroups of the device).
int launch_grid(const void* kernel, int block, int n_items, const int* ctr);

hipError_t launch_fwd_bf16(const FwdParams& p, int head_dim, hipStream_t s);
hipError_t launch_fwd_fp32(const FwdParams& p, int head_dim, hipStream_t s);
// Ulysses staging (layout kernels around the head-subset attention); op 0
// pack_qkv, 1 unpack_qkv, 2 pack_out, 3 unpack_out.
struct UlyssesParams {
  const void* a;              // source (q for pack_qkv)
  const void* b;              // k (pack_qkv)
  const void* c;              // v (pack_qkv)
  void* dst;                  // destination (q for unpack_qkv)
  void* dst2;                 // k (unpack_qkv)
  void* dst3;                 // v (unpack_qkv)
  const int32_t* row_map;     // rank-major row -> full row (unpack_qkv, pack_out)
  int64_t rows;               // local rows (ops 0, 3) or rank-major = full rows (ops 1, 2)
  int32_t heads;              // H of the local layout
  int32_t heads_local;        // H / group
  int32_t group;
};

hipError_t launch_merge(const MergeParams& p, int head_dim, bool out_bf16, bool part_bf16, hipStream_t s);

// Returns the calling thread's current device's scratch address in *ptr.
typedef zl_status (*ScratchFn)(void** ptr);

// zl_attn_bwd with its work tables and its D / LSE*log2(e) workspace in one
// block of device scratch of scratch_bytes, obtained from `acquire` once the
// call is validated and known to fit; the tables are built on the host
// (cached per descriptor) and copied in on the stream.  No allocation.
zl_status attn_bwd_scratch(const zl_seg_desc* desc, int32_t H, int32_t hd, zl_dtype dt, float scale, const void* q,
                           const void* k, const void* v, const void* out, const float* lse, const void* dout, void* dq,
                           void* dk, void* dv, size_t scratch_bytes, ScratchFn acquire, void* stream);
hipError_t launch_ulysses(const UlyssesParams& p, int op, int head_dim, hipStream_t s);
// stage 0: preprocess (D), 1: dK/dV, 2: dQ
hipError_t launch_bwd_bf16(const BwdParams& p, int head_dim, int stage, hipStream_t s);

}  // namespace zl
