/*
 * zl_attn.h -- C ABI of the packed whole+shard attention library (gfx950).
 *
 * One launch computes exact, non-causal softmax attention over a packed batch
 * that mixes WHOLE segments (a sequence kept whole: configuration (1,1,1),
 * Sec. IV-A of arXiv 2608.01150) with SHARD segments (a rank's local query
 * chunk of a context-parallel sequence attending to K/V blocks, the ring axis
 * of Tab. II).  This is the local compute of the paper's Coalesced Attention
 * Engine (Sec. IV-D): whole sequences on a rank run as one block-diagonal
 * call that never mixes attention across sequences and returns outputs in the
 * rank-local input order; ring-style shards return per-block partial outputs
 * that are accumulated into the exact result (Sec. II-B).
 *
 * Conventions shared by every entry point
 *   - Packed tensors are contiguous THD row-major: element (t, h, c) of a
 *     [T, H, d] tensor sits at ((t * H) + h) * d + c.  Q, O, dO, dQ have Tq =
 *     cu_seqlens_q[num_q_segs] rows; K, V, dK, dV have Tk =
 *     cu_seqlens_k[num_kv_ranges] rows.  LSE tensors are [T, H] fp32.
 *   - Partial buffers: o_part [num_slots, Tq, H, d] fp32 and lse_part
 *     [num_slots, Tq, H] fp32; slot b of a shard row holds the block-locally
 *     normalised output O_b = softmax_b(S) V_b and its LSE_b.
 *   - LSE is the natural-log log-sum-exp of the scaled scores.
 *   - Device pointers are caller-owned (the library never frees or retains
 *     them); tensor pointers must be 16-byte aligned, LSE pointers 4-byte.
 *   - Descriptor arrays are HOST memory, read during the call only.
 *   - `stream` is a hipStream_t (NULL: the null stream).  Work is enqueued
 *     asynchronously; a call returns once it is enqueued.
 *   - Every argument is validated before anything is enqueued: an error
 *     status means no device work was issued and no buffer was touched.
 *     zl_last_error() then describes the problem.  No C++ exception crosses
 *     this boundary.
 *   - The library owns one cache of device work tables (the schedule of a
 *     descriptor), created on the first call with a new descriptor (which
 *     allocates the table and uploads it on the call's stream), reused
 *     afterwards and kept until zl_shutdown(): no call frees a table, so a
 *     table's address stays valid for every graph that captured it, and no
 *     call synchronises the device.  A table takes 32 bytes per work item.
 *     The library allocates no other device memory.  Once a descriptor's
 *     tables exist, calls with it only launch kernels (no allocation, copy,
 *     memset or synchronisation), so they may be captured in a HIP graph;
 *     make the first call eagerly, and keep profiling off while capturing.
 *   - The attention kernels run one workgroup per compute unit and hand out
 *     a launch's work items at run time through atomic counters in a static
 *     device array (no allocation): each stream the library is called on
 *     gets its own counters (up to 64 streams per GPU; calls on further
 *     streams run one work item per workgroup, with the same results).  So
 *     calls that overlap on different streams are independent, and calls on
 *     one stream are ordered.  A captured graph uses the counters of the
 *     stream it was captured on: do not replay it while calls on that stream
 *     (or another replay of it) may still run.  Results do not depend on
 *     which workgroup runs an item.  ZL_STATIC_DISPATCH=1 in the environment
 *     (read once) selects one work item per workgroup for every call.
 */
#ifndef ZL_ATTN_H
#define ZL_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ZL_ABI_VERSION 1

typedef enum {
  ZL_OK = 0,
  ZL_ERR_INVALID_ARG = 1, /* malformed descriptor, pointer, size or scale */
  ZL_ERR_UNSUPPORTED = 2, /* valid request the library does not implement */
  ZL_ERR_WORKSPACE = 3,   /* workspace missing or too small               */
  ZL_ERR_HIP = 4,         /* the HIP runtime reported an error            */
  ZL_ERR_INFEASIBLE = 5   /* a planner found no feasible placement        */
} zl_status;

/* Segment kinds (Sec. IV-A: (1,1,1) keeps a sequence whole; a split
 * sequence's local query chunk is a shard). */
enum { ZL_WHOLE = 0, ZL_SHARD = 1 };

typedef enum { ZL_BF16 = 0, ZL_FP32 = 1 } zl_dtype;

/* Operations.  ZL_OP_BWD_DQ names the second backward schedule (query tiles
 * that produce dQ) and is accepted by zl_plan_dump only. */
enum { ZL_OP_FWD = 0, ZL_OP_BWD = 1, ZL_OP_BWD_DQ = 2 };

/*
 * A rank-local schedule of segments (Sec. IV-D: the placement lowered to the
 * tokens this rank materialises from the sequences' global token ranges).
 *
 * Query segment s owns packed query rows [cu_seqlens_q[s], cu_seqlens_q[s+1])
 * and attends to the K/V ranges kv_first[s] .. kv_first[s]+kv_count[s]-1.
 * K/V range j owns packed K/V rows [cu_seqlens_k[j], cu_seqlens_k[j+1]).
 *   WHOLE: kv_count == 1 and the range has exactly as many rows as the
 *          segment (queries and keys are the same tokens).  Output: final O
 *          and LSE in `out` / `lse`.
 *   SHARD: each listed range is one CP block; block_index[j] is its slot in
 *          the partial buffers (distinct within a segment, < num_slots).  An
 *          empty range yields O_b = 0, LSE_b = -inf.
 * q_offset / k_offset give the global token index of the first row of each
 * segment / range.  They change no value (attention is non-causal, Sec. II-A)
 * and may be NULL; when given they are checked: every offset in [0, 2^63 -
 * 2^31] (so offset + length fits in int64), a WHOLE
 * segment's q_offset equals its range's k_offset, and the blocks of one
 * SHARD cover disjoint global token ranges (overlapping blocks would count
 * keys twice and break exactness).
 * Forward and merge allow several shards to share a K/V range; backward
 * requires every range to be used by at most one segment (single owner of
 * each dK/dV row).
 */
typedef struct zl_seg_desc {
  int32_t num_q_segs;
  const int32_t* cu_seqlens_q; /* [num_q_segs + 1], starts at 0, non-decreasing */
  const uint8_t* kind;         /* [num_q_segs] ZL_WHOLE or ZL_SHARD               */
  const int64_t* q_offset;     /* [num_q_segs] or NULL                           */
  const int32_t* kv_first;     /* [num_q_segs]                                   */
  const int32_t* kv_count;     /* [num_q_segs] 1 for WHOLE, >= 1 for SHARD       */
  int32_t num_kv_ranges;
  const int32_t* cu_seqlens_k; /* [num_kv_ranges + 1], starts at 0, non-decreasing */
  const int64_t* k_offset;     /* [num_kv_ranges] or NULL                        */
  const int32_t* block_index;  /* [num_kv_ranges] CP block id = partial slot      */
  int32_t num_slots;           /* partial slots; >= 1 when any SHARD exists       */
} zl_seg_desc;

/* Largest num_heads any attention entry point accepts. */
#define ZL_MAX_HEADS 16384

/* ABI version this library was built with (ZL_ABI_VERSION). */
int32_t zl_abi_version(void);

/* Message of the last failed call on this thread ("" if none); valid until
 * the next zl_* call on this thread. */
const char* zl_last_error(void);

/* Device workspace in bytes that zl_attn_bwd needs for this batch (op =
 * ZL_OP_BWD: fp32 -D = -rowsum(dO*O) and LSE*log2(e), each [Tq,H]); 0 for
 * ZL_OP_FWD.  Validates like the call it sizes. */
zl_status zl_workspace_size(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim,
                            zl_dtype dtype, int32_t op, size_t* bytes);

/*
 * Forward of one coalesced launch (Sec. IV-D; ring per-block step of
 * Sec. II-B / Tab. II for SHARD rows).  For each head h:
 *   WHOLE row i: out[i,h,:] = sum_j P_ij v_j, lse[i,h] = LSE_i over its range.
 *   SHARD row i, block j (slot b = block_index[j]):
 *     o_part[b,i,h,:] = softmax over block j, lse_part[b,i,h] = LSE over j.
 * S_ij = softmax_scale * q_i . k_j, no mask other than the block diagonal.
 * q [Tq,H,d], k/v [Tk,H,d] in `dtype` (ZL_BF16; ZL_FP32 for plumbing runs),
 * out [Tq,H,d] in `dtype`, lse [Tq,H] fp32.  out/lse may be NULL when there
 * are no WHOLE rows, o_part/lse_part when there are no SHARD rows.  Rows of
 * other kinds are not written.  head_dim must be 64 or 128; num_heads at most
 * ZL_MAX_HEADS (ZL_ERR_UNSUPPORTED beyond: the kernels address the rows of a
 * 64-row tile with 32-bit byte offsets from its first row).
 */
zl_status zl_attn_fwd(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim, zl_dtype dtype,
                      float softmax_scale, const void* q, const void* k, const void* v,
                      void* out, float* lse, float* o_part, float* lse_part, int32_t num_slots,
                      void* stream);

/*
 * zl_attn_fwd with the SHARD partials stored in `part_dtype`: ZL_FP32 (as
 * zl_attn_fwd) or ZL_BF16, which rounds each block-normalised O_b once to
 * bf16 and halves the partial bytes written here and read by the merge (the
 * final O is then rounded twice: O_b, then the merged result).  o_part is
 * [num_slots, Tq, H, d] of that type; lse_part stays fp32.  ZL_BF16 partials
 * need dtype ZL_BF16 (ZL_ERR_UNSUPPORTED otherwise); an unknown part_dtype
 * is ZL_ERR_INVALID_ARG.  Everything else as zl_attn_fwd.
 */
zl_status zl_attn_fwd_ex(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim, zl_dtype dtype,
                         float softmax_scale, const void* q, const void* k, const void* v,
                         void* out, float* lse, void* o_part, zl_dtype part_dtype, float* lse_part,
                         int32_t num_slots, void* stream);

/* Flags of zl_attn_fwd_step. */
#define ZL_STEP_FIRST 1u /* this call carries every SHARD row's first block */
#define ZL_STEP_LAST 2u  /* this call carries every SHARD row's last block */

/*
 * One step of ring attention (Sec. II-B; the ring primitive (1,1,k) of
 * Tab. II) with the output accumulation fused into the forward epilogue, so
 * no per-block partials are stored and no merge kernel runs.  Every SHARD
 * segment carries exactly one K/V range in this call (kv_count == 1), the
 * block the ring delivers at this step; WHOLE segments (fillers) may ride
 * along in any step and are computed exactly as by zl_attn_fwd.  With O_b,
 * LSE_b the attention of SHARD row i over this call's block:
 *   ZL_STEP_FIRST:  (o_acc, lse_acc)[i,h] = (O_b, LSE_b)
 *   otherwise:      M = max(lse_acc, LSE_b), a = exp(lse_acc - M),
 *                   b = exp(LSE_b - M), o_acc = (a o_acc + b O_b) / (a + b),
 *                   lse_acc = M + ln(a + b)   (both -inf: O = 0, LSE = -inf)
 *   ZL_STEP_LAST:   the combined result goes to out (rounded to `dtype`) and
 *                   lse instead of o_acc / lse_acc.
 * o_acc [Tq,H,d] fp32 and lse_acc [Tq,H] fp32 are caller-owned, indexed by
 * packed query row like out/lse; only SHARD rows are read or written, and
 * they may be NULL when there are no SHARD rows or when flags is
 * ZL_STEP_FIRST|ZL_STEP_LAST.  Without ZL_STEP_FIRST they must hold the
 * previous step's result.  block_index and num_slots are not read (any
 * values, block_index may be NULL).  Calls
 * for different steps must be ordered on the stream (the accumulator is
 * read-modify-written).  Errors as zl_attn_fwd, plus ZL_ERR_INVALID_ARG for
 * a SHARD segment with kv_count != 1 or unknown flags.
 */
zl_status zl_attn_fwd_step(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim, zl_dtype dtype,
                           float softmax_scale, const void* q, const void* k, const void* v,
                           void* out, float* lse, float* o_acc, float* lse_acc, uint32_t flags,
                           void* stream);

/*
 * Ulysses (1,h,1) local staging (Sec. II-B; Tab. II; Sec. IV-D's coalesced
 * QKV-packed all-to-all): the layout kernels around one block-diagonal
 * attention call on a head subset.  A group of `group` ranks each hold a
 * token shard of every batched sequence with all num_heads heads; rank j
 * computes heads [j*Hl, (j+1)*Hl), Hl = num_heads / group, over the full
 * sequences.  The all-to-alls themselves are the caller's (RCCL); these calls
 * only lay out the buffers they move.  All tensors bf16, 16-byte aligned,
 * head_dim 64 or 128; rows of every layout are in sequence order.
 *
 *   zl_ulysses_pack_qkv    q, k, v [t_local, H, d] -> send [group][t_local][Hl][3][d]:
 *                          the chunk for rank j (contiguous) holds its heads, q/k/v
 *                          interleaved per head so one all-to-all moves all three.
 *   zl_ulysses_unpack_qkv  recv (rank-major: rank j's T_j rows, [T_j][Hl][3][d]) ->
 *                          q, k, v [T_full, Hl, d] in full-sequence order, ready for
 *                          zl_attn_fwd / zl_attn_bwd with WHOLE segments of the full
 *                          lengths and num_heads = Hl.
 *   zl_ulysses_pack_out    out [T_full, Hl, d] -> send, rank-major ([T_j][Hl][d] for
 *                          rank j: its shard rows of every sequence).
 *   zl_ulysses_unpack_out  recv [group][t_local][Hl][d] (rank j's head group) ->
 *                          out_local [t_local, H, d].
 *
 * cu_rank (HOST, [group][num_seqs+1], read during the call): cu_rank[j][s] is
 * where sequence s starts among rank j's local rows (cu_rank[j][0] = 0, non-
 * decreasing), so rank j holds T_j = cu_rank[j][num_seqs] rows and sequence s
 * has sum_j (cu_rank[j][s+1] - cu_rank[j][s]) tokens, rank j's shard after
 * those of ranks < j.  Shards may differ in length (all-to-all-v).  The
 * row map it implies is cached on the device like a work table.  Errors:
 * ZL_ERR_INVALID_ARG (group < 1, num_heads not a multiple of group, bad
 * cu_rank, NULL or misaligned pointers), ZL_ERR_UNSUPPORTED (dtype other
 * than bf16, head_dim), ZL_ERR_HIP; nothing is enqueued on error.
 */
zl_status zl_ulysses_pack_qkv(int32_t group, int32_t t_local, int32_t num_heads, int32_t head_dim, zl_dtype dtype,
                              const void* q, const void* k, const void* v, void* send, void* stream);
zl_status zl_ulysses_unpack_qkv(int32_t group, int32_t num_seqs, const int32_t* cu_rank, int32_t num_heads,
                                int32_t head_dim, zl_dtype dtype, const void* recv, void* q, void* k, void* v,
                                void* stream);
zl_status zl_ulysses_pack_out(int32_t group, int32_t num_seqs, const int32_t* cu_rank, int32_t num_heads,
                              int32_t head_dim, zl_dtype dtype, const void* out, void* send, void* stream);
zl_status zl_ulysses_unpack_out(int32_t group, int32_t t_local, int32_t num_heads, int32_t head_dim, zl_dtype dtype,
                                const void* recv, void* out_local, void* stream);

/*
 * LSE merge of shard partials into exact attention (the ring's output
 * accumulation, Sec. II-B).  For every SHARD row i and head h, over the slots
 * B of its blocks:  M = max_b LSE_b, LSE = M + ln sum_b exp(LSE_b - M),
 * O = sum_b exp(LSE_b - LSE) O_b; slots with LSE_b = -inf are ignored and a
 * row with no finite slot gets O = 0, LSE = -inf.  Writes out [Tq,H,d] in
 * `out_dtype` and lse [Tq,H] for SHARD rows only.
 */
zl_status zl_lse_merge(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim, zl_dtype out_dtype,
                       const float* o_part, const float* lse_part, int32_t num_slots,
                       void* out, float* lse, void* stream);

/* zl_lse_merge reading partials of `part_dtype` (ZL_FP32 or ZL_BF16, as
 * written by zl_attn_fwd_ex); otherwise identical. */
zl_status zl_lse_merge_ex(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim, zl_dtype out_dtype,
                          const void* o_part, zl_dtype part_dtype, const float* lse_part, int32_t num_slots,
                          void* out, float* lse, void* stream);

/*
 * Backward of the packed batch.  `out` and `lse` are the FINAL outputs (for
 * SHARD rows: merged over all blocks); dout is dL/dout.  With D_i = dO_i.O_i,
 * P_ij = exp(S_ij - LSE_i), dS_ij = P_ij (dO_i.v_j - D_i):
 *   dq_i = scale sum_j dS_ij k_j  (a SHARD row sums over all of its blocks),
 *   dk_j = scale sum_i dS_ij q_i,  dv_j = sum_i P_ij dO_i
 * (for a SHARD block: this query chunk's contribution).  All tensors in
 * `dtype` (ZL_BF16 only) except lse (fp32).  dq is [Tq,H,d] and every row of
 * it is written; dk, dv are [Tk,H,d]: every row of a range that a segment
 * uses is written (zeros for the ranges of a SHARD segment without query
 * rows, to which no query attends), rows of ranges no segment uses are not.
 * No atomics: results are deterministic.  `flags` must be 0.
 * workspace: at least zl_workspace_size(..., ZL_OP_BWD) bytes of device
 * memory, 256-byte aligned, used by this call until it completes.
 */
zl_status zl_attn_bwd(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim, zl_dtype dtype,
                      float softmax_scale, const void* q, const void* k, const void* v,
                      const void* out, const float* lse, const void* dout,
                      void* dq, void* dk, void* dv, uint32_t flags,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * Backward of one ring step (Sec. II-B ring attention, Tab. II (1,1,k); the
 * counterpart of zl_attn_fwd_step).  Every SHARD segment brings exactly one
 * K/V block (kv_count == 1; block_index may be NULL); out and lse are the
 * FINAL (merged) outputs of its rows.  The call writes that block's dK/dV
 * (this query chunk's contribution, for the block's owner) and folds the
 * block's dQ sum into the shard rows' running fp32 accumulator:
 *   flags & ZL_STEP_FIRST:  the accumulator starts from this block;
 *   flags & ZL_STEP_LAST:   dq (bf16) = scale * (accumulator + this block);
 *   otherwise the sum goes back to dq_acc and dq is not written for them.
 * WHOLE segments ride along in any step and are complete in it (dq, dk, dv
 * written).  FIRST|LAST equals zl_attn_bwd.  dq_acc: [Tq, H, d] fp32 device
 * memory indexed by packed query row (so a SHARD segment must occupy the
 * same packed rows in every step), caller-owned, 16-byte aligned; may be NULL
 * when flags is FIRST|LAST or no row is SHARD.  Sums are per row and head in
 * one workgroup: no atomics, deterministic.  Other arguments, workspace and
 * errors as zl_attn_bwd, plus ZL_ERR_INVALID_ARG for unknown flags, a SHARD
 * with kv_count != 1, or a missing dq_acc.
 */
zl_status zl_attn_bwd_step(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim, zl_dtype dtype,
                           float softmax_scale, const void* q, const void* k, const void* v,
                           const void* out, const float* lse, const void* dout,
                           void* dq, void* dk, void* dv, float* dq_acc, uint32_t flags,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of the static device scratch zl_attn_bwd_noalloc uses on each GPU. */
#define ZL_NOALLOC_SCRATCH_BYTES (32u << 20)

/*
 * zl_attn_bwd for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments and results as zl_attn_bwd with flags 0 (bit for bit: the same
 * work items on the same kernels), but no workspace argument and no
 * allocation on any call.  The batch's work tables (32 bytes per work item)
 * and its D / LSE*log2(e) workspace (8 bytes per query row and head, plus
 * 256-byte alignment) go into one library-owned static device array of
 * ZL_NOALLOC_SCRATCH_BYTES per GPU, held by every GPU the library runs on
 * until the process ends.  The tables are built on the host (and cached there
 * per descriptor) and copied into the array on `stream` by every call.
 * Errors: as zl_attn_bwd, plus ZL_ERR_WORKSPACE (nothing enqueued) when the
 * batch needs more than ZL_NOALLOC_SCRATCH_BYTES.  Every call on a GPU uses
 * that GPU's one array and overwrites what the last call left there: calls
 * ordered on one stream are safe, calls that overlap on one GPU (other
 * streams, other host threads) race.  Keep profiling off (it creates events).
 */
zl_status zl_attn_bwd_noalloc(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim, zl_dtype dtype,
                              float softmax_scale, const void* q, const void* k, const void* v,
                              const void* out, const float* lse, const void* dout,
                              void* dq, void* dk, void* dv, void* stream);

/*
 * Host-only view of the schedule a launch would use (no device work): the
 * work items of op in issue order, 8 int32 each:
 *   q_start, q_len, k_start, k_len, head, slot (-1 for WHOLE), segment, range.
 *   ZL_OP_FWD     query tiles of one (segment, head, range).
 *   ZL_OP_BWD     key tiles of one (segment, head, range) against all of the
 *                 segment's queries (they produce dK, dV).
 *   ZL_OP_BWD_DQ  query tiles of one (segment, head) against every key of
 *                 the segment, all of its ranges (they produce dQ); k_start is
 *                 the first range's first row, k_len the total key count,
 *                 slot -1, range the first range.
 * Order: cost = q_len * k_len descending, ties by (segment, head, q_start,
 * k_start, range) ascending.  Writes min(n, cap) items to `items` (may be
 * NULL when cap is 0) and the total count to *n.  *tile_m / *tile_n (may be
 * NULL) receive the query / key tile sizes of that schedule.
 */
zl_status zl_plan_dump(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim, zl_dtype dtype,
                       int32_t op, int32_t* items, size_t cap, size_t* n,
                       int32_t* tile_m, int32_t* tile_n);

/*
 * Filler Packing, Stage 2 of the two-stage planner (Sec. IV-C, Eq. 8).  Host
 * only: no device work, callable without a GPU.  Fillers stay whole and are
 * placed one at a time in decreasing price (equal prices keep their input
 * order).  With compute headroom h^C_r = F - C_r and memory headroom
 * h^M_r = M_cap - M_r, filler s may go to rank r when h^M_r >= M_{s,r}; it goes
 * to the feasible rank with the largest min((h^C_r - p_s) / F,
 * (h^M_r - M_{s,r}) / M_cap), the lowest rank on a tie, and that rank's
 * ledgers grow by p_s and M_{s,r}.  All arithmetic is IEEE double in exactly
 * that order, so the decisions are reproducible.
 *
 *   num_ranks    N >= 1;  num_fillers n >= 0
 *   price        [n]      p_s: the filler's profiled whole-sequence price (>= 0)
 *   mem          [n][N]   M_{s,whole,r}, row-major (>= 0)
 *   load_floor   F > 0: every batch sequence's whole price summed, over N
 *   mem_cap      M_cap > 0
 *   load         [N] in: C_r after anchor placement; out: plus the fillers placed
 *   mem_used     [N] in: M_r after anchor placement; out: likewise
 *   rank_of      [n] out: the rank of each filler, -1 if not placed
 *   failed       out (may be NULL): the first filler that fit on no rank, or -1
 * All arrays are caller-owned host memory; every value must be finite.
 * Returns ZL_OK when every filler is placed, ZL_ERR_INFEASIBLE when one fits
 * nowhere (planning fails; the outputs hold what was placed before it), and
 * ZL_ERR_INVALID_ARG (nothing written) for NULL arrays, negative or non-
 * finite values, or a non-positive F or M_cap.
 */
zl_status zl_fill_pack(int32_t num_ranks, int32_t num_fillers, const double* price, const double* mem,
                       double load_floor, double mem_cap, double* load, double* mem_used, int32_t* rank_of,
                       int32_t* failed);

/*
 * Per-kernel timing with HIP events (off by default).  While enabled, every
 * kernel this library launches is bracketed by two events recorded on the
 * stream it is launched on.  zl_profile_read waits for the pending events of
 * one kernel family, adds their elapsed times to its totals and returns the
 * totals since the last reset.  Kernel ids: ZL_K_FWD, ZL_K_MERGE,
 * ZL_K_BWD_PRE, ZL_K_BWD_DKDV, ZL_K_BWD_DQ, ZL_K_ULYSSES (the four Ulysses
 * staging calls together).
 */
enum {
  ZL_K_FWD = 0,
  ZL_K_MERGE = 1,
  ZL_K_BWD_PRE = 2,
  ZL_K_BWD_DKDV = 3,
  ZL_K_BWD_DQ = 4,
  ZL_K_ULYSSES = 5,
  ZL_K_COUNT = 6
};
zl_status zl_profile_enable(int32_t on);
zl_status zl_profile_read(int32_t kernel_id, double* total_ms, int64_t* launches);
void zl_profile_reset(void);

/* Releases the library's device work-table cache and any pending profiler
 * events (waits for the device first, so no enqueued kernel still reads a
 * table).  Graphs that captured library calls must not be replayed after it. */
void zl_shutdown(void);

#ifdef __cplusplus
}
#endif

#endif /* ZL_ATTN_H */
