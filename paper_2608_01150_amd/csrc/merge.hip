// LSE merge of shard partials: the ring's output accumulation (Sec. II-B of
// arXiv 2608.01150), done once over all blocks of every shard row.
//
// A unit is one (shard row, head).  D/4 (fp32 partials) or D/8 (bf16)
// consecutive lanes own a unit, each holding 4 or 8 consecutive values of the
// row, so every slot's partial row is read with one fully coalesced 16-byte
// load per lane.  Slots are taken
// in passes of 8 whose loads are all issued before any is used, combined
// online across passes (running maximum and sum).  The kernel is HBM-bound:
// per unit it reads S*(4d+4) bytes (S*(2d+4) with bf16 partials, one 8-byte
// load per lane and slot) and writes 2d+4 (bf16) or 4d+4 bytes.

#include "zl_device.h"
#include "zl_internal.h"

namespace zl {
namespace {

constexpr int NT = 256;
constexpr int kSlotsPerPass = 8;

template <int D, bool OUT_BF16, bool PART_BF16>
__global__ __launch_bounds__(NT) void merge_kernel(MergeParams p) {
  // A lane holds E consecutive values of the row: 4 fp32 or 8 bf16 partial
  // values, so each slot is read with one 16-byte load per lane either way.
  constexpr int E = PART_BF16 ? 8 : 4;
  constexpr int LPU = D / E;           // lanes per unit
  constexpr int UPB = NT / LPU;        // units per block
  const int sub = threadIdx.x % LPU;
  const int64_t u = (int64_t)blockIdx.x * UPB + threadIdx.x / LPU;
  if (u >= p.n_units) return;

  // Segment of this unit: the last segment whose unit_start <= u.
  int lo = 0, hi = p.n_segs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.segs[mid].unit_start <= u) lo = mid; else hi = mid - 1;
  }
  const MergeSeg sg = p.segs[lo];
  const int64_t row = (int64_t)sg.row_start * p.num_heads + (u - sg.unit_start);  // token*H + head
  const int32_t* slots = p.slots + sg.slot_first;

  // Online combine over passes of up to 8 slots: every pass issues all of its
  // LSE and partial loads before using any.  m is the running maximum, l the
  // running sum of exp(LSE_b - m), acc the running sum of exp(LSE_b - m) O_b.
  float m = -INFINITY, l = 0.f;
  float acc[E];
#pragma unroll
  for (int t = 0; t < E; ++t) acc[t] = 0.f;
  for (int b0 = 0; b0 < sg.slot_count; b0 += kSlotsPerPass) {
    const int nb = min(kSlotsPerPass, sg.slot_count - b0);
    float lb[kSlotsPerPass];
    u32x4 ob[kSlotsPerPass];
#pragma unroll
    for (int b = 0; b < kSlotsPerPass; ++b) {
      lb[b] = -INFINITY;
      ob[b] = u32x4{0u, 0u, 0u, 0u};
      if (b < nb) {
        const int64_t sl = slots[b0 + b];
        lb[b] = p.lse_part[sl * p.lse_slot_stride + row];
        const char* src = static_cast<const char*>(p.o_part) + (sl * p.slot_stride + row * D) * (PART_BF16 ? 2 : 4);
        ob[b] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src) + sub);
      }
    }
    float mb = lb[0];
#pragma unroll
    for (int b = 1; b < kSlotsPerPass; ++b) mb = fmaxf(mb, lb[b]);
    if (mb == -INFINITY) continue;  // every slot of this pass is empty
    const float mn = fmaxf(m, mb);
    const float r = expf(m - mn);   // 0 while m is still -inf
    l *= r;
#pragma unroll
    for (int t = 0; t < E; ++t) acc[t] *= r;
#pragma unroll
    for (int b = 0; b < kSlotsPerPass; ++b) {
      const float w = expf(lb[b] - mn);  // 0 for empty slots
      l += w;
#pragma unroll
      for (int t = 0; t < E; ++t) {
        const float x = PART_BF16 ? ((t & 1) ? bf16_hi(ob[b][t >> 1]) : bf16_lo(ob[b][t >> 1]))
                                  : __uint_as_float(ob[b][t]);
        acc[t] = fmaf(w, x, acc[t]);
      }
    }
    m = mn;
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
  const float lse = l > 0.f ? m + logf(l) : -INFINITY;
#pragma unroll
  for (int t = 0; t < E; ++t) acc[t] *= inv;
  if constexpr (OUT_BF16) {
    uint32_t wv[E / 2];
#pragma unroll
    for (int t = 0; t < E / 2; ++t) wv[t] = pack_bf16(acc[2 * t], acc[2 * t + 1]);
    uint16_t* dst = static_cast<uint16_t*>(p.out) + row * D + sub * E;
    if constexpr (E == 8) *reinterpret_cast<u32x4*>(dst) = u32x4{wv[0], wv[1], wv[2], wv[3]};
    else *reinterpret_cast<u32x2*>(dst) = u32x2{wv[0], wv[1]};
  } else {
    float* dst = static_cast<float*>(p.out) + row * D + sub * E;
#pragma unroll
    for (int t = 0; t < E; t += 4) *reinterpret_cast<f32x4*>(dst + t) = f32x4{acc[t], acc[t + 1], acc[t + 2], acc[t + 3]};
  }
  if (sub == 0) p.lse[row] = lse;
}

}  // namespace

template <int D, bool OUT_BF16>
void launch_merge_d(const MergeParams& p, bool part_bf16, dim3 grid, dim3 block, hipStream_t s) {
  if (part_bf16) hipLaunchKernelGGL((merge_kernel<D, OUT_BF16, true>), grid, block, 0, s, p);
  else hipLaunchKernelGGL((merge_kernel<D, OUT_BF16, false>), grid, block, 0, s, p);
}

hipError_t launch_merge(const MergeParams& p, int head_dim, bool out_bf16, bool part_bf16, hipStream_t s) {
  const int upb = NT / (head_dim / (part_bf16 ? 8 : 4));  // units per block (see merge_kernel)
  const dim3 grid((unsigned)((p.n_units + upb - 1) / upb)), block(NT);
  if (head_dim == 128) {
    if (out_bf16) launch_merge_d<128, true>(p, part_bf16, grid, block, s);
    else launch_merge_d<128, false>(p, part_bf16, grid, block, s);
  } else {
    if (out_bf16) launch_merge_d<64, true>(p, part_bf16, grid, block, s);
    else launch_merge_d<64, false>(p, part_bf16, grid, block, s);
  }
  return hipGetLastError();
}

}  // namespace zl
