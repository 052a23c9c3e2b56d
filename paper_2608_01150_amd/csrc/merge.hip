// LSE merge of shard partials: the ring's output accumulation (Sec. II-B of
// arXiv 2608.01150), done once over all blocks of every shard row.
//
// A unit is one (shard row, head).  D/4 consecutive lanes own a unit, each
// holding 4 consecutive fp32 of the output row, so every slot's partial row
// is read with one fully coalesced 16-byte load per lane.  Slots are taken
// in passes of 8 whose loads are all issued before any is used, combined
// online across passes (running maximum and sum).  The kernel is HBM-bound:
// per unit it reads S*(4d+4) bytes and writes 2d+4 (bf16) or 4d+4 bytes.

#include "zl_device.h"
#include "zl_internal.h"

namespace zl {
namespace {

constexpr int NT = 256;
constexpr int kSlotsPerPass = 8;

template <int D, bool OUT_BF16>
__global__ __launch_bounds__(NT) void merge_kernel(MergeParams p) {
  constexpr int LPU = D / 4;           // lanes per unit
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
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int b0 = 0; b0 < sg.slot_count; b0 += kSlotsPerPass) {
    const int nb = min(kSlotsPerPass, sg.slot_count - b0);
    float lb[kSlotsPerPass];
    f32x4 ob[kSlotsPerPass];
#pragma unroll
    for (int b = 0; b < kSlotsPerPass; ++b) {
      lb[b] = -INFINITY;
      ob[b] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (b < nb) {
        const int64_t sl = slots[b0 + b];
        lb[b] = p.lse_part[sl * p.lse_slot_stride + row];
        ob[b] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p.o_part + sl * p.slot_stride + row * D) + sub);
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
    for (int t = 0; t < 4; ++t) acc[t] *= r;
#pragma unroll
    for (int b = 0; b < kSlotsPerPass; ++b) {
      const float w = expf(lb[b] - mn);  // 0 for empty slots
      l += w;
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[t] = fmaf(w, ob[b][t], acc[t]);
    }
    m = mn;
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
  const float lse = l > 0.f ? m + logf(l) : -INFINITY;
#pragma unroll
  for (int t = 0; t < 4; ++t) acc[t] *= inv;
  if constexpr (OUT_BF16) {
    u32x2 wv = {pack_bf16(acc[0], acc[1]), pack_bf16(acc[2], acc[3])};
    *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(p.out) + row * D + sub * 4) = wv;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(p.out) + row * D + sub * 4) = acc;
  }
  if (sub == 0) p.lse[row] = lse;
}

}  // namespace

hipError_t launch_merge(const MergeParams& p, int head_dim, bool out_bf16, hipStream_t s) {
  const int upb = NT / (head_dim / 4);
  const dim3 grid((unsigned)((p.n_units + upb - 1) / upb)), block(NT);
  if (head_dim == 128) {
    if (out_bf16) hipLaunchKernelGGL((merge_kernel<128, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((merge_kernel<128, false>), grid, block, 0, s, p);
  } else {
    if (out_bf16) hipLaunchKernelGGL((merge_kernel<64, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((merge_kernel<64, false>), grid, block, 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace zl
