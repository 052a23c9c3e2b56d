// Packed whole+shard attention forward in fp32, for plumbing runs.
//
// Same work items and outputs as the bf16 MFMA kernel, computed with plain
// fp32 VALU arithmetic: one query row per lane, keys visited one at a time
// with the online-softmax recurrence (running max m, running sum l, output
// rescaled by exp(m_old - m_new)), K/V tiles staged through LDS.

#include "zl_device.h"
#include "zl_internal.h"

namespace zl {
namespace {

constexpr int BM = kFwd32TileM;
constexpr int BN = kFwd32TileN;

template <int D>
__global__ __launch_bounds__(BM) void fwd_fp32_kernel(FwdParams p) {
  __shared__ __attribute__((aligned(16))) float ks[BN][D];
  __shared__ __attribute__((aligned(16))) float vs[BN][D];
  const Item it = p.items[blockIdx.x];
  const int tid = threadIdx.x;
  const int64_t rs = (int64_t)p.num_heads * D;
  const float* qg = static_cast<const float*>(p.q) + ((int64_t)it.q_start * p.num_heads + it.head) * D;
  const float* kg = static_cast<const float*>(p.k) + ((int64_t)it.k_start * p.num_heads + it.head) * D;
  const float* vg = static_cast<const float*>(p.v) + ((int64_t)it.k_start * p.num_heads + it.head) * D;
  const bool q_ok = tid < it.q_len;

  float q[D], o[D];
#pragma unroll
  for (int c = 0; c < D; ++c) {
    q[c] = q_ok ? qg[tid * rs + c] : 0.f;
    o[c] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int kt = 0; kt < it.k_len; kt += BN) {
    const int n = min(BN, it.k_len - kt);
    __syncthreads();
    for (int e = tid; e < BN * D / 4; e += BM) {
      const int r = e / (D / 4), c = (e % (D / 4)) * 4;
      f32x4 kv = {0.f, 0.f, 0.f, 0.f}, vv = {0.f, 0.f, 0.f, 0.f};
      if (r < n) {
        kv = *reinterpret_cast<const f32x4*>(kg + (kt + r) * rs + c);
        vv = *reinterpret_cast<const f32x4*>(vg + (kt + r) * rs + c);
      }
      *reinterpret_cast<f32x4*>(&ks[r][c]) = kv;
      *reinterpret_cast<f32x4*>(&vs[r][c]) = vv;
    }
    __syncthreads();
    for (int j = 0; j < n; ++j) {
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < D; ++c) s = fmaf(q[c], ks[j][c], s);
      s *= p.scale;
      const float m_new = fmaxf(m, s);
      const float a = expf(m - m_new), e = expf(s - m_new);
      l = l * a + e;
#pragma unroll
      for (int c = 0; c < D; ++c) o[c] = fmaf(e, vs[j][c], o[c] * a);
      m = m_new;
    }
  }
  if (!q_ok) return;
  const float inv = l > 0.f ? 1.f / l : 0.f;
  const float lse = l > 0.f ? m + logf(l) : -INFINITY;
  const int64_t row = (int64_t)(it.q_start + tid) * p.num_heads + it.head;
  if (it.slot >= 0 && p.step_mode) {
    // Ring step: fold this block into the running accumulator (see the bf16 kernel).
    float* acc = p.o_acc + row * D;
    float wa, wb, lse_new;
    step_weights(p.step_first, p.step_first ? 0.f : p.lse_acc[row], lse, wa, wb, lse_new);
    wb *= inv;
    float* og = p.step_last ? static_cast<float*>(p.out) + row * D : acc;
#pragma unroll
    for (int c = 0; c < D; c += 4) {
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
      if (!p.step_first) a = *reinterpret_cast<const f32x4*>(acc + c);
#pragma unroll
      for (int t = 0; t < 4; ++t) a[t] = wa * a[t] + wb * o[c + t];
      *reinterpret_cast<f32x4*>(og + c) = a;
    }
    (p.step_last ? p.lse : p.lse_acc)[row] = lse_new;
    return;
  }
  float* og = it.slot < 0 ? static_cast<float*>(p.out) + row * D : static_cast<float*>(p.o_part) + it.slot * p.slot_stride + row * D;
#pragma unroll
  for (int c = 0; c < D; c += 4) {
    *reinterpret_cast<f32x4*>(og + c) = f32x4{o[c] * inv, o[c + 1] * inv, o[c + 2] * inv, o[c + 3] * inv};
  }
  if (it.slot < 0)
    p.lse[row] = lse;
  else
    p.lse_part[it.slot * p.lse_slot_stride + row] = lse;
}

}  // namespace

hipError_t launch_fwd_fp32(const FwdParams& p, int head_dim, hipStream_t s) {
  const dim3 grid(p.n_items), block(BM);
  if (head_dim == 128)
    hipLaunchKernelGGL(fwd_fp32_kernel<128>, grid, block, 0, s, p);
  else
    hipLaunchKernelGGL(fwd_fp32_kernel<64>, grid, block, 0, s, p);
  return hipGetLastError();
}

}  // namespace zl
