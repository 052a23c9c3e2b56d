// Packed whole+shard attention forward, bf16 inputs, gfx950 MFMA.
//
// One workgroup (4 waves) takes one work item: up to 128 query rows of one
// head against one K/V range (a whole segment's own keys, or one CP block of
// a shard, Sec. IV-D / Tab. II of arXiv 2608.01150).  Each wave owns 32 query
// rows.  Per 64-key step:
//   S^T = K Q^T          MFMA 32x32x16 bf16, K from LDS (A), Q in registers (B)
//   online softmax       per query in the lane's registers (exp2 domain)
//   O^T += V^T P^T       MFMA, V^T from LDS (A), P^T straight from registers (B)
// Computing the transposed products keeps one query per lane, so the row max
// needs a single cross-lane exchange (lanes l and l^32) and the softmax
// output is already the B operand of the next MFMA.  K and V tiles for the
// next step are fetched into registers while the current step computes.
//
// Epilogue: WHOLE items write the final bf16 output and the LSE; SHARD items
// write the block-normalised fp32 partial and its LSE into their CP slot.

#include "zl_device.h"
#include "zl_internal.h"

namespace zl {
namespace {

constexpr int BM = kFwdTileM;
constexpr int BN = kFwdTileN;
constexpr int NT = 256;

template <int D>
struct FwdTile {
  static constexpr int KCH = D / 8;                  // 16-byte chunks per K row
  static constexpr int K_LOADS = BN * KCH / NT;      // 16-byte K chunks per thread
  static constexpr int V_UNITS = (BN / 2) * KCH / NT;  // (key pair, chunk) units per thread
};

// Byte offset of 16-byte chunk `c` of K row `r` in the swizzled K tile.
template <int D>
__device__ __forceinline__ uint32_t k_off(int r, int c) {
  return r * (D * 2) + ((c ^ swz(r)) << 4);
}
// Byte offset of 16-byte chunk `c` (8 keys) of V^T row `d` (64 keys = 128 B).
__device__ __forceinline__ uint32_t vt_off(int d, int c) { return d * (BN * 2) + ((c ^ swz(d)) << 4); }

template <int D>
__global__ __launch_bounds__(NT, 2) void fwd_bf16_kernel(FwdParams p) {
  using T = FwdTile<D>;
  __shared__ __attribute__((aligned(16))) char smem_k[BN * D * 2];
  __shared__ __attribute__((aligned(16))) char smem_vt[D * BN * 2];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ln = lane & 31, g = lane >> 5;
  const Item it = p.items[dispatch_item(blockIdx.x, p.n_items, p.xcd_chunk)];
  const int64_t rs = (int64_t)p.num_heads * D;  // elements between consecutive tokens
  const uint16_t* qg = static_cast<const uint16_t*>(p.q) + ((int64_t)it.q_start * p.num_heads + it.head) * D;
  const uint16_t* kg = static_cast<const uint16_t*>(p.k) + ((int64_t)it.k_start * p.num_heads + it.head) * D;
  const uint16_t* vg = static_cast<const uint16_t*>(p.v) + ((int64_t)it.k_start * p.num_heads + it.head) * D;

  // Q fragments (B operand): query row wave*32+ln, d = 16*kk + 8*g .. +7.
  const int qr = wave * 32 + ln;
  const bool q_ok = qr < it.q_len;
  u32x4 qf[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    qf[kk] = q_ok ? *reinterpret_cast<const u32x4*>(qg + qr * rs + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
  }

  float m_run = kNegBig, l_part = 0.f;
  f32x16 o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) o[db] = f32x16{};

  u32x4 kreg[T::K_LOADS];
  u32x4 vreg[T::V_UNITS][2];

  auto fetch = [&](int kt) {
    const int nvalid = it.k_len - kt;
#pragma unroll
    for (int r = 0; r < T::K_LOADS; ++r) {
      const int c = tid + r * NT, row = c / T::KCH, col = c % T::KCH;
      kreg[r] = row < nvalid ? *reinterpret_cast<const u32x4*>(kg + (kt + row) * rs + col * 8) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int r = 0; r < T::V_UNITS; ++r) {
      const int u = tid + r * NT, pr = u % (BN / 2), cc = u / (BN / 2);
      const int k0 = 2 * pr;
      vreg[r][0] = k0 < nvalid ? *reinterpret_cast<const u32x4*>(vg + (kt + k0) * rs + cc * 8) : u32x4{0, 0, 0, 0};
      vreg[r][1] = k0 + 1 < nvalid ? *reinterpret_cast<const u32x4*>(vg + (kt + k0 + 1) * rs + cc * 8)
                                   : u32x4{0, 0, 0, 0};
    }
  };

  auto stash = [&]() {
#pragma unroll
    for (int r = 0; r < T::K_LOADS; ++r) {
      const int c = tid + r * NT, row = c / T::KCH, col = c % T::KCH;
      *reinterpret_cast<u32x4*>(smem_k + k_off<D>(row, col)) = kreg[r];
    }
#pragma unroll
    for (int r = 0; r < T::V_UNITS; ++r) {
      const int u = tid + r * NT, pr = u % (BN / 2), cc = u / (BN / 2);
      // keys 2pr, 2pr+1 of d = 8cc+j go to V^T row 8cc+j as one dword
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t a = vreg[r][0][j >> 1], b = vreg[r][1][j >> 1];
        const uint32_t w = (j & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
        const int d = cc * 8 + j;
        *reinterpret_cast<uint32_t*>(smem_vt + vt_off(d, pr >> 2) + (pr & 3) * 4) = w;
      }
    }
  };

  if (it.k_len > 0) fetch(0);
  for (int kt = 0; kt < it.k_len; kt += BN) {
    __syncthreads();
    stash();
    __syncthreads();
    if (kt + BN < it.k_len) fetch(kt + BN);

    // S^T for keys [kb*32, kb*32+32): D row m <-> key kb*32 + perm32(m).
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x16{};
      const int krow = kb * 32 + perm32(ln);
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(smem_k + k_off<D>(krow, 2 * kk + g));
        s[kb] = mfma32(a, qf[kk], s[kb]);
      }
    }
    // s[kb][i] is (key kb*32 + 16*(i/8) + 8*g + i%8, query qr).
    const int nvalid = it.k_len - kt;
    float mt = kNegBig;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = kb * 32 + 16 * (i >> 3) + 8 * g + (i & 7);
        float x = s[kb][i] * p.scale_log2;
        if (nvalid < BN && key >= nvalid) x = kNegBig;
        s[kb][i] = x;
        mt = fmaxf(mt, x);
      }
    }
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = fast_exp2(m_run - m_new);
    m_run = m_new;
    float lsum = 0.f;
    u32x4 pb[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; i += 2) {
        const float e0 = fast_exp2(s[kb][i] - m_new), e1 = fast_exp2(s[kb][i + 1] - m_new);
        lsum += e0 + e1;
        pb[kb][i >> 3][(i & 7) >> 1] = pack_bf16(e0, e1);
      }
    }
    l_part = l_part * alpha + lsum;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int i = 0; i < 16; ++i) o[db][i] *= alpha;
    }
    // O^T[d, q] += sum_key V^T[d, key] P^T[key, q]; A row m <-> d = db*32 + perm32(m).
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const int vrow = db * 32 + perm32(ln);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const u32x4 a = *reinterpret_cast<const u32x4*>(smem_vt + vt_off(vrow, 4 * kb + 2 * s2 + g));
          o[db] = mfma32(a, pb[kb][s2], o[db]);
        }
      }
    }
  }

  // Epilogue.  o[db][i] is (d = db*32 + 16*(i/8) + 8*g + i%8, query qr).
  const float l = l_part + __shfl_xor(l_part, 32);
  const float inv = l > 0.f ? 1.f / l : 0.f;
  const float lse = l > 0.f ? (m_run + __log2f(l)) * kLn2 : -INFINITY;
  if (!q_ok) return;
  const int64_t row = (int64_t)(it.q_start + qr) * p.num_heads + it.head;
  if (it.slot < 0) {
    uint16_t* og = static_cast<uint16_t*>(p.out) + row * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        u32x4 w;
#pragma unroll
        for (int t = 0; t < 4; ++t) w[t] = pack_bf16(o[db][8 * h + 2 * t] * inv, o[db][8 * h + 2 * t + 1] * inv);
        *reinterpret_cast<u32x4*>(og + db * 32 + 16 * h + 8 * g) = w;
      }
    }
    if (g == 0) p.lse[row] = lse;
  } else {
    float* og = p.o_part + it.slot * p.slot_stride + row * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        f32x4 a, b;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          a[t] = o[db][8 * h + t] * inv;
          b[t] = o[db][8 * h + 4 + t] * inv;
        }
        *reinterpret_cast<f32x4*>(og + db * 32 + 16 * h + 8 * g) = a;
        *reinterpret_cast<f32x4*>(og + db * 32 + 16 * h + 8 * g + 4) = b;
      }
    }
    if (g == 0) p.lse_part[it.slot * p.lse_slot_stride + row] = lse;
  }
}

}  // namespace

hipError_t launch_fwd_bf16(const FwdParams& p, int head_dim, hipStream_t s) {
  const dim3 grid(p.n_items), block(NT);
  if (head_dim == 128)
    hipLaunchKernelGGL(fwd_bf16_kernel<128>, grid, block, 0, s, p);
  else
    hipLaunchKernelGGL(fwd_bf16_kernel<64>, grid, block, 0, s, p);
  return hipGetLastError();
}

}  // namespace zl
