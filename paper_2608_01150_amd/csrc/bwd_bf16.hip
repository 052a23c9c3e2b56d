// Packed whole+shard attention backward, bf16 inputs, gfx950 MFMA.
//
// Three launches on one stream:
//   1. preprocess  D_i = dO_i . O_i (fp32) for every query row and head, and
//                  zero the fp32 dQ accumulator.
//   2. main        one workgroup per work item = up to 128 keys of one head of
//                  one K/V range, looping over every query of the owning
//                  segment in steps of 32 rows.  Each wave owns 32 keys:
//                    S    = Q K^T        (recomputed)       MFMA
//                    P    = exp(S - LSE) with the FINAL LSE (a shard's merged
//                           statistic, so block contributions add up exactly)
//                    dP   = dO V^T                           MFMA
//                    dS   = P (dP - D)
//                    dV^T += dO^T P,  dK^T += Q^T dS         MFMA, in registers
//                    dQ  += dS K  over the 128 keys          MFMA, fp32 atomics
//                  A shard row's dQ collects all of its blocks' items through
//                  the atomics; each dK/dV row has exactly one owning item.
//   3. finalize    dQ (bf16) = scale * accumulator.
// Keeping one key per lane makes P and dS directly the B operands of the
// dV/dK products; Q and dO are staged in LDS both row-major (for S and dP)
// and transposed (for dK and dV), K transposed once per item (for dQ).

#include <algorithm>

#include "zl_device.h"
#include "zl_internal.h"

namespace zl {
namespace {

constexpr int NT = 256;
constexpr int BKEY = kBwdTileN;   // keys per item (4 waves x 32)
constexpr int BQ = kBwdTileM;     // queries per step

// ------------------------------------------------------------------ preprocess
template <int D>
__global__ __launch_bounds__(NT) void bwd_pre_kernel(BwdParams p) {
  constexpr int LPU = D / 8;  // lanes per (row, head) unit, 8 bf16 each
  const int sub = threadIdx.x % LPU;
  const int64_t u = (int64_t)blockIdx.x * (NT / LPU) + threadIdx.x / LPU;
  const int64_t n = p.total_q * p.num_heads;
  const bool live = u < n;
  float acc = 0.f;
  if (live) {
    const u32x4 a = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p.out) + u * D + sub * 8);
    const u32x4 b = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p.dout) + u * D + sub * 8);
#pragma unroll
    for (int t = 0; t < 4; ++t) acc += bf16_lo(a[t]) * bf16_lo(b[t]) + bf16_hi(a[t]) * bf16_hi(b[t]);
    float* z = p.dq_acc + u * D + sub * 8;
    *reinterpret_cast<f32x4*>(z) = f32x4{0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<f32x4*>(z + 4) = f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int off = LPU / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (live && sub == 0) p.dsum[u] = acc;
}

// ------------------------------------------------------------------ finalize
template <int D>
__global__ __launch_bounds__(NT) void bwd_fin_kernel(BwdParams p) {
  const int64_t n8 = p.total_q * p.num_heads * D / 8;
  for (int64_t e = (int64_t)blockIdx.x * NT + threadIdx.x; e < n8; e += (int64_t)gridDim.x * NT) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p.dq_acc + e * 8);
    const f32x4 b = *reinterpret_cast<const f32x4*>(p.dq_acc + e * 8 + 4);
    const u32x4 w = {pack_bf16(a[0] * p.scale, a[1] * p.scale), pack_bf16(a[2] * p.scale, a[3] * p.scale),
                     pack_bf16(b[0] * p.scale, b[1] * p.scale), pack_bf16(b[2] * p.scale, b[3] * p.scale)};
    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.dq) + e * 8) = w;
  }
}

// ------------------------------------------------------------------ main
// LDS layouts (bytes), all 16-byte chunks XOR-swizzled by row:
//   qs, dos  [BQ rows][D]     row-major   chunk ^ swz(row)
//   qt, dot  [D rows][BQ]     transposed  chunk ^ swz4(row)   (4 chunks per row)
//   kt       [D rows][BKEY]   transposed  chunk ^ swz(row)
//   ds       [BQ rows][BKEY]  row-major   chunk ^ (row & 7)
__device__ __forceinline__ int swz4(int r) { return ((r >> 1) & 1) | (((r >> 3) & 1) << 1); }

template <int D>
struct BwdSmem {
  char qs[BQ * D * 2];
  char dos[BQ * D * 2];
  char qt[D * BQ * 2];
  char dot[D * BQ * 2];
  char kt[D * BKEY * 2];
  char ds[BQ * BKEY * 2];
  float lse2[BQ];
  float dsum[BQ];
};

template <int D>
__device__ __forceinline__ uint32_t rm_off(int r, int c) { return r * (D * 2) + ((c ^ swz(r)) << 4); }
__device__ __forceinline__ uint32_t tq_off(int r, int c) { return r * (BQ * 2) + ((c ^ swz4(r)) << 4); }
__device__ __forceinline__ uint32_t kt_off(int r, int c) { return r * (BKEY * 2) + ((c ^ swz(r)) << 4); }
__device__ __forceinline__ uint32_t ds_off(int r, int c) { return r * (BKEY * 2) + ((c ^ (r & 7)) << 4); }

// dword of bf16 element pairs: (a[j], b[j]) -> lo | hi << 16
__device__ __forceinline__ uint32_t pair_elem(const u32x4& a, const u32x4& b, int j) {
  const uint32_t x = a[j >> 1], y = b[j >> 1];
  return (j & 1) ? ((x >> 16) | (y & 0xFFFF0000u)) : ((x & 0xFFFFu) | (y << 16));
}

template <int D>
__global__ __launch_bounds__(NT, 1) void bwd_main_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(16))) BwdSmem<D> sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ln = lane & 31, g = lane >> 5;
  const Item it = p.items[dispatch_item(blockIdx.x, p.n_items, p.xcd_chunk)];
  const int H = p.num_heads;
  const int64_t rs = (int64_t)H * D;
  const uint16_t* qg = static_cast<const uint16_t*>(p.q) + ((int64_t)it.q_start * H + it.head) * D;
  const uint16_t* dog = static_cast<const uint16_t*>(p.dout) + ((int64_t)it.q_start * H + it.head) * D;
  const uint16_t* kg = static_cast<const uint16_t*>(p.k) + ((int64_t)it.k_start * H + it.head) * D;
  const uint16_t* vg = static_cast<const uint16_t*>(p.v) + ((int64_t)it.k_start * H + it.head) * D;
  const float* lseg = p.lse + (int64_t)it.q_start * H + it.head;
  const float* dsg = p.dsum + (int64_t)it.q_start * H + it.head;
  float* dqg = p.dq_acc + ((int64_t)it.q_start * H + it.head) * D;

  // This lane's key (B-operand column) and its K, V fragments.
  const int key = wave * 32 + ln;
  const bool k_ok = key < it.k_len;
  u32x4 kf[D / 16], vf[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    kf[kk] = k_ok ? *reinterpret_cast<const u32x4*>(kg + key * rs + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
    vf[kk] = k_ok ? *reinterpret_cast<const u32x4*>(vg + key * rs + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
  }
  // K^T into LDS once: thread unit = (key pair, d chunk).
  for (int u = tid; u < (BKEY / 2) * (D / 8); u += NT) {
    const int pr = u % (BKEY / 2), cc = u / (BKEY / 2), k0 = 2 * pr;
    const u32x4 a = k0 < it.k_len ? *reinterpret_cast<const u32x4*>(kg + k0 * rs + cc * 8) : u32x4{0, 0, 0, 0};
    const u32x4 b = k0 + 1 < it.k_len ? *reinterpret_cast<const u32x4*>(kg + (k0 + 1) * rs + cc * 8)
                                      : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 8; ++j)
      *reinterpret_cast<uint32_t*>(sm.kt + kt_off(cc * 8 + j, pr >> 2) + (pr & 3) * 4) = pair_elem(a, b, j);
  }

  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
    dk[db] = f32x16{};
    dv[db] = f32x16{};
  }

  // dQ work split: d-block and key range of this wave.
  constexpr int NDB = D / 32;
  constexpr int WPB = 4 / NDB;            // waves per d-block
  constexpr int KSTEPS = BKEY / 16 / WPB; // 16-key MFMA steps per wave
  const int dq_db = wave % NDB, dq_kpart = wave / NDB;

  for (int q0 = 0; q0 < it.q_len; q0 += BQ) {
    const int nq = min(BQ, it.q_len - q0);
    __syncthreads();  // previous step's LDS reads are done
    // Stage Q and dO rows [q0, q0+BQ): unit = (query pair, d chunk).
    for (int u = tid; u < (BQ / 2) * (D / 8); u += NT) {
      const int pr = u % (BQ / 2), cc = u / (BQ / 2), r0 = 2 * pr;
      const u32x4 z = {0, 0, 0, 0};
      const u32x4 qa = r0 < nq ? *reinterpret_cast<const u32x4*>(qg + (q0 + r0) * rs + cc * 8) : z;
      const u32x4 qb = r0 + 1 < nq ? *reinterpret_cast<const u32x4*>(qg + (q0 + r0 + 1) * rs + cc * 8) : z;
      const u32x4 oa = r0 < nq ? *reinterpret_cast<const u32x4*>(dog + (q0 + r0) * rs + cc * 8) : z;
      const u32x4 ob = r0 + 1 < nq ? *reinterpret_cast<const u32x4*>(dog + (q0 + r0 + 1) * rs + cc * 8) : z;
      *reinterpret_cast<u32x4*>(sm.qs + rm_off<D>(r0, cc)) = qa;
      *reinterpret_cast<u32x4*>(sm.qs + rm_off<D>(r0 + 1, cc)) = qb;
      *reinterpret_cast<u32x4*>(sm.dos + rm_off<D>(r0, cc)) = oa;
      *reinterpret_cast<u32x4*>(sm.dos + rm_off<D>(r0 + 1, cc)) = ob;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t off = tq_off(cc * 8 + j, pr >> 2) + (pr & 3) * 4;
        *reinterpret_cast<uint32_t*>(sm.qt + off) = pair_elem(qa, qb, j);
        *reinterpret_cast<uint32_t*>(sm.dot + off) = pair_elem(oa, ob, j);
      }
    }
    if (tid < BQ) {
      // Rows past the segment get LSE = +big so that P = 0 there.
      sm.lse2[tid] = tid < nq ? lseg[(int64_t)(q0 + tid) * H] * 1.4426950408889634f : 1.0e30f;
      sm.dsum[tid] = tid < nq ? dsg[(int64_t)(q0 + tid) * H] : 0.f;
    }
    __syncthreads();

    // S and dP: D row m <-> query perm32(m); register i <-> query 16*(i/8)+8g+i%8.
    f32x16 s = f32x16{}, dp = f32x16{};
    const int qrow = perm32(ln);
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(sm.qs + rm_off<D>(qrow, 2 * kk + g));
      s = mfma32(a, kf[kk], s);
      const u32x4 b = *reinterpret_cast<const u32x4*>(sm.dos + rm_off<D>(qrow, 2 * kk + g));
      dp = mfma32(b, vf[kk], dp);
    }
    u32x4 pp[2], pds[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const f32x4 l0 = *reinterpret_cast<const f32x4*>(&sm.lse2[16 * h + 8 * g]);
      const f32x4 l1 = *reinterpret_cast<const f32x4*>(&sm.lse2[16 * h + 8 * g + 4]);
      const f32x4 d0 = *reinterpret_cast<const f32x4*>(&sm.dsum[16 * h + 8 * g]);
      const f32x4 d1 = *reinterpret_cast<const f32x4*>(&sm.dsum[16 * h + 8 * g + 4]);
      float pv[8], dsv[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float l2 = t < 4 ? l0[t] : l1[t - 4];
        const float dd = t < 4 ? d0[t] : d1[t - 4];
        const int i = 8 * h + t;
        const float pr = k_ok ? fast_exp2(s[i] * p.scale_log2 - l2) : 0.f;
        pv[t] = pr;
        dsv[t] = pr * (dp[i] - dd);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        pp[h][t] = pack_bf16(pv[2 * t], pv[2 * t + 1]);
        pds[h][t] = pack_bf16(dsv[2 * t], dsv[2 * t + 1]);
      }
      // dS to LDS as [query][key] for the dQ product.
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int qq = 16 * h + 8 * g + t;
        const int kc = wave * 32 + ln;
        const __bf16 bv = (__bf16)dsv[t];
        *reinterpret_cast<uint16_t*>(sm.ds + ds_off(qq, kc >> 3) + (kc & 7) * 2) = __builtin_bit_cast(uint16_t, bv);
      }
    }
    // dV^T += dO^T P and dK^T += Q^T dS; A row m <-> d = db*32 + perm32(m).
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const int drow = db * 32 + perm32(ln);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(sm.dot + tq_off(drow, 2 * h + g));
        dv[db] = mfma32(a, pp[h], dv[db]);
        const u32x4 b = *reinterpret_cast<const u32x4*>(sm.qt + tq_off(drow, 2 * h + g));
        dk[db] = mfma32(b, pds[h], dk[db]);
      }
    }
    __syncthreads();  // dS of every wave is in LDS

    // dQ[q, d] = sum_key dS[q, key] K[key, d] for this wave's d-block and key part.
    // A = dS rows (query m = lane%32) from LDS, B = K^T rows (d) from LDS, so a
    // D register holds one query row and the 32 lanes of a half-wave hold 32
    // consecutive d: every atomic instruction covers two 128-byte row pieces.
    f32x16 dq = f32x16{};
    const int dcol = dq_db * 32 + ln;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const int kc = dq_kpart * KSTEPS * 2 + 2 * ks + g;  // 8-key chunk index
      const u32x4 a = *reinterpret_cast<const u32x4*>(sm.ds + ds_off(ln, kc));
      const u32x4 b = *reinterpret_cast<const u32x4*>(sm.kt + kt_off(dcol, kc));
      dq = mfma32(a, b, dq);
    }
    // dq[i] is (query 8*(i/4) + 4*g + i%4, d = dcol).
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int qq = 8 * (i >> 2) + 4 * g + (i & 3);
      if (qq < nq) unsafeAtomicAdd(dqg + (int64_t)(q0 + qq) * rs + dcol, dq[i]);
    }
  }

  // dK = scale * dK^T, dV = dV^T: register i <-> d = db*32 + 16*(i/8) + 8g + i%8, key = lane's key.
  if (!k_ok) return;
  uint16_t* dkg = static_cast<uint16_t*>(p.dk) + ((int64_t)(it.k_start + key) * H + it.head) * D;
  uint16_t* dvg = static_cast<uint16_t*>(p.dv) + ((int64_t)(it.k_start + key) * H + it.head) * D;
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      u32x4 wk, wv;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        wk[t] = pack_bf16(dk[db][8 * h + 2 * t] * p.scale, dk[db][8 * h + 2 * t + 1] * p.scale);
        wv[t] = pack_bf16(dv[db][8 * h + 2 * t], dv[db][8 * h + 2 * t + 1]);
      }
      *reinterpret_cast<u32x4*>(dkg + db * 32 + 16 * h + 8 * g) = wk;
      *reinterpret_cast<u32x4*>(dvg + db * 32 + 16 * h + 8 * g) = wv;
    }
  }
}

}  // namespace

hipError_t launch_bwd_bf16(const BwdParams& p, int head_dim, int stage, hipStream_t s) {
  const int64_t units = p.total_q * p.num_heads;
  const dim3 block(NT);
  if (stage == 0) {
    const int upb = NT / (head_dim / 8);
    const dim3 grid((unsigned)((units + upb - 1) / upb));
    if (head_dim == 128) hipLaunchKernelGGL(bwd_pre_kernel<128>, grid, block, 0, s, p);
    else hipLaunchKernelGGL(bwd_pre_kernel<64>, grid, block, 0, s, p);
  } else if (stage == 1) {
    if (p.n_items == 0) return hipSuccess;
    if (head_dim == 128) hipLaunchKernelGGL(bwd_main_kernel<128>, dim3(p.n_items), block, 0, s, p);
    else hipLaunchKernelGGL(bwd_main_kernel<64>, dim3(p.n_items), block, 0, s, p);
  } else {
    const int64_t n8 = units * head_dim / 8;
    const dim3 grid((unsigned)std::min<int64_t>((n8 + NT - 1) / NT, 65536));
    if (head_dim == 128) hipLaunchKernelGGL(bwd_fin_kernel<128>, grid, block, 0, s, p);
    else hipLaunchKernelGGL(bwd_fin_kernel<64>, grid, block, 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace zl
