// Packed whole+shard attention backward, bf16 inputs, gfx950 MFMA.
//
// Three launches on one stream, no atomics (results are deterministic):
//   1. preprocess  -D_i = -dO_i . O_i in fp32 for every query row and head
//                  (the dP MFMAs start their accumulation from it, so they
//                  produce dP - D directly), and LSE_i in log2 units.
//   2. dK/dV       an item = up to 128 keys of one head of one K/V range,
//                  looping over every query of the owning segment in steps
//                  of 64 rows.  One key per lane:
//                    S    = Q K^T,  dP = dO V^T      MFMA (K, V in registers)
//                    P    = exp(S - LSE_final),  dS = P (dP - D)
//                    dV^T += dO^T P,  dK^T += Q^T dS MFMA (P, dS as B operands)
//                  split between producer and consumer waves (see the kernel).
//                  LSE_final is a shard row's merged statistic, so each block's
//                  contribution is its exact share of the whole gradient.
//   3. dQ          an item = up to 256 query rows (8 waves x 32) of one head,
//                  looping over every key of the segment (all of a shard's
//                  blocks) in steps of 64.  One query per lane:
//                    S^T = K Q^T,  dP^T = V dO^T      MFMA (Q, dO in registers)
//                    dS^T = P^T (dP^T - D)
//                    dQ^T += K^T dS^T                 MFMA
//                  A shard row sums its blocks inside one item.
// Both run one workgroup per CU that takes items one after another from the
// launch's work queues (zl_device.h).  Q/dO (dK/dV) and K/V (dQ) tiles are
// staged row-major (padded pitch, conflict-free) in rotating LDS buffers by
// direct buffer-to-LDS loads issued ahead of use; the transposed operands
// (Q^T, dO^T, K^T) come straight from the row-major tiles through LDS
// transpose reads.

#include <algorithm>

#include "zl_device.h"
#include "zl_internal.h"

namespace zl {
namespace {

constexpr int NT = 256;

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
  }
#pragma unroll
  for (int off = LPU / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (live && sub == 0) {
    p.dsum[u] = -acc;
    p.lse2[u] = p.lse[u] * 1.4426950408889634f;
  }
}

// ------------------------------------------------------------------ dK / dV
// Warp-specialised: a workgroup of 8 waves takes 128 keys, as four key groups
// of 32.  Producer wave w (0-3) holds key group w; consumer waves 4-7 each
// hold the dV or dK accumulators of one half of d for all 128 keys (see the
// consumer), and every SIMD runs one producer and one consumer.  The segment's queries are
// processed as 32-query sub-blocks k (two per 64-query tile):
//   A(k)  producer: S = Q K^T, dP = dO V^T (MFMA, K and V in registers)
//   B(k)  producer: P = exp(S - LSE), dS = P (dP - D) (VALU), written to LDS
//         as the consumer's bf16 B operands
//   C(k)  consumers: dV^T += dO^T P, dK^T += Q^T dS (MFMA, dO^T and Q^T by
//         transpose reads of the staged tiles)
// Phase j (ended by a workgroup barrier) runs A(j) interleaved with B(j-1) on
// the producer and C(j-2) on the consumer, so each SIMD always has MFMA work
// from both waves and the producer's softmax hides under MFMAs.  Each role
// fits in half the register file (two waves per SIMD).  Tile t (sub-blocks
// 2t, 2t+1) is live from phase 2t to 2t+3; Q/dO tiles rotate through three
// buffers and tile t+1 is fetched at the start of phase 2t.
constexpr int kDkdvThreads = 512;

template <int D>
__global__ __launch_bounds__(kDkdvThreads, 1) void bwd_dkdv_kernel(BwdParams p) {
  constexpr int BQ = kBwdTileM;                 // 64 queries per tile
  constexpr int PITCH = Pad<D>::PITCH;
  constexpr int TILE = BQ * PITCH;              // bytes of one Q (or dO) tile
  constexpr int NBUF = 3;
  constexpr int NM = D / 8;                     // MFMAs per sub-block and role
  __shared__ __attribute__((aligned(16))) char qs[NBUF][TILE], dos[NBUF][TILE];
  __shared__ __attribute__((aligned(16))) float lss[NBUF][BQ], dss[NBUF][BQ];
  // P/dS exchange: [k%2][key group][word: P h0, P h1, dS h0, dS h1][lane].
  __shared__ __attribute__((aligned(16))) u32x4 xch[2][4][4][64];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool producer = wave < 4;
  const int kw = wave & 3;                      // key group
  const int ln = lane & 31, g = lane >> 5;
  const int H = p.num_heads;
  const int64_t rs = (int64_t)H * D;
  const int key = kw * 32 + ln;
  const uint32_t a_off = poff<D>(perm32(ln), g * 8);
  const uint32_t t_off = tr_lane_off<D>(lane);

  // Staging: producers load the Q tile and the tile's LSE (log2 units, even
  // waves) or D (odd waves; waves 2, 3 repeat 0, 1 with identical bytes);
  // consumers load the dO tile.  Rows past the segment read as zero (the
  // buffer range check), which adds exactly nothing to dK/dV: S = 0, dP = 0
  // and D = 0 give finite P and dS = 0, and the zero dO row cancels P in dV.
  // Tiles past the last one are fetched as all zero and never used.
  using Dma = TileDma<D, BQ>;
  const uint32_t row_bytes = (uint32_t)rs * 2u, stat_bytes = (uint32_t)H * 4u;
  Dma dma;
  dma.init(kw, lane, row_bytes);
  // Tile t of item `it` goes to buffer b = t % NBUF; callers pass b as a
  // literal so that every LDS address below folds to a per-lane base plus an
  // immediate.
  auto fetch = [&](const Item& it, int t, int b) __attribute__((always_inline)) {
    const int q0 = t * BQ, nq = it.q_len - q0;
    const int64_t row0 = (int64_t)(it.q_start + q0) * H + it.head;  // (row, head) of the tile's first query
    if (producer) {
      dma.issue(qs[b], static_cast<const uint16_t*>(p.q) + row0 * D, nq, row_bytes);
      const bool even = (kw & 1) == 0;
      const int nv = min(nq, BQ);
      const i32x4 rsrc = buf_rsrc((even ? p.lse2 : p.dsum) + row0, nv > 0 ? (nv - 1) * stat_bytes + 4u : 0u);
      dma4(rsrc, lane * stat_bytes, __builtin_amdgcn_readfirstlane(lds_addr(even ? lss[b] : dss[b])));
    } else {
      dma.issue(dos[b], static_cast<const uint16_t*>(p.dout) + row0 * D, nq, row_bytes);
    }
  };

  // Items from the launch's work queues, as in the forward.  Each role runs
  // its own item loop (their registers then need not coexist); both loops
  // pass the same barriers.  Thread 0 (a producer) claims the next item at
  // the start of the current item's last tile and publishes it through
  // s_item; next_item returns it to every wave, -1 at the end.
  __shared__ int s_item[2], s_tries;
  if (tid == 0) s_tries = 0;
  int parity = 0;
  auto next_item = [&](int pending) __attribute__((always_inline)) {
    const auto* pk = kernargs<BwdParams>();
    if (tid == 0)
      s_item[parity] = pk->wq_kv ? wq_next(pk->wq_kv, pk->n_kv_items, pk->xcd_chunk, &s_tries, pending) : -1;
    __syncthreads();  // also: both roles are done with this item's LDS
    const int idx = __builtin_amdgcn_readfirstlane(s_item[parity]);
    parity ^= 1;
    return idx;
  };
  const int first = dispatch_item(blockIdx.x, p.n_kv_items, p.xcd_chunk);

  if (producer) {
    // ---------------------------------------------------------- producer
    int pending = -1;
    for (int idx = first; idx >= 0; idx = next_item(pending)) {
      pending = -1;
      const Item it = p.kv_items[idx];
      const bool k_ok = key < it.k_len;
      const int nsteps = (it.q_len + BQ - 1) / BQ;  // tiles
      fetch(it, 0, 0);
      const uint16_t* kg = static_cast<const uint16_t*>(p.k) + ((int64_t)it.k_start * H + it.head) * D;
      const uint16_t* vg = static_cast<const uint16_t*>(p.v) + ((int64_t)it.k_start * H + it.head) * D;
      u32x4 kf[D / 16], vf[D / 16];
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        kf[kk] = k_ok ? *reinterpret_cast<const u32x4*>(kg + key * rs + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
        vf[kk] = k_ok ? *reinterpret_cast<const u32x4*>(vg + key * rs + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
      }
      // Retire the fragment loads (and tile 0) with a waitcnt the compiler
      // sees, so the loop carries no pending register loads.
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();  // tile 0 published

      constexpr int PFA = 4;
      // S and dP of sub-block k live in sc[k%2], dp[k%2]; register i <-> query
      // 32*(k%2) + 16*(i/8) + 8g + i%8 of tile k/2, lane = key.
      f32x16 sc[2], dp[2];
      // A(k) interleaved with B(k-1) (has_b); the A operand j is the Q (even j)
      // or dO (odd j) chunk j/2 of the sub-block's 32 rows.  Sub-block k is half
      // ka = k % 2 of the tile in buffer b; B(k-1) is half sbb of the tile in
      // buffer bb (all literals at the call sites).
      // A producer whose key group holds no key of the item (the ragged last
      // tile of a segment) skips its phases: their exchange words would only
      // feed the dK/dV of keys past the range, which are never stored.  Its
      // tile loads and barriers are outside the phases and still run.
      const bool live = kw * 32 < it.k_len;
      auto phase = [&](int ka, int b, int sbb, int bb, bool has_b, int xb) __attribute__((always_inline)) {
        if (!live) return;
        const char* qa = qs[b] + a_off + 32 * ka * PITCH;
        const char* oa = dos[b] + a_off + 32 * ka * PITCH;
        auto a_op = [&](int j) {
          return *reinterpret_cast<const u32x4*>(((j & 1) ? oa : qa) + poff<D>(0, (j >> 1) * 16));
        };
        // dP of sub-block k accumulates onto -D of its queries (staged with the
        // tile, in the accumulator's register order: register i <-> query
        // 16*(i/8) + 8g + i%8 of the sub-block), so it comes out as dP - D.
        f32x4 nd[2][2], lsv[2][2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
#pragma unroll
          for (int e = 0; e < 2; ++e)
            nd[h][e] = *reinterpret_cast<const f32x4*>(&dss[b][ka * 32 + 16 * h + 8 * g + 4 * e]);
        }
        u32x4 pp[2], pds[2];
        u32x4 ring[PFA];
#pragma unroll
        for (int j = 0; j < PFA; ++j) ring[j] = a_op(j);
        if (has_b) {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
#pragma unroll
            for (int e = 0; e < 2; ++e)
              lsv[h][e] = *reinterpret_cast<const f32x4*>(&lss[bb][sbb * 32 + 16 * h + 8 * g + 4 * e]);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        f32x16 s = f32x16{}, d_;
#pragma unroll
        for (int i = 0; i < 16; ++i) d_[i] = nd[i >> 3][(i >> 2) & 1][i & 3];
#pragma unroll
        for (int j = 0; j < NM; ++j) {
          const u32x4 a = ring[j % PFA];
          if (j + PFA < NM) ring[j % PFA] = a_op(j + PFA);
          if (j & 1)
            d_ = mfma32(a, vf[j >> 1], d_);
          else
            s = mfma32(a, kf[j >> 1], s);
          // Chunk c = j/(NM/8) of B(k-1): elements 2c, 2c+1 -> one packed word
          // of P and of dS.  A key past the range (k_ok false) only feeds its
          // own dK/dV, never stored.
          if (has_b && (j % (NM / 8)) == NM / 8 - 1) {
            const int c = j / (NM / 8), h = c >> 2, t2 = c & 3;
            float pv[2], dv_[2];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
              const int tt = 2 * t2 + e, i = 8 * h + tt;
              const float l2 = lsv[h][tt >> 2][tt & 3];
              pv[e] = fast_exp2(fmaf(sc[1 - ka][i], p.scale_log2, -l2));
              dv_[e] = pv[e] * dp[1 - ka][i];  // dp already holds dP - D
            }
            pp[h][t2] = pack_bf16(pv[0], pv[1]);
            pds[h][t2] = pack_bf16(dv_[0], dv_[1]);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
        // S and dP are read by the VALU in the next phase: move them to arch
        // VGPRs once, here, so they never share AGPRs with other MFMA results.
        asm volatile("" : "+v"(s), "+v"(d_));
        sc[ka] = s;
        dp[ka] = d_;
        if (has_b) {
          xch[xb][kw][0][lane] = pp[0];
          xch[xb][kw][1][lane] = pp[1];
          xch[xb][kw][2][lane] = pds[0];
          xch[xb][kw][3][lane] = pds[1];
        }
      };
      // Phase 0: A(0).  Phases 2t+1, 2t+2: A(2t+1)+B(2t), A(2t+2)+B(2t+1) (the
      // last A reads an all-zero tile past the end and is never used).  Phase
      // 2n+1: the consumer's last sub-block.  The tile loop is unrolled by
      // NBUF, r = t % NBUF.
      auto tile = [&](int t, int r) __attribute__((always_inline)) {
        phase(1, r, 0, r, true, 0);
        wait_vmem();  // own loads of tile t+1 landed
        __syncthreads();
        fetch(it, t + 2, (r + 2) % NBUF);
        if (t == nsteps - 1 && tid == 0 && p.wq_kv && s_tries < 8) pending = wq_claim(p.wq_kv, s_tries);
        phase(0, (r + 1) % NBUF, 1, r, true, 1);
        __syncthreads();
      };
      fetch(it, 1, 1);
      phase(0, 0, 0, 0, false, 0);
      __syncthreads();
      for (int t = 0; t < nsteps; t += NBUF) {
        tile(t, 0);
        if (t + 1 < nsteps) tile(t + 1, 1);
        if (t + 2 < nsteps) tile(t + 2, 2);
      }
      __syncthreads();
      wait_vmem();  // the lookahead loads must land before the LDS is reused
    }
    if (tid == 0 && p.wq_kv) wq_finish(p.wq_kv);
    return;
  }

  // ------------------------------------------------------------ consumer
  // Consumer wave 4 + ci owns one output, dV (ci < 2) or dK (ci >= 2), for
  // all 128 keys of the item and half of the d rows, dh = ci % 2.  Every
  // transpose-read operand (dO^T or Q^T rows of its d half) feeds four MFMAs,
  // one per key group, and the exchange words (P or dS of each key group) are
  // 16-byte reads: per sub-block 2*NDT operands of two transpose reads and
  // eight exchange reads for 16 MFMAs (d = 128).
  const int ci = wave - 4;
  const bool is_dk = ci >= 2;
  const int dh = ci & 1;
  constexpr int NDT = D / 64;                   // 32-row d tiles per consumer
  for (int idx = first; idx >= 0; idx = next_item(-1)) {
    const Item it = p.kv_items[idx];
    const int nsteps = (it.q_len + BQ - 1) / BQ;  // tiles
    fetch(it, 0, 0);
    f32x16 acc[4][NDT];                           // [key group][d tile]
#pragma unroll
    for (int kg = 0; kg < 4; ++kg) {
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) acc[kg][dt] = f32x16{};
    }
    wait_vmem();  // tile 0 landed (own loads)
    __syncthreads();  // tile 0 published

    // C(k): sub-block k = 2t + sb of tile t (buffer r), P or dS from exchange
    // buffer xb.  Operand (h, dt): rows d = (dh*NDT + dt)*32 + perm32(m) of dO^T
    // (dV) or Q^T (dK), k <-> queries 16h + 8g ... of the sub-block.
    auto phaseC = [&](int r, int sb, int xb) __attribute__((always_inline)) {
      const char* tbuf = (is_dk ? qs[r] : dos[r]) + t_off;
      u32x4 a[2][NDT], w[4][2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) a[h][dt] = tr_operand<D>(tbuf, sb * 32 + 16 * h, (dh * NDT + dt) * 32);
#pragma unroll
        for (int kg = 0; kg < 4; ++kg) w[kg][h] = xch[xb][kg][(is_dk ? 2 : 0) + h][lane];
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
#pragma unroll
          for (int kg = 0; kg < 4; ++kg) acc[kg][dt] = mfma32(a[h][dt], w[kg][h], acc[kg][dt]);
        }
      }
    };
    // Phases 0, 1: nothing to consume yet.  Phases 2t+2, 2t+3: C(2t), C(2t+1).
    auto tileC = [&](int t, int r) __attribute__((always_inline)) {
      fetch(it, t + 2, (r + 2) % NBUF);
      phaseC(r, 0, 0);
      __syncthreads();
      phaseC(r, 1, 1);
      wait_vmem();  // own loads of tile t+2 landed
      __syncthreads();
#pragma unroll
      for (int kg = 0; kg < 4; ++kg) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) asm volatile("" : "+v"(acc[kg][dt]));
      }
    };
    fetch(it, 1, 1);
    __syncthreads();
    wait_vmem();  // own loads of tile 1 landed
    __syncthreads();
    for (int t = 0; t < nsteps; t += NBUF) {
      tileC(t, 0);
      if (t + 1 < nsteps) tileC(t + 1, 1);
      if (t + 2 < nsteps) tileC(t + 2, 2);
    }

    // dK = scale * dK^T or dV = dV^T: register i <-> d = (dh*NDT + dt)*32 +
    // 16*(i/8) + 8g + i%8, key = key group kg's lane key.
    const float osc = is_dk ? p.scale : 1.f;
    uint16_t* og = static_cast<uint16_t*>(is_dk ? p.dk : p.dv);
#pragma unroll
    for (int kg = 0; kg < 4; ++kg) {
      const int okey = kg * 32 + ln;
      if (okey >= it.k_len) continue;
      uint16_t* dst = og + ((int64_t)(it.k_start + okey) * H + it.head) * D;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          u32x4 wo;
#pragma unroll
          for (int t = 0; t < 4; ++t)
            wo[t] = pack_bf16(acc[kg][dt][8 * h + 2 * t] * osc, acc[kg][dt][8 * h + 2 * t + 1] * osc);
          *reinterpret_cast<u32x4*>(dst + (dh * NDT + dt) * 32 + 16 * h + 8 * g) = wo;
        }
      }
    }
  }
}

// Epilogue of a dQ item for this lane's query row: dq[db][i] holds d = db*32 +
// 16*(i/8) + 8g + i%8.  Ring step, SHARD row: the block's raw sum is folded
// into the fp32 accumulator and only the last step writes dQ (one item per row
// and head: no atomics).
template <int D>
__device__ __forceinline__ void dq_store(const __attribute__((address_space(4))) BwdParams* pp, const Item& it,
                                         int64_t qrow, int g, const f32x16 (&dq)[D / 32]) {
  const auto& p = *pp;
  uint16_t* dqg = static_cast<uint16_t*>(p.dq) + qrow * D;
  if (!(p.step_mode && it.slot >= 0)) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        u32x4 w;
#pragma unroll
        for (int t = 0; t < 4; ++t)
          w[t] = pack_bf16(dq[db][8 * h + 2 * t] * p.scale, dq[db][8 * h + 2 * t + 1] * p.scale);
        *reinterpret_cast<u32x4*>(dqg + db * 32 + 16 * h + 8 * g) = w;
      }
    }
    return;
  }
  float* accg = p.dq_acc + qrow * D;
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int d0 = db * 32 + 16 * h + 8 * g;
      f32x4 a = {dq[db][8 * h], dq[db][8 * h + 1], dq[db][8 * h + 2], dq[db][8 * h + 3]};
      f32x4 b = {dq[db][8 * h + 4], dq[db][8 * h + 5], dq[db][8 * h + 6], dq[db][8 * h + 7]};
      f32x4* ap = reinterpret_cast<f32x4*>(accg + d0);
      if (!p.step_first) {
        a += ap[0];
        b += ap[1];
      }
      if (p.step_last) {
        const u32x4 w = {pack_bf16(a[0] * p.scale, a[1] * p.scale), pack_bf16(a[2] * p.scale, a[3] * p.scale),
                         pack_bf16(b[0] * p.scale, b[1] * p.scale), pack_bf16(b[2] * p.scale, b[3] * p.scale)};
        *reinterpret_cast<u32x4*>(dqg + d0) = w;
      } else {
        ap[0] = a;
        ap[1] = b;
      }
    }
  }
}

// ------------------------------------------------------------------ dQ
// An item is up to 256 query rows of one head (8 waves, two per SIMD, 32 query
// rows each).  A segment's K/V ranges are consecutive rows
// of K and V, and dQ sums over all of them against the final LSE, so the item
// streams the segment's keys [k_start, k_start + k_len) as one range: block
// boundaries play no part in the backward.  128-key K/V tiles rotate through
// two LDS buffers, fetched one tile ahead (waves 0-3 load K, 4-7 load V, each
// fetch's instructions spread over the S/dP MFMAs); a tile is two 64-key
// steps and one barrier.
constexpr int kDqThreads = 512;

template <int D>
__global__ __launch_bounds__(kDqThreads, 1) void bwd_dq_kernel(BwdParams p) {
  constexpr int BN = kDqTileN;                  // 64 keys per step
  constexpr int TN = 2 * BN;                    // keys per staged tile: two steps per barrier
  constexpr int PITCH = Pad<D>::PITCH;
  constexpr int TILE = TN * PITCH;
  using Dma = TileDma<D, BN>;                   // one 64-key half of a staged tile
  constexpr int DMA_PER_STEP = Dma::PER_WAVE;   // per wave and half (four waves share a tile)
  // Two buffers of each tile as separate objects (see the forward kernel).
  __shared__ __attribute__((aligned(16))) char ks0[TILE], ks1[TILE], vs0[TILE], vs1[TILE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ln = lane & 31, g = lane >> 5;
  // Items from the launch's work queues, as in the forward.
  __shared__ int s_item[2], s_tries;
  if (tid == 0) s_tries = 0;
  int pending = -1;
  int parity = 0;
  for (int idx = dispatch_item(blockIdx.x, p.n_q_items, p.xcd_chunk);;) {
    const Item it = p.q_items[idx];
    const int H = p.num_heads;
    const int64_t rs = (int64_t)H * D;

    // This lane's query row and its Q, dO fragments (B operands).
    const int qr = wave * 32 + ln;
    const bool q_ok = qr < it.q_len;
    const int64_t qrow = (int64_t)(it.q_start + qr) * H + it.head;
    const uint16_t* qg = static_cast<const uint16_t*>(p.q) + qrow * D;
    const uint16_t* dog = static_cast<const uint16_t*>(p.dout) + qrow * D;
    u32x4 qf[D / 16], of[D / 16];
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      qf[kk] = q_ok ? *reinterpret_cast<const u32x4*>(qg + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
      of[kk] = q_ok ? *reinterpret_cast<const u32x4*>(dog + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
    }
    const float lse2 = q_ok ? p.lse2[qrow] : 1.0e30f;  // +big: P = 0
    // -D of this lane's query, as the starting accumulator of every dP^T
    // block (all 16 registers hold the same query), so the MFMAs give dP - D.
    f32x16 negd;
    {
      const float nd = q_ok ? p.dsum[qrow] : 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) negd[i] = nd;
    }
    f32x16 dq[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) dq[db] = f32x16{};
    __builtin_amdgcn_s_waitcnt(0);  // prologue loads done (see the forward kernel)

    const uint32_t a_off = poff<D>(perm32(ln), g * 8);
    const uint32_t t_off = tr_lane_off<D>(lane);

    // Rows past the segment's keys read zero (the buffer range check).
    const uint16_t* kg = static_cast<const uint16_t*>(p.k) + ((int64_t)it.k_start * H + it.head) * D;
    const uint16_t* vg = static_cast<const uint16_t*>(p.v) + ((int64_t)it.k_start * H + it.head) * D;
    const bool loads_k = wave < 4;
    const uint16_t* src0 = loads_k ? kg : vg;
    const uint32_t row_bytes = (uint32_t)rs * 2u;
    Dma dma;
    dma.init(wave & 3, lane, row_bytes);
    auto fetch = [&](int kt, char* kdst, char* vdst) {
      char* dst = loads_k ? kdst : vdst;
      dma.issue(dst, src0 + (int64_t)kt * rs, it.k_len - kt, row_bytes);
      dma.issue(dst + BN * PITCH, src0 + (int64_t)(kt + BN) * rs, it.k_len - kt - BN, row_bytes);
    };
    // Inside the loop a fetch is only set up here; the S/dP MFMAs of the tile's
    // two steps issue its instructions one at a time, one half each.
    i32x4 next_rsrc[2];
    uint32_t next_lds[2];
    auto fetch_spread = [&](int kt, char* kdst, char* vdst) {
      char* dst = loads_k ? kdst : vdst;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        next_rsrc[h] = Dma::resource(src0 + (int64_t)(kt + h * BN) * rs, it.k_len - kt - h * BN, row_bytes);
        next_lds[h] = lds_addr(dst + h * BN * PITCH);
      }
    };

    // One 64-key step as two 32-key blocks kb, software-pipelined inside the
    // wave so that the softmax VALU work runs under MFMAs:
    //   S/dP MFMAs of kb 0; S/dP MFMAs of kb 1 with the softmax of kb 0;
    //   dQ MFMAs of kb 0 with the softmax of kb 1; dQ MFMAs of kb 1.
    // A operands come from LDS through a ring of loads issued PF MFMAs ahead.
    // half: which of the tile's two steps (0 or 1, a literal at the call sites).
    auto step = [&](const char* kbuf, const char* vbuf, int half) __attribute__((always_inline)) {
      const char* ka = kbuf + a_off;
      const char* va = vbuf + a_off;
      const char* kt_ = kbuf + t_off;
      constexpr int NSD = 2 * (D / 16) * 2;        // S/dP MFMAs per step (both key blocks)
      constexpr int NQ = 2 * (D / 32) * 2;         // dQ MFMAs per step
      // S/dP operand j: key block j/(NSD/2), d chunk (j%(NSD/2))/2, K (even j) or V (odd j).
      auto a_op = [&](int j) {
        return *reinterpret_cast<const u32x4*>(((j & 1) ? va : ka) +
                                               poff<D>((j / (NSD / 2)) * 32, ((j % (NSD / 2)) >> 1) * 16));
      };
      // dQ operand m: key block m/(NQ/2), d block (m%(NQ/2))/2, 16-key half m%2 (K^T by transpose reads).
      auto c_op = [&](int m) {
        return tr_operand<D>(kt_, (m / (NQ / 2)) * 32 + 16 * (m & 1), ((m % (NQ / 2)) >> 1) * 32);
      };
      constexpr int PF = 6, PFC = 3;
      constexpr int DMA_GAP = NSD / DMA_PER_STEP;  // S/dP MFMAs between the spread fetch's instructions
      static_assert(DMA_GAP >= 2 && (DMA_PER_STEP - 1) * DMA_GAP + 1 < NSD, "spread fetch must fit the S/dP MFMAs");
      // register i <-> key kb*32 + 16*(i/8) + 8g + i%8 of this tile, query = lane's row.
      // P is clamped to [0, 1] (exact: every true P is at most 1), a free
      // modifier of the exp.  That keeps dS finite for the keys past the
      // segment, whose K and V rows read as zero (S = 0, so P = 2^-lse2 could
      // overflow): their dS then multiplies a zero K row and adds exactly
      // nothing to dQ, so no per-key mask is needed.
      f32x16 sc[2], dpc[2];
      u32x4 pds[2][2];
      auto softmax2 = [&](int kb, int i) {  // elements i, i+1 of key block kb -> one packed dS word
        float e[2];
#pragma unroll
        for (int u = 0; u < 2; ++u)
          e[u] = __builtin_amdgcn_fmed3f(fast_exp2(fmaf(sc[kb][i + u], p.scale_log2, -lse2)), 0.f, 1.f) *
                 dpc[kb][i + u];
        pds[kb][i >> 3][(i & 7) >> 1] = pack_bf16(e[0], e[1]);
      };
      u32x4 ring[PF];
#pragma unroll
      for (int j = 0; j < PF; ++j) ring[j] = a_op(j);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) sc[kb] = f32x16{};
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < NSD; ++j) {
        const u32x4 a = ring[j % PF];
        if (j + PF < NSD) ring[j % PF] = a_op(j + PF);
        const int kb = j / (NSD / 2), kk = (j % (NSD / 2)) >> 1;
        if (j & 1)
          dpc[kb] = mfma32(a, of[kk], kk == 0 ? negd : dpc[kb]);
        else
          sc[kb] = mfma32(a, qf[kk], sc[kb]);
        if (j % DMA_GAP == 1 && j / DMA_GAP < DMA_PER_STEP) dma.issue_one(next_rsrc[half], next_lds[half], j / DMA_GAP);
        // kb 1's MFMAs carry kb 0's softmax: 16 elements over NSD/2 MFMAs.
        if (j >= NSD / 2 && ((j - NSD / 2) % (NSD / 16)) == NSD / 16 - 1) softmax2(0, 2 * ((j - NSD / 2) / (NSD / 16)));
        __builtin_amdgcn_sched_barrier(0);
      }
      u32x4 cring[PFC];
#pragma unroll
      for (int m = 0; m < PFC; ++m) cring[m] = c_op(m);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int m = 0; m < NQ; ++m) {
        const u32x4 a = cring[m % PFC];
        if (m + PFC < NQ) cring[m % PFC] = c_op(m + PFC);
        // kb 0's dQ MFMAs carry kb 1's softmax (finished before kb 1's MFMAs).
        if (m < NQ / 2) {
          softmax2(1, (16 / (NQ / 2)) * m);
          if (16 / (NQ / 2) == 4) softmax2(1, (16 / (NQ / 2)) * m + 2);
        }
        const int kb = m / (NQ / 2), db = (m % (NQ / 2)) >> 1, s2 = m & 1;
        dq[db] = mfma32(a, pds[kb][s2], dq[db]);
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    // Waves with no query rows skip the math (see the forward kernel).
    const bool wave_live = wave * 32 < it.q_len;
    auto run = [&](const char* kbuf, const char* vbuf, int half) __attribute__((always_inline)) {
      if (wave_live) {
        step(kbuf, vbuf, half);
      } else {
#pragma unroll
        for (int jj = 0; jj < DMA_PER_STEP; ++jj) dma.issue_one(next_rsrc[half], next_lds[half], jj);
      }
    };
    // One staged tile as two steps with no barrier between them (see the
    // forward kernel); keys past the range add zero, so a tile whose second
    // half lies past the range skips that step.
    auto tile = [&](const char* kbuf, const char* vbuf, int kt) __attribute__((always_inline)) {
      run(kbuf, vbuf, 0);
      if (kt + BN < it.k_len) run(kbuf + BN * PITCH, vbuf + BN * PITCH, 1);
    };

    auto claim_ahead = [&]() __attribute__((always_inline)) {
      if (tid == 0 && p.wq_q && s_tries < 8) pending = wq_claim(p.wq_q, s_tries);
    };

    // Two buffer sets in rotation, unrolled by two, as in the forward.  An
    // item without keys (a shard whose blocks are all empty) runs one step on
    // an all-zero tile, which adds exactly zero (K = 0), rather than branching
    // around the loop.
    fetch(0, ks0, vs0);
    for (int kt = 0;;) {
      wait_vmem();
      __syncthreads();  // tile in buffers 0 complete; buffers 1 no longer read
      fetch_spread(kt + TN, ks1, vs1);
      if (kt + TN >= it.k_len) claim_ahead();
      tile(ks0, vs0, kt);
      kt += TN;
      if (kt >= it.k_len) break;
      wait_vmem();
      __syncthreads();  // tile in buffers 1 complete; buffers 0 no longer read
      fetch_spread(kt + TN, ks0, vs0);
      if (kt + TN >= it.k_len) claim_ahead();
      tile(ks1, vs1, kt);
      kt += TN;
      if (kt >= it.k_len) break;
    }
    wait_vmem();  // the lookahead loads must land before the LDS is reused

    // dq[db][i] is (d = db*32 + 16*(i/8) + 8g + i%8, query qr).
    if (q_ok) dq_store<D>(kernargs<BwdParams>(), it, qrow, g, dq);
    const auto* pk = kernargs<BwdParams>();
    if (tid == 0) s_item[parity] = pk->wq_q ? wq_next(pk->wq_q, pk->n_q_items, pk->xcd_chunk, &s_tries, pending) : -1;
    pending = -1;
    __syncthreads();  // also: every wave is done with this item's LDS tiles
    idx = __builtin_amdgcn_readfirstlane(s_item[parity]);
    parity ^= 1;
    if (idx < 0) break;
  }
  if (tid == 0 && p.wq_q) wq_finish(p.wq_q);
}

}  // namespace

hipError_t launch_bwd_bf16(const BwdParams& p, int head_dim, int stage, hipStream_t s) {
  const dim3 block(NT);
  if (stage == 0) {
    const int64_t units = p.total_q * p.num_heads;
    if (units == 0) return hipSuccess;
    const int upb = NT / (head_dim / 8);
    const dim3 grid((unsigned)((units + upb - 1) / upb));
    if (head_dim == 128) hipLaunchKernelGGL(bwd_pre_kernel<128>, grid, block, 0, s, p);
    else hipLaunchKernelGGL(bwd_pre_kernel<64>, grid, block, 0, s, p);
  } else if (stage == 1) {
    if (p.n_kv_items == 0) return hipSuccess;
    const void* kern = head_dim == 128 ? reinterpret_cast<const void*>(bwd_dkdv_kernel<128>)
                                       : reinterpret_cast<const void*>(bwd_dkdv_kernel<64>);
    const int grid = launch_grid(kern, kDkdvThreads, p.n_kv_items, p.wq_kv);
    if (grid < 0) return hipErrorInvalidValue;
    if (head_dim == 128) hipLaunchKernelGGL(bwd_dkdv_kernel<128>, dim3(grid), dim3(kDkdvThreads), 0, s, p);
    else hipLaunchKernelGGL(bwd_dkdv_kernel<64>, dim3(grid), dim3(kDkdvThreads), 0, s, p);
  } else {
    if (p.n_q_items == 0) return hipSuccess;
    const void* kern = head_dim == 128 ? reinterpret_cast<const void*>(bwd_dq_kernel<128>)
                                       : reinterpret_cast<const void*>(bwd_dq_kernel<64>);
    const int grid = launch_grid(kern, kDqThreads, p.n_q_items, p.wq_q);
    if (grid < 0) return hipErrorInvalidValue;
    if (head_dim == 128) hipLaunchKernelGGL(bwd_dq_kernel<128>, dim3(grid), dim3(kDqThreads), 0, s, p);
    else hipLaunchKernelGGL(bwd_dq_kernel<64>, dim3(grid), dim3(kDqThreads), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace zl
