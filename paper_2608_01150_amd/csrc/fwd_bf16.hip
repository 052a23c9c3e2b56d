// Packed whole+shard attention forward, bf16 inputs, gfx950 MFMA.
//
// A work item is up to 256 query rows of one head against one K/V range (a
// whole segment's own keys, or one CP block of a shard, Sec. IV-D / Tab. II of
// arXiv 2608.01150).  One workgroup (8 waves, two per SIMD) per CU runs items
// one after another, taking them from the launch's work queues (zl_device.h).
// Each wave owns 32 query rows of an item.  Per 64-key step:
//   S^T = K Q^T          MFMA 32x32x16 bf16, K from LDS (A), Q in registers (B)
//   online softmax       per query in the lane's registers (exp2 domain)
//   O^T += V^T P^T       MFMA, V^T from LDS by transpose reads (A), P^T
//                        straight from registers (B)
// Computing the transposed products keeps one query per lane, so the row max
// needs a single cross-lane exchange (lanes l and l^32) and the softmax
// output is already the B operand of the next MFMA.  K and V are staged
// row-major (padded pitch, conflict-free) in 128-key tiles, two LDS buffers
// of each, by direct global-to-LDS loads issued one tile ahead (waves 0-3
// load K, waves 4-7 load V, each fetch's instructions spread over the S
// MFMAs); a tile is two 64-key steps and one barrier.  A staged tile serves
// 256 queries, so the staging costs half as much per MFMA as with 128-row
// items.
//
// Epilogue: WHOLE items write the final bf16 output and the LSE; SHARD items
// write the block-normalised partial (fp32, or bf16 on request) and its LSE
// into their CP slot.

#include "zl_device.h"
#include "zl_internal.h"

namespace zl {
namespace {

constexpr int BN = kFwdTileN;
constexpr int NT = 512;

// Scores are exponentiated against the running maximum as it stands, without
// first taking the new block's maximum.  While the block's scores exceed it by
// at most 64 (log2 units) every P stays within 2^64 and O, l sum it exactly as
// against any other common reference (fp32 keeps its relative precision far
// beyond that).  A block whose exponentials sum (per lane: 16 of a query's
// keys) past 2^64 (+inf included, as for the first block against the initial
// -1e30) takes a slow path: its true maximum, a rescale of O and l to it, and
// its exponentials again.  So the common path needs one compare per block in
// place of a max over its scores.
constexpr float kSumBound = 0x1p64f;

// Epilogue of a forward item: normalises the running output of this lane's
// query and stores it by the item's kind.  o[db][i] is (d = db*32 +
// 16*(i/8) + 8*g + i%8, query qr); m_run is the running maximum (log2
// units), l_part this lane's half of the row sum of the exponentials and
// l_rnd the whole row's sum of the same values rounded to bf16, as they
// entered O += P V.  The output is normalised by the rounded sum, so its
// weights sum to one exactly: the rounding of a dominant P (any value in
// [1, 2^64) against a running maximum that a later key exceeds) cancels
// instead of scaling the output.  The LSE takes the unrounded sum.
template <int D>
__device__ __forceinline__ void fwd_store(const __attribute__((address_space(4))) FwdParams* pp, const Item& it, int qr,
                                          bool q_ok, int g, const f32x16 (&o)[D / 32], float m_run, float l_part,
                                          float l_rnd) {
  const auto& p = *pp;
  const float l = xor32_sum(l_part), lr = l_rnd;
  const float inv = lr > 0.f ? 1.f / lr : 0.f;
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
  } else if (p.step_mode) {
    // Ring step: fold this block (O_b = o * inv, LSE_b = lse) into the
    // running accumulator; the last step writes the final output instead.
    float* acc = p.o_acc + row * D;
    float wa, wb, lse_new;
    step_weights(p.step_first, p.step_first ? 0.f : p.lse_acc[row], lse, wa, wb, lse_new);
    wb *= inv;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c0 = db * 32 + 16 * h + 8 * g;
        f32x4 a = {0.f, 0.f, 0.f, 0.f}, b = {0.f, 0.f, 0.f, 0.f};
        if (!p.step_first) {
          a = *reinterpret_cast<const f32x4*>(acc + c0);
          b = *reinterpret_cast<const f32x4*>(acc + c0 + 4);
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          a[t] = wa * a[t] + wb * o[db][8 * h + t];
          b[t] = wa * b[t] + wb * o[db][8 * h + 4 + t];
        }
        if (p.step_last) {
          u32x4 w = {pack_bf16(a[0], a[1]), pack_bf16(a[2], a[3]), pack_bf16(b[0], b[1]), pack_bf16(b[2], b[3])};
          *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.out) + row * D + c0) = w;
        } else {
          *reinterpret_cast<f32x4*>(acc + c0) = a;
          *reinterpret_cast<f32x4*>(acc + c0 + 4) = b;
        }
      }
    }
    if (g == 0) (p.step_last ? p.lse : p.lse_acc)[row] = lse_new;
  } else if (p.part_bf16) {
    // bf16 partial: this lane's 8 consecutive d values in one 16-byte store
    uint16_t* og = static_cast<uint16_t*>(p.o_part) + it.slot * p.slot_stride + row * D;
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
    if (g == 0) p.lse_part[it.slot * p.lse_slot_stride + row] = lse;
  } else {
    float* og = static_cast<float*>(p.o_part) + it.slot * p.slot_stride + row * D;
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

template <int D>
__global__ __launch_bounds__(NT, 1) void fwd_bf16_kernel(FwdParams p) {
  constexpr int PITCH = Pad<D>::PITCH;
  constexpr int TN = 2 * BN;  // keys per staged tile: two steps per barrier
  constexpr int TILE = TN * PITCH;
  // A staged tile is loaded as two 64-key halves with the same per-lane
  // offsets; per wave DMA_PER_STEP direct-to-LDS instructions per half (four
  // waves share a tile), the next tile's half h issued during step h.
  using Dma = TileDma<D, BN>;
  constexpr int DMA_PER_STEP = Dma::PER_WAVE;
  // Two buffers of each tile as separate objects, so the compiler can tell
  // the direct-to-LDS loads filling one buffer from the reads of another.
  __shared__ __attribute__((aligned(16))) char ks0[TILE], ks1[TILE], vs0[TILE], vs1[TILE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ln = lane & 31, g = lane >> 5;
  // Items come from the launch's work queues (zl_device.h): the workgroup's
  // first-round item, then claimed ones.  Only thread 0 claims; it publishes
  // each item index through s_item (two slots, alternating, so that one
  // barrier per item suffices).  A claim is issued at the start of an item's
  // last tile, so its latency overlaps that tile.
  __shared__ int s_item[2], s_tries;
  if (tid == 0) s_tries = 0;
  int pending = -1;  // thread 0: claim issued ahead
  int parity = 0;
  for (int idx = dispatch_item(blockIdx.x, p.n_items, p.xcd_chunk);;) {
    const Item it = p.items[idx];
    const int64_t rs = (int64_t)p.num_heads * D;  // elements between consecutive tokens
    const uint16_t* qg = static_cast<const uint16_t*>(p.q) + ((int64_t)it.q_start * p.num_heads + it.head) * D;
    const uint16_t* kg = static_cast<const uint16_t*>(p.k) + ((int64_t)it.k_start * p.num_heads + it.head) * D;
    const uint16_t* vg = static_cast<const uint16_t*>(p.v) + ((int64_t)it.k_start * p.num_heads + it.head) * D;

    // Q fragments (B operand): query row wave*32+ln, d = 16*kk + 8*g .. +7.
    const int qr = wave * 32 + ln;
    const bool q_ok = qr < it.q_len;
    u32x4 qf[D / 16];
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
      qf[kk] = q_ok ? *reinterpret_cast<const u32x4*>(qg + qr * rs + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};

    // Wait for the prologue's register loads here, with a waitcnt the compiler
    // sees: the step loop then carries no pending VGPR loads, so it inserts no
    // vmcnt wait there (which would also drain the in-flight tile DMAs).
    __builtin_amdgcn_s_waitcnt(0);

    float m_run = kNegBig, l_part = 0.f;
    // The rounded sum comes from the matrix core: one mfma16 per 16-key P word
    // (the PV B operand, lane l holding 8 keys of query l%32) against a 0/1
    // selector A.  Lane l of A is all ones where bit 4 of l equals bit 2, so
    // output row m sums the lanes of query (column + 16 * ((m/4) % 2)) over
    // both key halves, and every register of lane l ends up holding the full
    // rounded sum of query l%32.
    f32x4 racc = f32x4{0.f, 0.f, 0.f, 0.f};
    const uint32_t selw = ((lane >> 4) & 1) == ((lane >> 2) & 1) ? 0x3F803F80u : 0u;
    const u32x4 rsel = {selw, selw, selw, selw};
    f32x16 o[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) o[db] = f32x16{};

    // Per-lane LDS offsets: A-operand row perm32(ln), transpose piece.
    const uint32_t a_off = poff<D>(perm32(ln), g * 8);
    const uint32_t t_off = tr_lane_off<D>(lane);

    // K/V tile starting at key kt; rows past the range (and whole tiles past
    // it, fetched by the lookahead) read zero and are masked below.  Waves 0-3
    // load the K tile, waves 4-7 the V tile; the choice is wave-uniform.
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
    // Inside the loop a fetch is only set up here; the S MFMAs of the tile's
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

    // One 64-key step as two 32-key blocks kb, each its own online-softmax
    // update (exponentials against the running maximum, the sum check and, in
    // rare cases, the slow path of kSumBound), software-pipelined inside the
    // wave so that the softmax VALU work runs under MFMAs:
    //   S of kb 0;  S of kb 1 with the softmax of kb 0;  check of kb 0;
    //   PV of kb 0 with the exponentials of kb 1;  check of kb 1;  PV of kb 1.
    // A operands come from LDS through rings of loads issued ahead of use.
    // half: which of the tile's two steps (0 or 1, a literal at the call sites).
    auto step = [&](const char* kbuf, const char* vbuf, int kt, int half) __attribute__((always_inline)) {
      const char* ka = kbuf + a_off;
      const char* vt = vbuf + t_off;
      constexpr int NS = 2 * (D / 16);        // S MFMAs per step
      constexpr int NP = 2 * (D / 32) * 2;    // PV MFMAs per step
      constexpr int PF = 6, PFC = 3;
      constexpr int DMA_GAP = NS / DMA_PER_STEP;  // S MFMAs between the spread fetch's instructions
      static_assert(DMA_GAP >= 2 && (DMA_PER_STEP - 1) * DMA_GAP + 1 < NS, "spread fetch must fit the S MFMAs");
      // S operand j: keys of block j/(NS/2) (rows perm32), d chunk j%(NS/2).
      auto a_op = [&](int j) {
        return *reinterpret_cast<const u32x4*>(ka + poff<D>((j / (NS / 2)) * 32, (j % (NS / 2)) * 16));
      };
      // PV operand m: key block m/(NP/2), d block (m%(NP/2))/2, 16-key half m%2.
      auto c_op = [&](int m) {
        return tr_operand<D>(vt, (m / (NP / 2)) * 32 + 16 * (m & 1), ((m % (NP / 2)) >> 1) * 32);
      };
      const int nvalid = it.k_len - kt;
      // s[kb][i] is the raw score of (key kb*32 + 16*(i/8) + 8*g + i%8, query qr).
      f32x16 s[2];
      u32x4 pb[2][2];
      // Each block's sum in two partial accumulators (words of even and
      // odd c), which halves their dependency chains.
      float lsum[2][2] = {};
      // Keys past the range on a partial tile: score -inf, exact at any positive scale.
      auto mask = [&](int kb) {
        if (nvalid < BN) {
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = kb * 32 + 16 * (i >> 3) + 8 * g + (i & 7);
            if (key >= nvalid) s[kb][i] = -INFINITY;
          }
        }
      };
      // Exponentials of elements 2c, 2c+1 of block kb: one packed P word.
      auto expo = [&](int kb, int c) {
        const float e0 = fast_exp2(fmaf(s[kb][2 * c], p.scale_log2, -m_run));
        const float e1 = fast_exp2(fmaf(s[kb][2 * c + 1], p.scale_log2, -m_run));
        lsum[kb][c & 1] += e0 + e1;
        pb[kb][c >> 2][c & 3] = pack_bf16(e0, e1);
      };
      // The slow path of block kb (see kSumBound): when it is taken for block 1,
      // block 0 has entered O already, and the rescale covers it there.
      auto block_fix = [&](int kb) {
        float mt = s[kb][0];
#pragma unroll
        for (int i = 1; i < 16; ++i) mt = fmaxf(mt, s[kb][i]);
        mt = xor32_max(mt) * p.scale_log2;
        const float m_new = fmaxf(m_run, mt);
        const float alpha = fast_exp2(m_run - m_new);
        m_run = m_new;
        l_part *= alpha;
        racc *= alpha;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
#pragma unroll
          for (int i = 0; i < 16; ++i) o[db][i] *= alpha;
        }
        lsum[kb][0] = lsum[kb][1] = 0.f;
#pragma unroll
        for (int c = 0; c < 8; ++c) expo(kb, c);
      };
      auto block_done = [&](int kb) {
        if (__any(lsum[kb][0] + lsum[kb][1] > kSumBound)) block_fix(kb);
        l_part += lsum[kb][0] + lsum[kb][1];
      };

      u32x4 ring[PF];
#pragma unroll
      for (int j = 0; j < PF; ++j) ring[j] = a_op(j);
      s[0] = s[1] = f32x16{};
      __builtin_amdgcn_sched_barrier(0);
      // Raised issue priority while this wave's MFMA loops run: when the SIMD's
      // two waves drift apart, the one with MFMAs ready issues first and keeps
      // the matrix core fed.
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int j = 0; j < NS; ++j) {
        const u32x4 a = ring[j % PF];
        if (j + PF < NS) ring[j % PF] = a_op(j + PF);
        const int kb = j / (NS / 2);
        s[kb] = mfma32(a, qf[j % (NS / 2)], s[kb]);
        if (j % DMA_GAP == 1 && j / DMA_GAP < DMA_PER_STEP) dma.issue_one(next_rsrc[half], next_lds[half], j / DMA_GAP);
        // Block 1's MFMAs carry block 0's softmax: the mask of a partial tile
        // first, then the eight exponential pairs spread over the remaining
        // slots.  Each packed word and the block's sum are pinned where they are
        // computed: block 1's mask is a branch, and without the pin the compiler
        // sinks this work past it, next to its first use, out of the MFMAs.
        if (j == NS / 2) mask(0);
        if (j > NS / 2) {
          constexpr int SLOTS = NS / 2 - 1;
          const int c0 = (j - NS / 2 - 1) * 8 / SLOTS, c1 = (j - NS / 2) * 8 / SLOTS;
#pragma unroll
          for (int c = c0; c < c1; ++c) {
            expo(0, c);
            asm volatile("" : "+v"(pb[0][c >> 2][c & 3]), "+v"(lsum[0][c & 1]));
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      u32x4 cring[PFC];
#pragma unroll
      for (int m = 0; m < PFC; ++m) cring[m] = c_op(m);
      block_done(0);
      mask(1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int m = 0; m < NP; ++m) {
        const u32x4 a = cring[m % PFC];
        if (m + PFC < NP) cring[m % PFC] = c_op(m + PFC);
        // Block 0's PV MFMAs carry block 1's exponentials; block 1's sum is
        // checked before its own PV MFMAs.
        // Each packed word is pinned here too: otherwise the compiler sinks the
        // conversions past the sum check, in front of block 1's first PV MFMA.
        if (m < NP / 2) {
#pragma unroll
          for (int c = m * 8 / (NP / 2); c < (m + 1) * 8 / (NP / 2); ++c) {
            expo(1, c);
            asm volatile("" : "+v"(pb[1][c >> 2][c & 3]), "+v"(lsum[1][c & 1]));
          }
        }
        if (m == NP / 2) block_done(1);
        const int kb = m / (NP / 2), db = (m % (NP / 2)) >> 1, s2 = m & 1;
        o[db] = mfma32(a, pb[kb][s2], o[db]);
        // The rounded sum of each P word, after its block's sum check.
        if ((m % (NP / 2)) % (NP / 4) == 1) racc = mfma16(rsel, pb[kb][(m % (NP / 2)) / (NP / 4)], racc);
        __builtin_amdgcn_sched_barrier(0);
      }
      __builtin_amdgcn_s_setprio(0);
    };

    // A wave with no query rows in this item (the ragged last tile of a
    // segment) skips the math and only issues its share of the next tile's
    // loads, which the other waves need; the SIMD's other wave then has the
    // matrix core to itself.
    const bool wave_live = wave * 32 < it.q_len;
    auto run = [&](const char* kbuf, const char* vbuf, int kt, int half) __attribute__((always_inline)) {
      if (wave_live) {
        step(kbuf, vbuf, kt, half);
      } else {
#pragma unroll
        for (int jj = 0; jj < DMA_PER_STEP; ++jj) dma.issue_one(next_rsrc[half], next_lds[half], jj);
      }
    };
    // One staged tile of TN keys as two steps, with no barrier between them;
    // a tile whose second half lies past the range runs only its first step
    // (the loop ends there, so the fetch that step would finish is not needed).
    auto tile = [&](const char* kbuf, const char* vbuf, int kt) __attribute__((always_inline)) {
      run(kbuf, vbuf, kt, 0);
      if (kt + BN < it.k_len) run(kbuf + BN * PITCH, vbuf + BN * PITCH, kt + BN, 1);
    };

    auto claim_ahead = [&]() __attribute__((always_inline)) {
      if (tid == 0 && p.wq && s_tries < 8) pending = wq_claim(p.wq, s_tries);
    };

    // Two buffer sets in rotation, the loop unrolled by two.  Tile t+1 is
    // fetched during tile t, after the barrier that retires tile t-1's buffers;
    // a fetch past the range reads zero (an empty resource) and is never used.
    // Before the barrier a wave waits for all of its loads: only tile t+1's
    // are outstanding.  Two 64-key steps per barrier halve the barriers of a
    // 64-key tile rotation at the same prefetch distance in time.
    if (it.k_len > 0) {
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
      wait_vmem();  // the lookahead loads must land before the workgroup's LDS is released
    }

    fwd_store<D>(kernargs<FwdParams>(), it, qr, q_ok, g, o, m_run, l_part, racc[0]);
    const auto* pk = kernargs<FwdParams>();
    if (tid == 0) s_item[parity] = pk->wq ? wq_next(pk->wq, pk->n_items, pk->xcd_chunk, &s_tries, pending) : -1;
    pending = -1;
    __syncthreads();  // also: every wave is done with this item's LDS tiles
    idx = __builtin_amdgcn_readfirstlane(s_item[parity]);
    parity ^= 1;
    if (idx < 0) break;
  }
  if (tid == 0 && p.wq) wq_finish(p.wq);
}

}  // namespace

hipError_t launch_fwd_bf16(const FwdParams& p, int head_dim, hipStream_t s) {
  const void* kern = head_dim == 128 ? reinterpret_cast<const void*>(fwd_bf16_kernel<128>)
                                     : reinterpret_cast<const void*>(fwd_bf16_kernel<64>);
  const int grid = launch_grid(kern, NT, p.n_items, p.wq);
  if (grid < 0) return hipErrorInvalidValue;
  if (head_dim == 128)
    hipLaunchKernelGGL(fwd_bf16_kernel<128>, dim3(grid), dim3(NT), 0, s, p);
  else
    hipLaunchKernelGGL(fwd_bf16_kernel<64>, dim3(grid), dim3(NT), 0, s, p);
  return hipGetLastError();
}

}  // namespace zl
