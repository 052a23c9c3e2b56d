// Device-side helpers shared by the gfx950 kernels: vector types, the bf16
// MFMA wrapper, bf16 packing and the LDS swizzles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "zl_internal.h"

namespace zl {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// D(32x32 fp32) += A(32x16 bf16) * B(16x32 bf16).
// Lane l supplies row l%32 of A and column l%32 of B, each as the 8 values of
// k-group l/32.  D register i of lane l is element (row 8*(i/4) + 4*(l/32) +
// i%4, column l%32).
__device__ __forceinline__ f32x16 mfma32(const u32x4& a, const u32x4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

// D(16x16 fp32) += A(16x32 bf16) * B(32x16 bf16), half the cycles of mfma32.
// Lane l supplies row l%16 of A and column l%16 of B, each as the 8 values of
// k-group l/16; D register i of lane l is element (row 4*(l/16) + i, column
// l%16).
__device__ __forceinline__ f32x4 mfma16(const u32x4& a, const u32x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Round-to-nearest-even fp32 -> bf16 of two values, packed lo | hi << 16
// (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Row permutation of a 32-row MFMA operand tile.  Loading A-operand row m
// with tile row perm32(m) makes D register i of lane l hold tile row
// 16*(i/8) + 8*(l/32) + i%8: each lane's registers 0-7 and 8-15 cover two runs
// of 8 consecutive rows, so a D fragment is directly the (lane-major) B
// operand of the next MFMA over those rows, and epilogue stores are 8-wide.
__device__ __forceinline__ int perm32(int m) {
  const int blk4 = m >> 3, g = (m >> 2) & 1, lo = m & 3;
  return ((blk4 >> 1) << 4) + (g << 3) + ((blk4 & 1) << 2) + lo;
}

// Row-major bf16 LDS tile with a padded row pitch: 304 bytes for D = 128
// (256 + 48), 144 for D = 64.  With 64 four-byte banks and 16 lanes served
// per cycle, both MFMA operand access patterns are conflict-free:
//  * A-operand 16-byte reads, where 16 lanes read one 16-byte chunk from the
//    16 rows perm32 gives them, and
//  * transpose reads, where 16 lanes read 4 consecutive rows x 32 bytes.
// Every address is a per-lane base plus a compile-time offset, so the loops
// do no address arithmetic.
template <int D>
struct Pad {
  static constexpr int PITCH = D == 128 ? 304 : 144;
};
template <int D>
__device__ __forceinline__ constexpr uint32_t poff(int row, int col) {
  return row * Pad<D>::PITCH + col * 2;
}

// 32-bit LDS byte address of a pointer into a __shared__ object.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(size_t)((const __attribute__((address_space(3))) char*)p);
}

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer resource (stride 0, no swizzle) over `bytes` bytes at `base`.
// A buffer load at a byte offset at or past `bytes` reads zero: the hardware
// range check replaces per-lane clamping of addresses.
__device__ __forceinline__ i32x4 buf_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)base;
  return i32x4{(int)(uint32_t)a, (int)((a >> 32) & 0xFFFFu), (int)bytes, 0x00020000};
}

// One direct buffer->LDS load per lane (buffer_load_dwordx4 ... lds): lane l's
// 16 bytes, read at byte offset voff of the resource, land at the
// wave-uniform LDS address `lds` + 16*l.  Issued as inline asm (M0 saved and
// restored around it) so that the compiler does not treat it as an LDS store
// that every later LDS read must wait for; callers wait for vmcnt themselves
// before the barrier that publishes the data.  The s_nop is the one wait
// state an LDS DMA needs after an SALU write of M0.
__device__ __forceinline__ void dma16(const i32x4& rsrc, uint32_t voff, uint32_t lds) {
  uint32_t save;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds\n\ts_mov_b32 m0, %0"
               : "=&s"(save)
               : "v"(voff), "s"(rsrc), "s"(lds)
               : "memory");
}

// Same for 4 bytes per lane (buffer_load_dword ... lds): lane l lands at lds + 4*l.
__device__ __forceinline__ void dma4(const i32x4& rsrc, uint32_t voff, uint32_t lds) {
  uint32_t save;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds\n\ts_mov_b32 m0, %0"
               : "=&s"(save)
               : "v"(voff), "s"(rsrc), "s"(lds)
               : "memory");
}

// Staging of a [ROWS][D] bf16 tile of one head of a packed [T, H, D] tensor
// (consecutive rows `row_bytes` apart in memory) into a padded LDS tile with
// direct 16-byte loads.  The tile is NJ = ROWS * PITCH / 1024 whole wave
// instructions; NW waves share them, each issuing PER_WAVE, the surplus ones
// clamped onto the last block (rewriting identical bytes), so there is no
// branch.  Padding slots reload chunk 0 of their row.  A lane's byte offsets
// do not depend on the tile's position, so they are computed once; per tile
// only the (scalar) buffer resource changes, and rows at or past the range
// end read as zero through its range check.
template <int D, int ROWS, int NW = 4>
struct TileDma {
  static constexpr int SPR = Pad<D>::PITCH / 16;
  static constexpr int NJ = ROWS * SPR / 64;
  static constexpr int PER_WAVE = (NJ + NW - 1) / NW;
  static_assert(ROWS * SPR % 64 == 0, "tile must be whole wave instructions");
  uint32_t voff[PER_WAVE];
  int wave;  // wave-uniform index in [0, NW)

  __device__ __forceinline__ void init(int wave_, int lane, uint32_t row_bytes) {
    wave = wave_;
#pragma unroll
    for (int jj = 0; jj < PER_WAVE; ++jj) {
      const int j = min(wave + NW * jj, NJ - 1);
      const int slot = j * 64 + lane;
      const int row = slot / SPR, chunk = slot % SPR;
      voff[jj] = (uint32_t)row * row_bytes + (uint32_t)(chunk < D / 8 ? chunk : 0) * 16u;
    }
  }

  // The resource of rows [0, ROWS) starting at g_row0; rows at or past
  // nvalid read zero.
  __device__ __forceinline__ static i32x4 resource(const void* g_row0, int nvalid, uint32_t row_bytes) {
    const int nv = min(nvalid, ROWS);
    const uint32_t bytes = nv > 0 ? (uint32_t)(nv - 1) * row_bytes + D * 2 : 0u;
    return buf_rsrc(g_row0, bytes);
  }

  // This wave's instruction jj (of PER_WAVE) of a fetch into the tile at LDS
  // address tile_lds.  Issuing a fetch's instructions one at a time between
  // MFMAs keeps a wave from stalling at issue behind its own burst of DMAs.
  __device__ __forceinline__ void issue_one(const i32x4& rsrc, uint32_t tile_lds, int jj) const {
    const int j = min(wave + NW * jj, NJ - 1);
    dma16(rsrc, voff[jj], __builtin_amdgcn_readfirstlane(tile_lds + j * 1024));
  }

  // The whole fetch at once.
  __device__ __forceinline__ void issue(char* tile, const void* g_row0, int nvalid, uint32_t row_bytes) const {
    const i32x4 rsrc = resource(g_row0, nvalid, row_bytes);
#pragma unroll
    for (int jj = 0; jj < PER_WAVE; ++jj) issue_one(rsrc, lds_addr(tile), jj);
  }
};

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Wait until at most N of this wave's vector memory loads are outstanding.
// Loads complete in issue order, so this retires everything but the N most
// recent (a tile fetched ahead of the one about to be used).
template <int N>
__device__ __forceinline__ void wait_vmem_keep() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

typedef short s16x4 __attribute__((ext_vector_type(4)));

// LDS transpose read (ds_read_b64_tr_b16).  Within each group of 16 lanes,
// lane i receives in slot t the 16-bit element (i % 4) of the 8 bytes that
// lane 4*t + i/4 addresses.
__device__ __forceinline__ u32x2 lds_read_tr16(const void* p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p);
  return __builtin_bit_cast(u32x2, v);
}

// Per-lane byte offset for tr_operand on a padded [k][D] tile.  A lane's
// transpose-read piece is row 8*g + i/4 and 4 columns starting at
// perm32(16*(i/16 % 2) + 4*(i%4)), with i the lane's index within its
// 16-lane group.
template <int D>
__device__ __forceinline__ uint32_t tr_lane_off(int lane) {
  const int grp = lane >> 4, i = lane & 15;
  return poff<D>(8 * (lane >> 5) + (i >> 2), perm32(16 * (grp & 1) + 4 * (i & 3)));
}

// MFMA operand whose 8 k-values run down a column of a row-major [k][D] LDS
// tile: lane l (m = l%32, g = l/32) receives rows k0 + 8g .. k0 + 8g + 7 of
// column col_base + perm32(m).  `lane_ptr` is the tile base plus
// tr_lane_off(lane); k0 and col_base are compile-time after unrolling.  Two
// transpose reads, each lane addressing one 8-byte piece of a 4-row x
// 16-column block.
template <int D>
__device__ __forceinline__ u32x4 tr_operand(const char* lane_ptr, int k0, int col_base) {
  const u32x2 lo = lds_read_tr16(lane_ptr + poff<D>(k0, col_base));
  const u32x2 hi = lds_read_tr16(lane_ptr + poff<D>(k0 + 4, col_base));
  return u32x4{lo[0], lo[1], hi[0], hi[1]};
}

// One online merge step of ring attention: with the running statistic
// lse_acc (unless `first`) and a new block's lse_b, the merged output is
// a * o_acc + b * O_b and the merged statistic `lse` (natural log).  Both
// -inf (no key seen yet) gives a = b = 0 and lse = -inf.
__device__ __forceinline__ void step_weights(bool first, float lse_acc, float lse_b, float& a, float& b, float& lse) {
  if (first) {
    a = 0.f;
    b = 1.f;
    lse = lse_b;
    return;
  }
  const float m = fmaxf(lse_acc, lse_b);
  if (m == -INFINITY) {
    a = b = 0.f;
    lse = -INFINITY;
    return;
  }
  const float wa = expf(lse_acc - m), wb = expf(lse_b - m), den = wa + wb;
  a = wa / den;
  b = wb / den;
  lse = m + logf(den);
}

// Max / sum of a value over lanes l and l^32 with v_permlane32_swap (a VALU
// exchange of the two 32-lane halves, no LDS round trip).  With both operands
// equal, the swap returns the lower half's values in every lane of the first
// result and the upper half's in the second.
__device__ __forceinline__ float xor32_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ----------------------------------------------------------- work queues
// Dynamic distribution of a launch's work items over resident workgroups.
// The work table in dispatch order (dispatch_item) is split into 8 queues:
// queue y holds the dispatch positions y, y+8, y+16, ..., which the hardware's
// round-robin placement of workgroups would send to XCD y.  Workgroup b
// (grid G <= n) first runs position b, i.e. the first round of a
// one-item-per-workgroup launch; afterwards it claims further positions of
// its own XCD's queue with a device-scope atomic counter, and once that queue
// is empty those of the other XCDs' queues in turn.  The XCDs of one GPU run
// at different speeds (several percent apart under load), and a fixed share
// of the items per XCD leaves the fast ones idle while the slowest finishes;
// here an XCD that runs ahead takes over the tail of the others' queues.
// ctr[y] counts the claims on queue y beyond its first round and ctr[8] the
// workgroups that have finished; the last one to finish resets all nine, so
// the next launch that uses the same counters finds them at zero.

__device__ __forceinline__ int xcd_id() {
  uint32_t r;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(r));
  return (int)(r & 7u);
}

// Claim of the next position of the queue this workgroup is working on
// (queue (xcd + tries) % 8), issued ahead of need so that its latency
// overlaps work; its result goes to wq_next as `pending`.
__device__ __forceinline__ int wq_claim(int* ctr, int tries) { return atomicAdd(&ctr[(xcd_id() + tries) & 7], 1); }

// Work-table index of this workgroup's next item, or -1 when every queue is
// empty.  *tries (workgroup state, in LDS) counts the queues found empty;
// pending is a claim from wq_claim on the current queue, or -1.
__device__ __forceinline__ int wq_next(int* ctr, int n, int chunk, int* tries, int pending) {
  int t = *tries;
  const int grid = (int)gridDim.x;
  while (t < 8) {
    const int y = (xcd_id() + t) & 7;
    const int len = (n - y + 7) >> 3;      // positions y + 8k below n
    const int first = (grid - y + 7) >> 3;  // of those, taken by the first round
    const int k = first + (pending >= 0 ? pending : atomicAdd(&ctr[y], 1));
    pending = -1;
    if (k < len) {
      *tries = t;
      return dispatch_item(8 * k + y, n, chunk);
    }
    ++t;
  }
  *tries = t;
  return -1;
}

// Called once per workgroup after its last item.
__device__ __forceinline__ void wq_finish(int* ctr) {
  if ((unsigned)atomicAdd(&ctr[8], 1) == gridDim.x - 1u) {
#pragma unroll
    for (int y = 0; y < 9; ++y) atomicExch(&ctr[y], 0);
  }
}

// The launch's parameters read afresh from the kernel-argument segment, by
// scalar loads at the point of use.  A persistent kernel would otherwise hold
// arguments that only an item's epilogue needs in registers across its whole
// item loop.
template <class P>
__device__ __forceinline__ const __attribute__((address_space(4))) P* kernargs() {
  auto* k = (const __attribute__((address_space(4))) P*)__builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(k));
  return k;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

constexpr float kNegBig = -1.0e30f;    // finite "minus infinity" for masked scores
constexpr float kLn2 = 0.69314718055994531f;

}  // namespace zl
