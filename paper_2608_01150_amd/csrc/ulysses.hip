// Local staging of the Ulysses (1,h,1) primitive (Sec. II-B; Tab. II; the
// coalesced QKV-packed all-to-all of Sec. IV-D): layout kernels that surround
// one block-diagonal attention call on a head subset.  Every kernel moves
// 16-byte chunks of a head's d-vector, with the destination written in order
// (coalesced); they are HBM-bound and do no arithmetic.
//
// Layouts (Hl = H / group heads per rank, rows in sequence order):
//   local   q, k, v, out_local   [T_local, H, d]
//   qkv send (to rank j)         [group][T_local][Hl][3][d]   (q, k, v of head j*Hl+hh)
//   qkv recv (from rank j)       rank-major: rank j's T_j rows, [T_j][Hl][3][d]
//   full    q, k, v, out         [T_full, Hl, d]  (whole sequences, block-diagonal attention)
//   out send / recv              rank-major rows like qkv recv, [T_j][Hl][d]
// row_map[r] (r over the rank-major rows) is the full row of rank-major row r.

#include "zl_device.h"
#include "zl_internal.h"

namespace zl {
namespace {

constexpr int NT = 256;

template <int D>
__global__ __launch_bounds__(NT) void pack_qkv_kernel(UlyssesParams p) {
  constexpr int C = D / 8;  // 16-byte chunks per head vector
  const int64_t u = (int64_t)blockIdx.x * NT + threadIdx.x;
  const int64_t n = (int64_t)p.group * p.rows * p.heads_local * 3 * C;
  if (u >= n) return;
  const int c = (int)(u % C);
  int64_t r = u / C;
  const int which = (int)(r % 3);
  r /= 3;
  const int hh = (int)(r % p.heads_local);
  r /= p.heads_local;
  const int64_t t = r % p.rows;
  const int j = (int)(r / p.rows);
  const uint16_t* src = static_cast<const uint16_t*>(which == 0 ? p.a : which == 1 ? p.b : p.c) +
                        (t * p.heads + (int64_t)j * p.heads_local + hh) * D + c * 8;
  *(reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.dst)) + u) = *reinterpret_cast<const u32x4*>(src);
}

template <int D>
__global__ __launch_bounds__(NT) void unpack_qkv_kernel(UlyssesParams p) {
  constexpr int C = D / 8;
  // one thread per (full-layout destination chunk), reading the rank-major source
  const int64_t u = (int64_t)blockIdx.x * NT + threadIdx.x;
  const int64_t n = (int64_t)p.rows * p.heads_local * 3 * C;
  if (u >= n) return;
  const int c = (int)(u % C);
  int64_t r = u / C;
  const int which = (int)(r % 3);
  r /= 3;
  const int hh = (int)(r % p.heads_local);
  const int64_t row = r / p.heads_local;  // rank-major row
  const int64_t full = p.row_map[row];
  const u32x4 v = *(reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p.a)) + u);
  uint16_t* dst = static_cast<uint16_t*>(which == 0 ? p.dst : which == 1 ? p.dst2 : p.dst3);
  *reinterpret_cast<u32x4*>(dst + (full * p.heads_local + hh) * D + c * 8) = v;
}

template <int D>
__global__ __launch_bounds__(NT) void pack_out_kernel(UlyssesParams p) {
  constexpr int C = D / 8;
  const int64_t u = (int64_t)blockIdx.x * NT + threadIdx.x;
  const int64_t n = (int64_t)p.rows * p.heads_local * C;
  if (u >= n) return;
  const int c = (int)(u % C);
  int64_t r = u / C;
  const int hh = (int)(r % p.heads_local);
  const int64_t row = r / p.heads_local;
  const int64_t full = p.row_map[row];
  const uint16_t* src = static_cast<const uint16_t*>(p.a) + (full * p.heads_local + hh) * D + c * 8;
  *(reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.dst)) + u) = *reinterpret_cast<const u32x4*>(src);
}

template <int D>
__global__ __launch_bounds__(NT) void unpack_out_kernel(UlyssesParams p) {
  constexpr int C = D / 8;
  const int64_t u = (int64_t)blockIdx.x * NT + threadIdx.x;
  const int64_t n = (int64_t)p.rows * p.heads * C;
  if (u >= n) return;
  const int c = (int)(u % C);
  int64_t r = u / C;
  const int hd = (int)(r % p.heads);
  const int64_t t = r / p.heads;
  const int j = hd / p.heads_local, hh = hd % p.heads_local;
  const uint16_t* src = static_cast<const uint16_t*>(p.a) + (((int64_t)j * p.rows + t) * p.heads_local + hh) * D + c * 8;
  *(reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.dst)) + u) = *reinterpret_cast<const u32x4*>(src);
}

}  // namespace

hipError_t launch_ulysses(const UlyssesParams& p, int op, int head_dim, hipStream_t s) {
  int64_t units = 0;
  const int64_t c = head_dim / 8;
  switch (op) {
    case 0: units = (int64_t)p.group * p.rows * p.heads_local * 3 * c; break;
    case 1: units = (int64_t)p.rows * p.heads_local * 3 * c; break;
    case 2: units = (int64_t)p.rows * p.heads_local * c; break;
    default: units = (int64_t)p.rows * p.heads * c; break;
  }
  if (units == 0) return hipSuccess;
  const dim3 grid((unsigned)((units + NT - 1) / NT)), block(NT);
#define ZL_LAUNCH(KERN)                                                   \
  if (head_dim == 128) hipLaunchKernelGGL(KERN<128>, grid, block, 0, s, p); \
  else hipLaunchKernelGGL(KERN<64>, grid, block, 0, s, p);
  switch (op) {
    case 0: ZL_LAUNCH(pack_qkv_kernel); break;
    case 1: ZL_LAUNCH(unpack_qkv_kernel); break;
    case 2: ZL_LAUNCH(pack_out_kernel); break;
    default: ZL_LAUNCH(unpack_out_kernel); break;
  }
#undef ZL_LAUNCH
  return hipGetLastError();
}

}  // namespace zl
