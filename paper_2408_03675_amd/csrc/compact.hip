// Cache update K0, V0 <- K_S, V_S (NaCl Section 3, encoding-phase eviction):
// a row gather.  One thread moves one 16-byte vector: the lanes covering a
// row read it contiguously and write it to a contiguous output row, so both
// sides are coalesced.  K and V rows go to separate blocks (blockIdx.z), and
// with no loop every thread's load is in flight from its first instruction;
// many small blocks keep the whole chip issuing.  Rows are bit copies.

#include "device_common.h"
#include "internal.h"

namespace nacl {

constexpr int kCompactThreads = 512;

__global__ __launch_bounds__(kCompactThreads) void compact_kernel(CompactLaunch a) {
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const int vpr = a.row_vecs;
  const int r = blockIdx.x * (kCompactThreads / vpr) + (int)threadIdx.x / vpr;
  if (r >= a.C) return;
  const int vec = threadIdx.x % vpr;
  const bool is_v = blockIdx.z != 0;
  const int64_t* st = is_v ? a.vs : a.ks;
  const int64_t j = a.keep[(int64_t)bh * a.C + r];
  const u32x4* src = static_cast<const u32x4*>(is_v ? a.v : a.k) + b * st[0] + h * st[1] + j * st[2] + vec;
  u32x4* dst = static_cast<u32x4*>(is_v ? a.v_out : a.k_out) + ((int64_t)bh * a.C + r) * vpr + vec;
  __builtin_nontemporal_store(__builtin_nontemporal_load(src), dst);
}

hipError_t launch_compact(const CompactLaunch& a, hipStream_t stream) {
  if (a.C == 0) return hipSuccess;
  if (a.row_vecs <= 0 || kCompactThreads % a.row_vecs != 0) return hipErrorInvalidValue;
  const int rows_per_block = kCompactThreads / a.row_vecs;
  dim3 grid((a.C + rows_per_block - 1) / rows_per_block, a.B * a.H, 2);
  hipLaunchKernelGGL(compact_kernel, grid, dim3(kCompactThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace nacl
