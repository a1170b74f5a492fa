// Cache update K0, V0 <- K_S, V_S (NaCl Section 3, encoding-phase eviction):
// a row gather.  Each thread moves 16-byte vectors; the lanes covering one
// row read it contiguously and the output rows are written contiguously, so
// both sides are coalesced.  Rows are bit copies.

#include "device_common.h"
#include "internal.h"

namespace nacl {

constexpr int kCompactThreads = 256;
constexpr int kCompactRowsPerBlock = 64;

__global__ __launch_bounds__(kCompactThreads) void compact_kernel(CompactLaunch a) {
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const int vpr = a.row_vecs;
  const int rows_per_pass = kCompactThreads / vpr;
  const int vec = threadIdx.x % vpr;
  const int r_begin = blockIdx.x * kCompactRowsPerBlock;
  const int r_end = min(r_begin + kCompactRowsPerBlock, a.C);
  const u32x4* k = static_cast<const u32x4*>(a.k) + b * a.ks[0] + h * a.ks[1] + vec;
  const u32x4* v = static_cast<const u32x4*>(a.v) + b * a.vs[0] + h * a.vs[1] + vec;
  const int32_t* keep = a.keep + (int64_t)bh * a.C;
  u32x4* ko = static_cast<u32x4*>(a.k_out) + (int64_t)bh * a.C * vpr + vec;
  u32x4* vo = static_cast<u32x4*>(a.v_out) + (int64_t)bh * a.C * vpr + vec;
#pragma unroll 4
  for (int r = r_begin + (int)threadIdx.x / vpr; r < r_end; r += rows_per_pass) {
    const int64_t j = keep[r];
    const u32x4 kv = __builtin_nontemporal_load(k + j * a.ks[2]);
    const u32x4 vv = __builtin_nontemporal_load(v + j * a.vs[2]);
    __builtin_nontemporal_store(kv, ko + (int64_t)r * vpr);
    __builtin_nontemporal_store(vv, vo + (int64_t)r * vpr);
  }
}

hipError_t launch_compact(const CompactLaunch& a, hipStream_t stream) {
  if (a.C == 0) return hipSuccess;
  dim3 grid((a.C + kCompactRowsPerBlock - 1) / kCompactRowsPerBlock, a.B * a.H);
  hipLaunchKernelGGL(compact_kernel, grid, dim3(kCompactThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace nacl
