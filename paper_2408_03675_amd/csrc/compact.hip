// Cache update K0, V0 <- K_S, V_S (NaCl Section 3, encoding-phase eviction):
// a row gather.  One thread moves one 16-byte vector: the lanes covering a
// row read it contiguously and write it to a contiguous output row, so both
// sides are coalesced.  K and V rows go to separate blocks (blockIdx.z), and
// with no loop every thread's load is in flight from its first instruction;
// many small blocks keep the whole chip issuing.  Rows are bit copies.
//
// Also here: the in-place form of the same update for a decode-time cache
// (Section 3, generation-phase eviction: the kept rows move to the front of
// each head's own rows), and the append of new decode steps' rows to the
// cache (Algorithm 1, generation phase).

#include "device_common.h"
#include "internal.h"

namespace nacl {

constexpr int kCompactThreads = 512;

// A keep index outside [0, L) gives a zero row and sets bit 2 of the health
// words (when the launch has them) instead of reading outside the head.
__device__ __forceinline__ void flag_bad_index(uint32_t* health) {
  if (health) {
    atomicOr(health, 4u);
    atomicOr(health + 1, 4u);
  }
}

// VPR: 16-byte vectors per row (D * element size / 16), a compile-time
// constant so the row and vector of a thread are shifts, not divisions.
template <int VPR>
__global__ __launch_bounds__(kCompactThreads) void compact_kernel(CompactLaunch a) {
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  constexpr int vpr = VPR;
  const int r = blockIdx.x * (kCompactThreads / vpr) + (int)threadIdx.x / vpr;
  if (r >= a.C) return;
  const int vec = threadIdx.x % vpr;
  const bool is_v = blockIdx.z != 0;
  const int64_t* st = is_v ? a.vs : a.ks;
  const int j = a.keep[(int64_t)bh * a.C + r];
  // The load is unconditional (an out-of-range index reads row 0 of the
  // head) so it issues as soon as the index arrives; its value is replaced
  // by zeros afterwards.
  const bool ok = (unsigned)j < (unsigned)a.L;
  const u32x4* src = static_cast<const u32x4*>(is_v ? a.v : a.k) + b * st[0] + h * st[1] +
                     (int64_t)(ok ? j : 0) * st[2] + vec;
  u32x4 x = __builtin_nontemporal_load(src);
  if (!ok) {
    x = u32x4{0u, 0u, 0u, 0u};
    if (vec == 0) flag_bad_index(a.health);
  }
  u32x4* dst = static_cast<u32x4*>(is_v ? a.v_out : a.k_out) + ((int64_t)bh * a.C + r) * vpr + vec;
  __builtin_nontemporal_store(x, dst);
}

// In place: row c of each head takes row keep[c] of the same head, in the
// input's own layout.  keep is strictly ascending, so keep[c] >= c and the
// rows a chunk of destinations [c0, c1) reads lie at or after c0: rows that
// no earlier chunk writes.  One work-group per (head, K or V) walks the
// chunks in order; inside a chunk every source is read (the barrier waits
// for the loads) before any destination is written, since a source of one
// row may be the destination of another row of the same chunk.  Rows with
// keep[c] == c stay where they are.
constexpr int kInplaceThreads = 1024;
constexpr int kInplaceVecs = 16;  // vectors per thread and chunk (all loads in flight at once)

template <int VPR>
__global__ __launch_bounds__(kInplaceThreads) void compact_inplace_kernel(CompactLaunch a) {
  const int bh = blockIdx.x, b = bh / a.H, h = bh % a.H;
  const bool is_v = blockIdx.y != 0;
  const int64_t* st = is_v ? a.vs : a.ks;
  u32x4* base = static_cast<u32x4*>(is_v ? a.v_out : a.k_out) + b * st[0] + h * st[1];
  constexpr int vpr = VPR;
  const int rows_per_chunk = kInplaceThreads * kInplaceVecs / vpr;
  const int32_t* keep = a.keep + (int64_t)bh * a.C;
  for (int c0 = 0; c0 < a.C; c0 += rows_per_chunk) {
    u32x4 x[kInplaceVecs];
    int dst[kInplaceVecs];
#pragma unroll
    for (int u = 0; u < kInplaceVecs; ++u) {
      const int idx = u * kInplaceThreads + (int)threadIdx.x;
      const int r = c0 + idx / vpr, vec = idx % vpr;
      dst[u] = -1;
      x[u] = u32x4{0u, 0u, 0u, 0u};
      if (r < a.C) {
        const int j = keep[r];
        if ((unsigned)j >= (unsigned)a.L) {
          dst[u] = r;  // zero row
          if (vec == 0) flag_bad_index(a.health);
        } else if (j != r) {
          x[u] = base[(int64_t)j * st[2] + vec];
          dst[u] = r;
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kInplaceVecs; ++u) {
      const int idx = u * kInplaceThreads + (int)threadIdx.x;
      if (dst[u] >= 0) base[(int64_t)dst[u] * st[2] + idx % vpr] = x[u];
    }
  }
}

// Slot form of the in-place update (generation-phase eviction with a cache
// whose rows need not stay in token order): with S the ascending keep set of
// a head, the kept rows below C stay in their slots, and the kept rows at or
// past C (the movers, S[n_low..C)) fill the other slots below C (the free
// slots), both in ascending order.  Only the movers' rows are copied; their
// sources lie at or past C and their destinations below C, so no copy reads
// a row another one writes.  slots[c] = the old row slot c holds afterwards.
// Free slot number fi is f = fi + i*, i* the first i < n_low with
// S[i] - i > fi (S[i] - i free slots lie below S[i], a non-decreasing count),
// found by a binary search over S.  One work-group per head; VPR lanes per
// moved row (K and V).  A mover outside [C, L) (a keep list that is not an
// ascending set of rows) gives zero rows and sets bit 2 of the health words.
constexpr int kSlotThreads = 1024;
constexpr int kSlotLdsKeep = 16384;  // keep lists up to this long are searched in LDS

template <int VPR>
__global__ __launch_bounds__(kSlotThreads) void compact_slots_kernel(CompactLaunch a) {
  __shared__ int n_low_s;
  __shared__ int32_t keep_lds[kSlotLdsKeep];
  const int bh = blockIdx.x, b = bh / a.H, h = bh % a.H;
  const int32_t* Sg = a.keep + (int64_t)bh * a.C;
  int32_t* Y = a.slots + (int64_t)bh * a.C;
  u32x4* kb = static_cast<u32x4*>(a.k_out) + b * a.ks[0] + h * a.ks[1];
  u32x4* vb = static_cast<u32x4*>(a.v_out) + b * a.vs[0] + h * a.vs[1];
  constexpr int kRowsPerPass = kSlotThreads / VPR;
  const int vec = threadIdx.x % VPR;
  // The steps, over the keep list S (called with the LDS copy or with the
  // list in memory, each call on a pointer whose memory the compiler knows:
  // no generic pointer into LDS is formed).
  auto run = [&](const int32_t* S) {
    if (threadIdx.x == 0) n_low_s = a.C;
    __syncthreads();
    // The first entry at or past C (one writer when S ascends).
    for (int i = threadIdx.x; i < a.C; i += kSlotThreads)
      if (S[i] >= a.C && (i == 0 || S[i - 1] < a.C)) n_low_s = i;
    __syncthreads();
    const int n_low = n_low_s, n_move = a.C - n_low;
    for (int i = threadIdx.x; i < n_low; i += kSlotThreads) {
      const int r = S[i];
      if ((unsigned)r < (unsigned)a.C) Y[r] = r;  // a kept row below C keeps its slot
    }
    for (int fi0 = 0; fi0 < n_move; fi0 += kRowsPerPass) {
      const int fi = fi0 + (int)threadIdx.x / VPR;
      if (fi >= n_move) continue;
      int lo = 0, hi = n_low;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (S[mid] - mid > fi) hi = mid;
        else lo = mid + 1;
      }
      const int f = fi + lo;           // < n_move + n_low = C
      const int r = S[n_low + fi];     // the mover
      const bool ok = r >= a.C && r < a.L;
      if (vec == 0) {
        Y[f] = r;
        if (!ok) flag_bad_index(a.health);
      }
      const u32x4 z = {0u, 0u, 0u, 0u};
      const u32x4 xk = ok ? kb[(int64_t)r * a.ks[2] + vec] : z;
      const u32x4 xv = ok ? vb[(int64_t)r * a.vs[2] + vec] : z;
      kb[(int64_t)f * a.ks[2] + vec] = xk;
      vb[(int64_t)f * a.vs[2] + vec] = xv;
    }
  };
  // The binary searches read the keep list many times: from LDS when it fits.
  if (a.C <= kSlotLdsKeep) {
    for (int i = threadIdx.x; i < a.C; i += kSlotThreads) keep_lds[i] = Sg[i];
    run(keep_lds);
  } else {
    run(Sg);
  }
}

// Append: rows [row0, row0 + m) of every head of the cache take the m rows
// of k_new / v_new ([B, H, m, D] contiguous).
__global__ __launch_bounds__(kCompactThreads) void append_kernel(AppendLaunch a) {
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const int vpr = a.row_vecs;
  const int r = blockIdx.x * (kCompactThreads / vpr) + (int)threadIdx.x / vpr;
  if (r >= a.m) return;
  const int vec = threadIdx.x % vpr;
  const bool is_v = blockIdx.z != 0;
  const int64_t* st = is_v ? a.vs : a.ks;
  const u32x4* src = static_cast<const u32x4*>(is_v ? a.v_new : a.k_new) + ((int64_t)bh * a.m + r) * vpr + vec;
  u32x4* dst = static_cast<u32x4*>(is_v ? a.v : a.k) + b * st[0] + h * st[1] + (int64_t)(a.row0 + r) * st[2] + vec;
  *dst = *src;
}

namespace {

template <int VPR>
hipError_t launch_compact_t(const CompactLaunch& a, hipStream_t stream) {
  if (a.in_place) {
    hipLaunchKernelGGL(compact_inplace_kernel<VPR>, dim3(a.B * a.H, 2), dim3(kInplaceThreads), 0, stream, a);
    return hipGetLastError();
  }
  constexpr int rows_per_block = kCompactThreads / VPR;
  dim3 grid((a.C + rows_per_block - 1) / rows_per_block, a.B * a.H, 2);
  hipLaunchKernelGGL(compact_kernel<VPR>, grid, dim3(kCompactThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_compact(const CompactLaunch& a, hipStream_t stream) {
  if (a.C == 0) return hipSuccess;
  switch (a.row_vecs) {  // D in {64, 128} x element size in {2, 4}
    case 8: return launch_compact_t<8>(a, stream);
    case 16: return launch_compact_t<16>(a, stream);
    case 32: return launch_compact_t<32>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_compact_slots(const CompactLaunch& a, hipStream_t stream) {
  if (a.C == 0) return hipSuccess;
  if (!a.slots || a.k_out != a.k || a.v_out != a.v) return hipErrorInvalidValue;
  switch (a.row_vecs) {
    case 8: hipLaunchKernelGGL(compact_slots_kernel<8>, dim3(a.B * a.H), dim3(kSlotThreads), 0, stream, a); break;
    case 16: hipLaunchKernelGGL(compact_slots_kernel<16>, dim3(a.B * a.H), dim3(kSlotThreads), 0, stream, a); break;
    case 32: hipLaunchKernelGGL(compact_slots_kernel<32>, dim3(a.B * a.H), dim3(kSlotThreads), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_append(const AppendLaunch& a, hipStream_t stream) {
  if (a.m == 0) return hipSuccess;
  if (a.row_vecs <= 0 || kCompactThreads % a.row_vecs != 0) return hipErrorInvalidValue;
  const int rows_per_block = kCompactThreads / a.row_vecs;
  dim3 grid((a.m + rows_per_block - 1) / rows_per_block, a.B * a.H, 2);
  hipLaunchKernelGGL(append_kernel, grid, dim3(kCompactThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace nacl
