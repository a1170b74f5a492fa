// Keep-set selection (NaCl Section 5.1 argmax, Section 5.2 random eviction,
// Algorithm 1 union) for every (b, h):
//
//   Pi       the last n_protect proxy tokens, always kept
//   u_score  top-Cp of F over R = [0, L) \ Pi, ties to the lower index
//   u_random top-Cr of the Gumbel-perturbed keys over R \ u_score, ties to the
//            lower index: Gumbel-top-k, a draw of Cr tokens without
//            replacement from the weights (Softmax(F) by default)
//   keep     Pi | u_score | u_random, ascending, exactly C entries
//
// Keys are order-preserving uint32 images of the binary32 values (0 marks a
// token that is not a candidate).  Heads of up to kRegMaxL tokens take one
// work-group each, every thread holding up to 32 tokens' keys in registers
// (select_kernel_regs, described with it below).  Longer heads are cut into
// slices of kSelSlice tokens, one work-group each, every thread holding
// kSelPer consecutive tokens in registers; the work-groups of a head exchange
// data through the workspace in rounds (publish, count one arrival on the
// head's counter, wait for the other slices), and every work-group takes the
// same decisions from the same published data.
//
// (Both kernels are described with their code below.)

#include <type_traits>

#include "../../include/nacl.h"
#include "device_common.h"
#include "internal.h"
#include "gumbel.h"
#include "philox.h"

namespace nacl {

constexpr int kSelWaves = kSelThreads / kWave;
// Word 3 of a raw buffer descriptor on gfx9-family parts (32-bit data format).
constexpr int kSelBufferRsrcWord3 = 0x00020000;

// Calls f(std::integral_constant<int, i>) for i = 0 .. N-1.
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}
constexpr uint32_t kSelSpinLimit = 1u << 24;
constexpr int kSelMaxRounds = 80;

// Gumbel keys of every token (gumbel_order_key<MODE>), for a selection run
// on its own.  One kernel per mode keeps each straight-line.  One thread per
// Philox block, i.e. four consecutive tokens: 16-byte loads and stores when
// the rows allow (vec), the block evaluated once.
template <int MODE>
__global__ __launch_bounds__(256) void gumbel_keys_kernel(const float* __restrict__ F, int H, int L,
                                                          uint32_t k0, uint32_t k1, uint32_t layer, int vec,
                                                          uint32_t* __restrict__ keys) {
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int blk = blockIdx.x * 256 + threadIdx.x;
  const int j0 = 4 * blk;
  if (j0 >= L) return;
  const float* f = F + (int64_t)bh * L + j0;
  uint32_t* out = keys + (int64_t)bh * L + j0;
  const int n = min(4, L - j0);
  float fv[4] = {0.f, 0.f, 0.f, 0.f};
  if constexpr (MODE != 2) {
    if (vec) {
      const float4 v4 = *reinterpret_cast<const float4*>(f);
      fv[0] = v4.x;
      fv[1] = v4.y;
      fv[2] = v4.z;
      fv[3] = v4.w;
    } else {
      for (int e = 0; e < n; ++e) fv[e] = f[e];
    }
  }
  const U32x4 w = philox4x32_10(U32x4{(uint32_t)blk, (uint32_t)h, (uint32_t)b, layer}, k0, k1);
  const uint32_t word[4] = {w.x, w.y, w.z, w.w};
  uint32_t kv[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) kv[e] = gumbel_order_key<MODE>(fv[e], word[e]);
  if (vec) {
    *reinterpret_cast<uint4*>(out) = uint4{kv[0], kv[1], kv[2], kv[3]};
  } else {
    for (int e = 0; e < n; ++e) out[e] = kv[e];
  }
}

// Inclusive prefix sum over the wave by DPP: shifts of 1, 2, 4 and 8 lanes
// within each 16-lane row, then the last lane of a row broadcast into the
// next row (rows 1 and 3) and lane 31 into the upper half (rows 2 and 3).
// Lanes a shift leaves without a source add 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_or_zero(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROW_MASK, 0xf, false);
}

__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  x += dpp_or_zero<0x111, 0xf>(x);  // row_shr:1
  x += dpp_or_zero<0x112, 0xf>(x);  // row_shr:2
  x += dpp_or_zero<0x114, 0xf>(x);  // row_shr:4
  x += dpp_or_zero<0x118, 0xf>(x);  // row_shr:8
  x += dpp_or_zero<0x142, 0xa>(x);  // row_bcast:15
  x += dpp_or_zero<0x143, 0xc>(x);  // row_bcast:31
  return x;
}

// Exclusive prefix sum of v over the work-group in thread order.  scan_buf
// holds 2 * kSelWaves words of LDS: the wave totals, then their scan.  A
// call may follow another directly: a thread only writes the first half
// after every thread has left the previous call's second barrier, and the
// second half after every thread has read the previous call's result.
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* scan_buf) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t x = wave_inclusive_scan(v);
  if (lane == kWave - 1) scan_buf[wave] = x;
  __syncthreads();
  if (wave == 0) {
    uint32_t t = lane < kSelWaves ? scan_buf[lane] : 0u;
    t = wave_inclusive_scan(t);
    if (lane < kSelWaves) scan_buf[kSelWaves + lane] = t;
  }
  __syncthreads();
  const uint32_t base = wave ? scan_buf[kSelWaves + wave - 1] : 0u;
  return base + x - v;
}


// ===========================================================================
// Heads of up to kRegMaxL tokens: one work-group per head.
//
// Thread t holds the keys of the NR consecutive tokens NR t .. NR t + NR - 1
// in registers (NR = 32, or 16 or 8 for heads of at most 16 or 8 times the
// work-group's threads: fewer slots per thread, the same steps).  Each key
// set (scores, then Gumbel keys) is staged in LDS by direct buffer->LDS loads
// (contiguous 16-byte pieces per lane) and read back as NR / 4 16-byte pieces
// per thread in the rotated order (q + t) mod (NR / 4), which spreads the
// lanes an LDS cycle serves over the banks (for NR = 32 over distinct ones);
// so register slot i holds token NR t + ((i + 4 t) mod NR), and a mask over
// the slots is a mask over the thread's tokens rotated by 4 t mod NR.  The
// Gumbel keys are loaded into the staging buffer while the scores are
// searched.
// Top-k of one key set (the k-th largest key T, and `need`, how many keys
// equal to T the top k holds; ties go to the lower index):
//   1. window: one sampled key per thread (a different slot in each thread,
//      so the sample spans the head) goes into a histogram of its top 12
//      bits; the bins holding the sample's ranks k*m/n -/+ three standard
//      deviations give a window [lo, hi) that holds the k-th largest key in
//      all likelihood.  The largest key M is reduced at the same time;
//   2. every key at or above lo is counted in 4095 equal bins of width 2^sh
//      covering [lo, min(hi, M + 1)), plus one bin for everything above, and
//      the bin holding the k-th largest key is picked: its keys share all
//      bits at and above sh;
//   3. when every key of that bin is taken, "key >= the bin's lower edge"
//      is the top k; otherwise a bin of at most kRegCand keys is gathered and
//      ranked in one wave, and a larger one takes radix passes over the bits
//      below sh.  When the window misses the k-th key, a plain radix select
//      (12-, 12- and 8-bit digits) over all keys runs instead.
// Each histogram is read by one wave (64 bins per lane, a wave scan over the
// lanes, then one bin per lane inside the crossing lane's range), so a pass
// costs two barriers.  Membership is then a register compare, with a block
// scan of the per-thread counts of keys equal to T when only some of them
// are taken.  Assembly scans the per-thread counts of kept tokens, and every
// thread stores its kept indices in order at the offset the scan gives.

constexpr int kRegKeys = 32;
constexpr int kRegMaxL = kRegKeys * kSelThreads;
// Shorter heads hold 8 or 16 tokens per thread (up to 8 or 16 times
// kSelThreads tokens): the same steps with fewer slots per thread.
static_assert(kRegMaxL == kSelRegMaxL, "register selection length");
constexpr int kHistBins = 4096;
static_assert(kHistBins == 64 * kWave, "histogram scan: 64 bins per lane of one wave");

constexpr int kRegCand = kWave;  // bins resolved by one wave

// A barrier without the full fence of __syncthreads(): it waits for this
// wave's LDS operations (so LDS writes before it are seen by every wave after
// it) but not for its vector memory operations, so the buffer->LDS loads of
// the Gumbel keys stay in flight across it (a fence would wait for them,
// since they write LDS).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// LDS atomics written as instructions the compiler does not see as memory
// accesses: it makes every LDS atomic that follows a buffer->LDS load wait
// for that load (it cannot tell them apart), which would make the score
// search wait for the Gumbel keys.  Every LDS location they touch is read
// only after a barrier (which waits for them), and the LDS counter counts
// them in issue order, so the compiler's own LDS waits stay sufficient.
__device__ __forceinline__ uint32_t lds_off(const uint32_t* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint32_t*)p;
}
__device__ __forceinline__ void lds_add(uint32_t* p, uint32_t v) {
  asm volatile("ds_add_u32 %0, %1" ::"v"(lds_off(p)), "v"(v));
}
__device__ __forceinline__ void lds_or(uint32_t* p, uint32_t v) {
  asm volatile("ds_or_b32 %0, %1" ::"v"(lds_off(p)), "v"(v));
}
__device__ __forceinline__ void lds_max(uint32_t* p, uint32_t v) {
  asm volatile("ds_max_u32 %0, %1" ::"v"(lds_off(p)), "v"(v));
}
// Clears 16 bytes (the compiler also makes LDS stores it cannot tell apart
// from the buffer->LDS loads wait for them).
__device__ __forceinline__ void lds_zero16(uint32_t* p) {
  const u32x4 z = {0u, 0u, 0u, 0u};
  asm volatile("ds_write_b128 %0, %1" ::"v"(lds_off(p)), "v"(z));
}
// Returns the old value (waits for it).
__device__ __forceinline__ uint32_t lds_add_rtn(uint32_t* p, uint32_t v) {
  uint32_t r;
  asm volatile("ds_add_rtn_u32 %0, %1, %2\n\ts_waitcnt lgkmcnt(0)" : "=v"(r) : "v"(lds_off(p)), "v"(v));
  return r;
}

// LDS of a work-group of NT threads.
template <int NT>
struct RegLds {
  static constexpr int kWaves = NT / kWave;
  alignas(16) uint32_t hist[kHistBins];  // all zero between passes
  uint32_t fixed[NT];                    // Pi, one bit per token (word t: tokens 32 t ..)
  uint32_t cand[kRegCand];               // keys of the k-th bin (step 3)
  uint32_t pick[2][4];                   // per rank: found, bin, rank within the bin, bin count
  uint32_t scan[2 * kWaves];
  uint32_t shv[8];                       // 0-2 ranked result, 4 gather counter, 5 max key, 6 valid samples
};

struct TopK {
  uint32_t T, need, n_eq;
};

__device__ __forceinline__ uint32_t rotr32(uint32_t x, uint32_t r) { return __builtin_amdgcn_alignbit(x, x, r); }
__device__ __forceinline__ uint32_t rotl32(uint32_t x, uint32_t r) { return __builtin_amdgcn_alignbit(x, x, (32u - r) & 31u); }
// Rotations of the low NR bits of a mask (NR slots per thread, r < NR).
template <int NR>
__device__ __forceinline__ uint32_t rotr_n(uint32_t x, uint32_t r) {
  if constexpr (NR == 32) return rotr32(x, r);
  else return ((x >> r) | (x << ((NR - r) & 31u))) & ((1u << NR) - 1u);
}
template <int NR>
__device__ __forceinline__ uint32_t rotl_n(uint32_t x, uint32_t r) {
  return rotr_n<NR>(x, (NR - r) % NR);
}

// Maximum over the wave (the inclusive scan's shifts with max).
__device__ __forceinline__ uint32_t wave_max(uint32_t x) {
  x = max(x, dpp_or_zero<0x111, 0xf>(x));
  x = max(x, dpp_or_zero<0x112, 0xf>(x));
  x = max(x, dpp_or_zero<0x114, 0xf>(x));
  x = max(x, dpp_or_zero<0x118, 0xf>(x));
  x = max(x, dpp_or_zero<0x142, 0xa>(x));
  x = max(x, dpp_or_zero<0x143, 0xc>(x));
  return (uint32_t)__builtin_amdgcn_readlane((int)x, kWave - 1);
}

// Exclusive prefix sum of v over the work-group in thread order (the scan of
// block_exclusive_scan with barriers that leave the buffer->LDS loads in
// flight).
template <int NW>
__device__ __forceinline__ uint32_t reg_block_scan(uint32_t v, uint32_t* scan_buf) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t x = wave_inclusive_scan(v);
  if (lane == kWave - 1) scan_buf[wave] = x;
  lds_barrier();
  if (wave == 0) {
    uint32_t t = lane < NW ? scan_buf[lane] : 0u;
    t = wave_inclusive_scan(t);
    if (lane < NW) scan_buf[NW + lane] = t;
  }
  lds_barrier();
  const uint32_t base = wave ? scan_buf[NW + wave - 1] : 0u;
  return base + x - v;
}

// Sorts the 64 * R keys v[r] of lane l (element l * R + r) of one wave into
// descending order by a bitonic network in registers: stages within a lane
// swap registers, stages across lanes exchange with the partner lane.
template <int R>
__device__ __forceinline__ void wave_sort_desc(uint32_t (&v)[R]) {
  const int lane = threadIdx.x & 63;
  static_for<__builtin_ctz(64 * R)>([&](auto kc) {
    constexpr int k = 2 << decltype(kc)::value;
    static_for<decltype(kc)::value + 1>([&](auto jc) {
      constexpr int j = k >> (1 + decltype(jc)::value);
      if constexpr (j < R) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          if ((r & j) == 0) {
            const bool desc = ((lane * R + r) & k) == 0;
            const uint32_t x = v[r], y = v[r | j];
            v[r] = desc ? max(x, y) : min(x, y);
            v[r | j] = desc ? min(x, y) : max(x, y);
          }
        }
      } else {
        constexpr int lm = j / R;  // partner lane = lane ^ lm
        const bool lower = (lane & lm) == 0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const bool desc = ((lane * R + r) & k) == 0;
          const uint32_t y = (uint32_t)__shfl_xor((int)v[r], lm);
          v[r] = (lower == desc) ? max(v[r], y) : min(v[r], y);
        }
      }
    });
  });
}

// Called by every thread once a histogram is complete (after its barrier).
// For each rank kr[r] (1-based from the top; 0: none), wave 0 finds the bin
// at which the count from the top reaches it and stores (found, bin, rank
// within the bin, bin count) in s.pick[r]; it also clears the histogram.
// Lane l owns bins 4095 - 64 l down to 4032 - 64 l, read and cleared as 16
// pieces of four bins in the order (q + l) mod 16, so that the eight lanes
// an LDS cycle serves touch distinct banks.  Ends with a barrier.
template <int NRK>
__device__ __forceinline__ void pick_bins(uint32_t* hist, uint32_t (*pick)[4], const uint32_t (&kr)[NRK]) {
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    uint4* own = reinterpret_cast<uint4*>(hist + kHistBins - 64 * (lane + 1));
    uint32_t sum = 0u;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const uint4 v = own[(q + lane) & 15];
      sum += v.x + v.y + v.z + v.w;
    }
    const uint32_t incl = wave_inclusive_scan(sum);
    const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, kWave - 1);
#pragma unroll
    for (int r = 0; r < NRK; ++r) {
      const uint32_t want = kr[r];
      if (want == 0u || want > total) {
        if (lane == 0) pick[r][0] = 0u;
        continue;
      }
      const int l0 = (int)__builtin_ctzll(__ballot(incl >= want));
      const uint32_t above = (uint32_t)__builtin_amdgcn_readlane((int)(incl - sum), l0);
      const int b = kHistBins - 1 - 64 * l0 - lane;  // lane m: the m-th bin of lane l0 from the top
      const uint32_t c = hist[b];
      const uint32_t inc2 = above + wave_inclusive_scan(c);
      const int m = (int)__builtin_ctzll(__ballot(inc2 >= want));
      if (lane == m) {
        pick[r][0] = 1u;
        pick[r][1] = (uint32_t)b;
        pick[r][2] = want - (inc2 - c);
        pick[r][3] = c;
      }
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) lds_zero16(reinterpret_cast<uint32_t*>(own + ((q + lane) & 15)));
  }
  lds_barrier();
}

template <int NRK, class Lds>
__device__ __forceinline__ void pick_bins(Lds& s, const uint32_t (&kr)[NRK]) {
  pick_bins(s.hist, s.pick, kr);
}

// The kr-th largest of the keys whose bits at and above `bits` equal those
// of prefix (its lower bits zero; bits == 32: every key), by radix passes of
// 12 bits (the last one narrower) over the bits below; key 0 never counts.
// At least kr keys must match.
template <int NR, class Lds>
__device__ __forceinline__ TopK radix_rest(const uint32_t (&key)[NR], Lds& s, uint32_t prefix, int bits,
                                           uint32_t kr) {
  uint32_t n_eq = 0u;
#pragma unroll 1
  while (bits > 0) {
    const int d = bits > 12 ? 12 : bits;
    const int shift = bits - d;
    const uint32_t hm = bits >= 32 ? 0u : (0xFFFFFFFFu << bits);
    const uint32_t dmask = (1u << d) - 1u;
#pragma unroll
    for (int i = 0; i < NR; ++i)
      if (key[i] != 0u && ((key[i] ^ prefix) & hm) == 0u) lds_add(&s.hist[(key[i] >> shift) & dmask], 1u);
    lds_barrier();
    const uint32_t want[1] = {kr};
    pick_bins(s, want);
    prefix |= s.pick[0][1] << shift;
    kr = s.pick[0][2];
    n_eq = s.pick[0][3];
    bits = shift;  // s.pick is next written after the next histogram's barrier
  }
  return TopK{prefix, kr, n_eq};
}

// Top k (1 <= k <= number of nonzero keys) of the register keys; n_valid is
// the number of nonzero keys of the head (it only scales the sample ranks).
template <int NR, class Lds>
__device__ __forceinline__ TopK reg_top_k(const uint32_t (&key)[NR], uint32_t k, uint32_t n_valid, Lds& s) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // 1. One sampled key per thread (slot 0, whose token offset rotates from
  // thread to thread), and the largest key.
  const uint32_t smp = key[0];
  uint32_t vmax = 0u;
#pragma unroll
  for (int i = 0; i < NR; ++i) vmax = max(vmax, key[i]);
  vmax = wave_max(vmax);
  const uint64_t sb = __ballot(smp != 0u);
  if (lane == 0) {
    lds_max(&s.shv[5], vmax);
    lds_add(&s.shv[6], (uint32_t)__popcll(sb));
  }
  if (smp != 0u) lds_add(&s.hist[smp >> 20], 1u);
  lds_barrier();
  const uint32_t M = s.shv[5], n_s = s.shv[6];
  const float e = (float)k * (float)n_s / (float)n_valid;
  const float dev = 3.f * sqrtf(e) + 3.f;
  const uint32_t want[2] = {n_s ? min(n_s, (uint32_t)ceilf(e + dev)) : 0u,
                            e - dev >= 1.f ? (uint32_t)(e - dev) : 0u};
  pick_bins(s, want);
  const bool have_lo = s.pick[0][0] != 0u, have_hi = s.pick[1][0] != 0u;
  const uint64_t lo = (uint64_t)s.pick[0][1] << 20;
  const uint64_t hi = have_hi ? min((uint64_t)(s.pick[1][1] + 1u) << 20, (uint64_t)M + 1u) : (uint64_t)M + 1u;
  // Every thread read the maximum and the sample count before pick_bins's
  // barrier; s.pick is next written after the next histogram's barrier.
  if (tid == 0) {
    s.shv[4] = 0u;
    s.shv[5] = 0u;
    s.shv[6] = 0u;
  }
  // Radix passes left to do: over the bits below rbits of the keys matching
  // rprefix, for the rkr-th largest.
  uint32_t rprefix = 0u, rkr = k;
  int rbits = 32;
  if (have_lo) {
    // 2. Bins 0..4094 of width 2^sh cover [lo, hi); bin 4095 takes the rest.
    //    sh <= 20 unless lo == 0, so lo is a multiple of 2^sh.
    const uint64_t range = hi > lo ? hi - lo : 1u;
    int sh = 0;
    while (((uint64_t)(kHistBins - 1) << sh) < range) ++sh;
    const uint32_t lo32 = (uint32_t)lo, lo_nz = lo32 ? lo32 : 1u;  // key 0 never counts
#pragma unroll
    for (int i = 0; i < NR; ++i)
      if (key[i] >= lo_nz) lds_add(&s.hist[min((key[i] - lo32) >> sh, (uint32_t)(kHistBins - 1))], 1u);
    lds_barrier();
    const uint32_t want1[1] = {k};
    pick_bins(s, want1);
    const bool found = s.pick[0][0] != 0u && s.pick[0][1] != (uint32_t)(kHistBins - 1);
    const uint32_t pfx = (lo32 >> sh) + s.pick[0][1];
    const uint32_t kr = s.pick[0][2], n1 = s.pick[0][3];
    if (found) {
      // 3. Keys with high bits pfx: the kr-th largest of the n1 of them.
      if (sh == 0) return TopK{pfx, kr, n1};
      if (kr == n1) return TopK{pfx << sh, n1, n1};
      rprefix = pfx << sh;
      rbits = sh;
      rkr = kr;
      if (n1 <= (uint32_t)kRegCand) {
#pragma unroll
        for (int i = 0; i < NR; ++i) {
          const bool m = key[i] != 0u && (key[i] >> sh) == pfx;
          if (m) s.cand[lds_add_rtn(&s.shv[4], 1u)] = key[i];
        }
        lds_barrier();
        if (wave == 0) {
          // Lane l holds candidate l; it counts the candidates above and
          // equal to its own.  The lanes whose key is the kr-th largest
          // publish it.
          const uint32_t v = lane < (int)n1 ? s.cand[lane] : 0u;
          uint32_t n_gt = 0u, n_eq = 0u;
          for (int j = 0; j < (int)n1; ++j) {
            const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)v, j);
            n_gt += c > v ? 1u : 0u;
            n_eq += c == v ? 1u : 0u;
          }
          if (lane < (int)n1 && n_gt < kr && kr <= n_gt + n_eq) {
            s.shv[0] = v;
            s.shv[1] = kr - n_gt;
            s.shv[2] = n_eq;
          }
          if (lane == 0) s.shv[4] = 0u;
        }
        lds_barrier();
        // shv[0..2] are next written after several more barriers.
        return TopK{s.shv[0], s.shv[1], s.shv[2]};
      }
    }
  }
  return radix_rest(key, s, rprefix, rbits, rkr);
}

// Bit i: the token of slot i belongs to the top k described by r (rot: the
// thread's slot rotation).
template <int NR, class Lds>
__device__ __forceinline__ uint32_t top_members(const uint32_t (&key)[NR], const TopK& r, uint32_t rot,
                                                Lds& s) {
  uint32_t in = 0u;
  if (r.need == r.n_eq) {
#pragma unroll
    for (int i = 0; i < NR; ++i) in |= (key[i] >= r.T ? 1u : 0u) << i;
    return in;
  }
  // Only the first `need` keys equal to T, in token order, are taken.
  uint32_t tie = 0u;
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    in |= (key[i] > r.T ? 1u : 0u) << i;
    tie |= (key[i] == r.T ? 1u : 0u) << i;
  }
  uint32_t t_tok = rotl_n<NR>(tie, rot);  // token order
  const uint32_t n = (uint32_t)__popc(t_tok);
  const uint32_t before = reg_block_scan<Lds::kWaves>(n, s.scan);
  uint32_t take = min(r.need - min(r.need, before), n);  // need - before, or 0 past the need-th tie
  uint32_t kept_tok = 0u;
  while (take--) {
    const uint32_t low = t_tok & (0u - t_tok);
    kept_tok |= low;
    t_tok ^= low;
  }
  return in | rotr_n<NR>(kept_tok, rot);
}

template <int NT, int NR>
__global__ __launch_bounds__(NT) void select_kernel_regs(SelectLaunch a) {
  static_assert(NR == 8 || NR == 16 || NR == 32, "keys per thread");
  constexpr int kNW = NT / kWave;          // waves
  constexpr int kMaxL = NR * NT;           // tokens the work-group holds
  __shared__ RegLds<NT> s;
  __shared__ uint32_t stage[kMaxL];  // one key set of the head, by buffer->LDS loads
  const int L = a.L;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bh = blockIdx.x;
  const uint32_t* fsrc = reinterpret_cast<const uint32_t*>(a.scores) + (int64_t)bh * L;
  const uint32_t* gsrc = a.keys2 + (int64_t)bh * L;

  const int pbase = a.P - a.n_protect;
  const int p0 = pbase + tid < a.P ? a.pos[pbase + tid] : -1;

  // Stages the head's L words at src in `stage` (reads at or past L, or all
  // of them when n == 0, return zeros).  Rows that allow it move 16 bytes
  // per lane: instruction r of wave w moves tokens [256 (16 r + w), + 256).
  auto stage_keys = [&](const uint32_t* src, int n) {
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint32_t*>(src), (short)0, (int)((uint32_t)n * 4u), kSelBufferRsrcWord3);
    if ((L & 3) == 0 && ((uintptr_t)src & 15u) == 0) {
#pragma unroll
      for (int r = 0; r < kMaxL / (256 * kNW); ++r) {
        const uint32_t t0 = 256u * (uint32_t)(kNW * r + wave);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(stage + t0), 16,
                                                 (t0 + 4u * (uint32_t)lane) * 4u, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int r = 0; r < kMaxL / (64 * kNW); ++r) {
        const uint32_t t0 = 64u * (uint32_t)(kNW * r + wave);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(stage + t0), 4,
                                                 (t0 + (uint32_t)lane) * 4u, 0, 0, 0);
      }
    }
  };
  // Thread t's NR staged words, slot i = token NR t + ((i + rot) mod NR).
  const uint32_t rot = (4u * (uint32_t)tid) & (uint32_t)(NR - 1);
  uint32_t key[NR];
  auto read_stage = [&]() {
    const uint4* row = reinterpret_cast<const uint4*>(stage + NR * tid);
#pragma unroll
    for (int q = 0; q < NR / 4; ++q) {
      const uint4 v = row[(q + tid) & (NR / 4 - 1)];
      key[4 * q] = v.x;
      key[4 * q + 1] = v.y;
      key[4 * q + 2] = v.z;
      key[4 * q + 3] = v.w;
    }
  };

  stage_keys(fsrc, a.Cp > 0 ? L : 0);
  s.fixed[tid] = 0u;
#pragma unroll
  for (int q = 0; q < kHistBins / NT; ++q) s.hist[q * NT + tid] = 0u;
  if (tid < 8) s.shv[tid] = 0u;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's loads
  lds_barrier();                                    // everyone's, and the clears
  if (p0 >= 0) lds_or(&s.fixed[p0 >> 5], 1u << (p0 & 31));
  for (int i = pbase + tid + NT; i < a.P; i += NT) {
    const int j = a.pos[i];
    lds_or(&s.fixed[j >> 5], 1u << (j & 31));
  }
  read_stage();
  lds_barrier();  // Pi marked; every thread has read the scores
  // The Gumbel keys arrive while the scores are searched.  (Without random
  // tokens the loads read nothing and write zeros; they are issued anyway,
  // which keeps the compiler's wait counts the same on every path.)
  stage_keys(gsrc, a.Cr > 0 ? L : 0);

  // Bit i of each mask: the token of slot i is in Pi (mp), u_score (ms),
  // u_random (mr).  Tokens past the end are in none.
  const int nt = L - NR * tid;
  const uint32_t all = NR == 32 ? 0xFFFFFFFFu : (1u << NR) - 1u;
  const uint32_t live_tok = nt >= NR ? all : (nt > 0 ? (1u << nt) - 1u : 0u);
  const uint32_t live = rotr_n<NR>(live_tok, rot);
  // This thread's NR bits of the token bitmap (word w: tokens 32 w .. 32 w + 31).
  const uint32_t fixed_tok = NR == 32 ? s.fixed[tid] : (s.fixed[(NR * tid) >> 5] >> ((NR * tid) & 31)) & all;
  const uint32_t mp = rotr_n<NR>(fixed_tok, rot);
  uint32_t ms = 0u, mr = 0u;

  // u_score: top-Cp of F over R = [0, L) \ Pi.
  if (a.Cp > 0) {
#pragma unroll
    for (int i = 0; i < NR; ++i)
      key[i] = ((live & ~mp) >> i) & 1u ? float_order_key(__uint_as_float(key[i])) : 0u;
    const TopK r = reg_top_k(key, (uint32_t)a.Cp, (uint32_t)(L - a.n_protect), s);
    ms = top_members(key, r, rot, s);
  }

  // u_random: top-Cr of the Gumbel keys over R \ u_score.
  if (a.Cr > 0) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's loads
    lds_barrier();                                    // everyone's
    read_stage();
    const uint32_t cand = live & ~mp & ~ms;
#pragma unroll
    for (int i = 0; i < NR; ++i)
      if (!((cand >> i) & 1u)) key[i] = 0u;
    const TopK r = reg_top_k(key, (uint32_t)a.Cr, (uint32_t)(L - a.n_protect - a.Cp), s);
    mr = top_members(key, r, rot, s);
  }

  // keep = Pi | u_score | u_random in index order: C entries by construction
  // (the bound only guards the write).  The list is assembled in the staging
  // buffer (every thread has read the Gumbel keys from it before the last
  // selection's barriers), then copied out with coalesced stores.
  uint32_t kept = rotl_n<NR>(mp | ms | mr, rot);
  if (a.Cr == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the zero loads into the buffer
  uint32_t o = reg_block_scan<kNW>((uint32_t)__popc(kept), s.scan);  // (its barriers: everyone's)
  while (kept) {
    const int b = __builtin_ctz(kept);
    if (o < (uint32_t)a.C) stage[o] = (uint32_t)(NR * tid + b);
    ++o;
    kept &= kept - 1u;
  }
  lds_barrier();
  int32_t* out = a.keep + (int64_t)bh * a.C;
  for (int c = tid; c < a.C; c += NT) out[c] = (int32_t)stage[c];
}

// ===========================================================================
// Longer heads: slices of kSelSlice tokens, one work-group each.
//
// Thread t of slice p holds the scores and Gumbel keys of the kSelPer
// consecutive tokens p * kSelSlice + kSelPer * t + i in registers.  The
// work-groups of a head take the same decisions from the same data: each
// derives the window from the same sampled tokens (read from memory), and
// they exchange histograms and candidate lists through the workspace in
// rounds (publish with device-coherent stores, count an arrival on the
// head's counter, wait for the other slices).  Top-k of one key set:
//   1. window: 1024 tokens spread evenly over the head are sampled (Pi and
//      tokens already taken left out); the bins of their top 12 bits that
//      hold the sample ranks k*m/n -/+ three standard deviations give
//      [lo, hi);
//   2. each slice counts its keys in [lo, top) in 4095 equal bins of width
//      2^sh over [lo, hi) plus one bin for the rest (top is unbounded in the
//      first pass), and publishes the bins and their totals per group of
//      64; after the round every work-group reads the group totals of all
//      slices, then the bins of the group holding the k-th key, and so the
//      bin holding it and how many keys each slice has above it and in it;
//   3. if that bin is one key value wide, or the top k takes all of it, the
//      threshold follows from the counts; if it holds at most kSelCandMax
//      keys, the slices publish them (key, index) in index order and every
//      work-group ranks them; otherwise, or if the window missed the k-th
//      key, the window moves to that bin (or below lo, or above the regular
//      bins) and step 2 repeats.
// The top k is then "key > T, or key == T with a rank among the T-keys, in
// index order, below need"; every work-group knows each slice's count of
// taken keys, so the assembly writes each slice's kept indices at their
// offset of the keep list without another round.

constexpr int kSliceHistWords = kHistBins + kHistBins / kWave;  // bins, then the 64 group totals
static_assert(kSliceHistWords == kSelHistWords, "published histogram size");
constexpr int kSelMaxPasses = 16;

struct SliceLds {
  alignas(16) uint32_t hist[kHistBins];  // all zero between passes
  uint32_t ppos[NACL_MAX_P];             // protected positions, ascending
  uint32_t ckey[kSelCandMax], cidx[kSelCandMax];
  uint32_t above[kSelMaxSlices];  // per slice: keys above the current window (this selection)
  uint32_t inbin[kSelMaxSlices];  // per slice: keys in the k-th bin
  uint32_t gt[kSelMaxSlices];     // per slice: keys of the k-th bin above T
  uint32_t eq[kSelMaxSlices];     // per slice: keys equal to T
  uint32_t taken[2][kSelMaxSlices];
  uint32_t prot[kSelMaxSlices];
  uint32_t pick[2][4];
  uint32_t scan[2 * kSelWaves];
  uint32_t shv[16];
  uint32_t list[kSelSlice];       // this slice's kept indices, in order
};

// Sum over the wave.
__device__ __forceinline__ uint32_t wave_sum(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_inclusive_scan(x), kWave - 1);
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectLaunch a) {
  __shared__ SliceLds s;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = a.L, nb = a.nb;
  if (tid == 0) s.shv[0] = atomicAdd(a.sync, 1u);
  __syncthreads();
  const int ticket = (int)s.shv[0];
  if (ticket >= a.B * a.H * nb) {  // counters not cleared (never expected)
    if (tid == 0 && a.health) {
      atomicOr(a.health, 8u);
      atomicOr(a.health + 1, 8u);
    }
    return;
  }
  const int bh = ticket / nb, part = ticket % nb;
  uint32_t* counter = a.sync + 64 + bh;
  const int j0 = part * kSelSlice + tid * kSelPer;  // this thread's first token
  const int nrem = L - j0;                          // tokens of the head from j0 on
  const int pbase = a.P - a.n_protect;
  const uint32_t* frow = reinterpret_cast<const uint32_t*>(a.scores) + (int64_t)bh * L;
  const uint32_t* grow = a.keys2 + (int64_t)bh * L;
  int round = 0;
  bool gave_up = false;  // a wait or the pass limit gave up (never expected)

  // Arrival on the head's counter, then wait for every slice of the head.
  auto exchange = [&]() {
    wait_stores();
    __syncthreads();
    if (tid == 0) {
      atomicAdd(counter, 1u);
      const uint32_t target = (uint32_t)nb * (uint32_t)(round + 1);
      uint32_t spins = 0;
      while (load_coherent(counter) < target) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins > kSelSpinLimit) {
          s.shv[9] = 1u;
          break;
        }
      }
    }
    ++round;
    __syncthreads();
    gave_up = gave_up || s.shv[9] != 0u;
  };

  // This thread's kSelPer consecutive tokens of a row (16-byte loads when
  // the row allows; past the end of the head the last token repeats and is
  // masked below).
  auto load_row = [&](const uint32_t* row, uint32_t (&out)[kSelPer]) {
    if ((L % 4 == 0) && j0 + kSelPer <= L && ((uintptr_t)row % 16u) == 0) {
#pragma unroll
      for (int q = 0; q < kSelPer / 4; ++q) {
        const uint4 v = *reinterpret_cast<const uint4*>(row + j0 + 4 * q);
        out[4 * q] = v.x;
        out[4 * q + 1] = v.y;
        out[4 * q + 2] = v.z;
        out[4 * q + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < kSelPer; ++i) out[i] = row[nrem > 0 ? j0 + min(i, nrem - 1) : L - 1];
    }
  };
  uint32_t fk[kSelPer];
  load_row(frow, fk);
  // This thread's sampled token, the same in every slice of the head.
  const int js = (int)(((int64_t)tid * L) >> 10);
  const uint32_t f_smp = frow[js], g_smp = a.Cr > 0 ? grow[js] : 0u;

  // The protected positions staged in LDS.
  const int np = a.n_protect;
  for (int i = tid; i < np; i += kSelThreads) s.ppos[i] = (uint32_t)a.pos[pbase + i];
  if (tid >= 1 && tid < 16) s.shv[tid] = 0u;  // shv[0] (the ticket) is next written after barriers
  for (int i = tid; i < kHistBins; i += kSelThreads) s.hist[i] = 0u;
  __syncthreads();
  auto first_at_least = [&](int x) {  // first staged position >= x
    int lo = 0, hi = np;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if ((int)s.ppos[mid] < x) lo = mid + 1;
      else hi = mid;
    }
    return lo;
  };
  auto protected_token = [&](int j) {
    const int i = first_at_least(j);
    return i < np && (int)s.ppos[i] == j;
  };
  uint32_t prot = 0u;  // bit i: token j0 + i is protected
  if (np > 0 && j0 < L)
    for (int i = first_at_least(j0); i < np && (int)s.ppos[i] < j0 + kSelPer; ++i) prot |= 1u << (s.ppos[i] - j0);
#pragma unroll
  for (int i = 0; i < kSelPer; ++i) {
    const bool cand = i < nrem && !((prot >> i) & 1u);
    fk[i] = cand ? float_order_key(__uint_as_float(fk[i])) : 0u;
  }
  // Protected proxies per slice (for the assembly offsets).
  if (tid < nb) s.prot[tid] = (uint32_t)(first_at_least((tid + 1) * kSelSlice) - first_at_least(tid * kSelSlice));

  // Top k (1 <= k <= the head's nonzero keys, n_valid of them) of the key
  // sets key[] of the head's slices; thread t's sampled key is that of token
  // (t * L) / 1024 (0: not a candidate).  Sets s.taken[which][q] for every
  // slice; returns this thread's member mask.
  auto top_k = [&](const uint32_t (&key)[kSelPer], uint32_t k, uint32_t n_valid, int which, uint32_t sk,
                   uint32_t& T_out) -> uint32_t {
    // 1. The window from the sample (sk: this thread's sampled key).
    if (tid < nb) s.above[tid] = 0u;
    const uint64_t sb = __ballot(sk != 0u);
    if (lane == 0 && sb) atomicAdd(&s.shv[6], (uint32_t)__popcll(sb));
    if (sk != 0u) atomicAdd(&s.hist[sk >> 20], 1u);
    __syncthreads();
    const uint32_t n_s = s.shv[6];
    const float e = (float)k * (float)n_s / (float)n_valid;
    const float dev = 3.f * sqrtf(e) + 3.f;
    const uint32_t want[2] = {n_s ? min(n_s, (uint32_t)ceilf(e + dev)) : 0u,
                              n_s ? (e - dev >= 1.f ? (uint32_t)(e - dev) : 1u) : 0u};
    pick_bins(s.hist, s.pick, want);
    uint32_t lo = 1u;
    uint64_t hi = 1ull << 32;
    if (s.pick[0][0] != 0u) {
      lo = max(1u, s.pick[0][1] << 20);
      hi = (uint64_t)(s.pick[1][1] + 1u) << 20;  // rank 1 always exists when rank want[0] does
    }
    __syncthreads();  // pick and sample count read
    if (tid == 0) s.shv[6] = 0u;

    // 2-3. Passes over [lo, top) until the k-th key's bin is resolved.
    bool open = true;  // top unbounded: bin 4095 takes every key past the regular bins
    uint32_t krem = k, T = 0u, need = 0u;
    bool all_bin = false;
#pragma unroll 1
    for (int pass = 0;; ++pass) {
      const uint64_t range = hi > (uint64_t)lo ? hi - lo : 1u;
      int sh = 0;
      while (((uint64_t)(kHistBins - 1) << sh) < range) ++sh;
#pragma unroll
      for (int i = 0; i < kSelPer; ++i)
        if (key[i] >= lo && (open || (uint64_t)key[i] < hi))
          atomicAdd(&s.hist[min((key[i] - lo) >> sh, (uint32_t)(kHistBins - 1))], 1u);
      __syncthreads();
      // Publish the bins (thread t: bins 4t .. 4t + 3, then clears them) and
      // the group totals (group g: bins 4095 - 64 g down to 4032 - 64 g, the
      // bins of the 16 threads of one 16-lane row).
      {
        uint32_t* xh = a.xhist + (((int64_t)bh * 2 + (round & 1)) * nb + part) * kSliceHistWords;
        u32x4* mine = reinterpret_cast<u32x4*>(s.hist + 4 * tid);
        const u32x4 v = *mine;
        store_coherent16(xh + 4 * tid, v);
        *mine = u32x4{0u, 0u, 0u, 0u};
        uint32_t r = v.x + v.y + v.z + v.w;
        r += dpp_or_zero<0x111, 0xf>(r);
        r += dpp_or_zero<0x112, 0xf>(r);
        r += dpp_or_zero<0x114, 0xf>(r);
        r += dpp_or_zero<0x118, 0xf>(r);
        if ((tid & 15) == 15) store_coherent(xh + kHistBins + (kWave - 1 - (tid >> 4)), r);
      }
      exchange();
      if (wave == 0) {
        // Lane g: group g's totals; then lane m: the m-th bin of the group
        // holding the k-th key.  The slices' words are loaded eight at a time.
        const uint32_t* base = a.xhist + ((int64_t)bh * 2 + ((round - 1) & 1)) * nb * kSliceHistWords;
        auto sum_over_slices = [&](int word) {
          uint32_t sum = 0u;
          for (int q0 = 0; q0 < nb; q0 += 8) {
            uint32_t v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
              v[u] = q0 + u < nb ? load_coherent(base + (q0 + u) * kSliceHistWords + word) : 0u;
#pragma unroll
            for (int u = 0; u < 8; ++u) sum += v[u];
          }
          return sum;
        };
        // Up to eight slices keep their words in registers between the
        // steps; more slices load them again.
        uint32_t tg8[8], cb8[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          tg8[u] = u < nb ? load_coherent(base + u * kSliceHistWords + kHistBins + lane) : 0u;
        uint32_t gsum = 0u;
#pragma unroll
        for (int u = 0; u < 8; ++u) gsum += tg8[u];
        if (nb > 8) gsum = sum_over_slices(kHistBins + lane);
        const uint32_t incl = wave_inclusive_scan(gsum);
        const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, kWave - 1);
        if (total < krem) {
          // Every key at or above lo is taken; the k-th key lies below lo.
          for (int q = 0; q < nb; ++q) {
            const uint32_t tq = wave_sum(load_coherent(base + q * kSliceHistWords + kHistBins + lane));
            if (lane == 0) s.above[q] += tq;
          }
          if (lane == 0) {
            s.shv[0] = 1u;
            s.shv[1] = total;
          }
        } else {
          const int g0 = (int)__builtin_ctzll(__ballot(incl >= krem));
          const uint32_t above_g = (uint32_t)__builtin_amdgcn_readlane((int)(incl - gsum), g0);
          const int b = kHistBins - 1 - kWave * g0 - lane;  // lane m: the m-th bin of group g0 from the top
#pragma unroll
          for (int u = 0; u < 8; ++u) cb8[u] = u < nb ? load_coherent(base + u * kSliceHistWords + b) : 0u;
          uint32_t csum = 0u;
#pragma unroll
          for (int u = 0; u < 8; ++u) csum += cb8[u];
          if (nb > 8) csum = sum_over_slices(b);
          const uint32_t inc2 = above_g + wave_inclusive_scan(csum);
          const int m = (int)__builtin_ctzll(__ballot(inc2 >= krem));
          for (int q0 = 0; q0 < nb; q0 += 8) {
            uint32_t tg[8], cb[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const bool ok = q0 + u < nb;
              tg[u] = q0 == 0 ? tg8[u] : (ok ? load_coherent(base + (q0 + u) * kSliceHistWords + kHistBins + lane) : 0u);
              cb[u] = q0 == 0 ? cb8[u] : (ok ? load_coherent(base + (q0 + u) * kSliceHistWords + b) : 0u);
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const uint32_t ab = wave_sum((lane < g0 ? tg[u] : 0u) + (lane < m ? cb[u] : 0u));
              const uint32_t ib = (uint32_t)__builtin_amdgcn_readlane((int)cb[u], m);
              if (lane == 0 && q0 + u < nb) {
                s.above[q0 + u] += ab;
                s.inbin[q0 + u] = ib;
              }
            }
          }
          const uint32_t cm = (uint32_t)__builtin_amdgcn_readlane((int)csum, m);
          const uint32_t im = (uint32_t)__builtin_amdgcn_readlane((int)inc2, m);
          if (lane == 0) {
            s.shv[0] = 0u;
            s.shv[1] = (uint32_t)(kHistBins - 1 - kWave * g0 - m);
            s.shv[2] = krem - (im - cm);
            s.shv[3] = cm;
          }
        }
      }
      __syncthreads();
      const uint32_t state = s.shv[0], b1 = s.shv[1], kr = s.shv[2], n1 = s.shv[3];
      __syncthreads();  // read before the next pass rewrites them
      if (pass + 1 >= kSelMaxPasses || gave_up) {  // never expected: give up with a valid-looking answer
        gave_up = true;
        T = lo;
        need = 0u;
        all_bin = true;
        if (tid < nb) s.inbin[tid] = 0u;
        break;
      }
      if (state == 1) {  // below the window
        krem -= b1;
        hi = lo;
        lo = 1u;
        open = false;
        continue;
      }
      const uint64_t blo = (uint64_t)lo + ((uint64_t)b1 << sh);
      if (open && b1 == (uint32_t)(kHistBins - 1)) {  // past the regular bins
        lo = (uint32_t)blo;
        hi = 1ull << 32;
        continue;
      }
      if (sh == 0) {  // one key value: T, and how many of its keys to take
        T = (uint32_t)blo;
        need = kr;
        if (tid < nb) {
          s.gt[tid] = 0u;
          s.eq[tid] = s.inbin[tid];
        }
        break;
      }
      if (kr == n1) {  // the whole bin is taken
        T = (uint32_t)blo;
        all_bin = true;
        break;
      }
      if (n1 <= (uint32_t)kSelCandMax) {
        // The bin's keys, in index order, from every slice.
        const uint32_t bhi1 = (uint32_t)(blo + ((1ull << sh) - 1u));  // last key value of the bin
        uint32_t off = 0u;
        for (int q = 0; q < part; ++q) off += s.inbin[q];
        uint32_t cnt = 0u;
#pragma unroll
        for (int i = 0; i < kSelPer; ++i) cnt += key[i] >= (uint32_t)blo && key[i] <= bhi1;
        uint32_t w = off + block_exclusive_scan(cnt, s.scan);
        uint32_t* xc = a.xcand + ((int64_t)bh * 2 + (round & 1)) * kSelCandMax * 2;
#pragma unroll
        for (int i = 0; i < kSelPer; ++i)
          if (key[i] >= (uint32_t)blo && key[i] <= bhi1) {
            if (w < (uint32_t)kSelCandMax) {
              store_coherent(xc + 2 * w, key[i]);
              store_coherent(xc + 2 * w + 1, (uint32_t)(j0 + i));
            }
            ++w;
          }
        if (tid < nb) {
          s.gt[tid] = 0u;
          s.eq[tid] = 0u;
        }
        exchange();
        const uint32_t* xr = a.xcand + ((int64_t)bh * 2 + ((round - 1) & 1)) * kSelCandMax * 2;
        if (tid < (int)n1) {
          s.ckey[tid] = load_coherent(xr + 2 * tid);
          s.cidx[tid] = load_coherent(xr + 2 * tid + 1);
        }
        __syncthreads();
        // Candidate t counts the candidates above and equal to its key;
        // those whose key is the kr-th largest publish it.
        uint32_t v = 0u, c_gt = 0u, c_eq = 0u;
        if (tid < (int)n1) {
          v = s.ckey[tid];
          for (int j = 0; j < (int)n1; ++j) {
            const uint32_t c = s.ckey[j];
            c_gt += c > v ? 1u : 0u;
            c_eq += c == v ? 1u : 0u;
          }
          if (c_gt < kr && kr <= c_gt + c_eq) {
            s.shv[4] = v;
            s.shv[5] = kr - c_gt;
          }
        }
        __syncthreads();
        T = s.shv[4];
        need = s.shv[5];
        if (tid < (int)n1) {
          const uint32_t q = s.cidx[tid] / (uint32_t)kSelSlice;
          if (v > T) atomicAdd(&s.gt[q], 1u);
          if (v == T) atomicAdd(&s.eq[q], 1u);
        }
        __syncthreads();
        break;
      }
      // Narrow the window to the bin.
      lo = (uint32_t)blo;
      hi = blo + (1ull << sh);
      open = false;
      krem = kr;
    }
    T_out = T;  // the same in every work-group of the head
    // Each slice's taken keys, this slice's offset among the T-keys, and
    // whether its T-keys are split (some taken, some not).
    if (tid == 0) {
      uint32_t toff = 0u, mine = 0u, split = 0u;
      for (int q = 0; q < nb; ++q) {
        uint32_t t = s.above[q];
        if (all_bin) {
          t += s.inbin[q];
        } else {
          const uint32_t tq = s.eq[q];
          const uint32_t tk = min(need - min(need, toff), tq);
          t += s.gt[q] + tk;
          if (q == part) {
            mine = toff;
            split = tk != 0u && tk != tq;
          }
          toff += tq;
        }
        s.taken[which][q] = t;
      }
      s.shv[7] = mine;
      s.shv[10] = split;
      s.shv[11] = mine < need;  // this slice's T-keys, if any, are taken when not split
    }
    __syncthreads();
    uint32_t mask = 0u;
    if (!all_bin && s.shv[10] == 0u) {
      const bool take_t = s.shv[11] != 0u;  // this slice's T-keys: all taken, or none
#pragma unroll
      for (int i = 0; i < kSelPer; ++i) mask |= ((take_t ? key[i] >= T : key[i] > T) ? 1u : 0u) << i;
    } else if (all_bin) {
#pragma unroll
      for (int i = 0; i < kSelPer; ++i) mask |= (key[i] >= T && key[i] != 0u ? 1u : 0u) << i;
    } else {
      uint32_t nt = 0u;
#pragma unroll
      for (int i = 0; i < kSelPer; ++i) nt += key[i] == T;
      uint32_t rank = s.shv[7] + block_exclusive_scan(nt, s.scan);
#pragma unroll
      for (int i = 0; i < kSelPer; ++i) {
        bool take = key[i] > T;
        if (key[i] == T) {
          take = rank < need;
          ++rank;
        }
        if (take) mask |= 1u << i;
      }
    }
    __syncthreads();  // shv[7] and the scan buffer read before reuse
    return mask;
  };

  uint32_t sel[2] = {0u, 0u};  // bit i: token j0 + i in u_score / u_random
  if (tid < nb) {
    s.taken[0][tid] = 0u;
    s.taken[1][tid] = 0u;
  }
  __syncthreads();
  const uint32_t fs_key = protected_token(js) ? 0u : float_order_key(__uint_as_float(f_smp));
  // The score threshold (every work-group of the head has the same), for
  // leaving u_score out of the draw's sample: tokens whose score key reaches
  // it count as taken (the sample is only a guess).
  uint32_t T1 = 0xFFFFFFFFu;
  if (a.Cp > 0) sel[0] = top_k(fk, (uint32_t)a.Cp, (uint32_t)(L - a.n_protect), 0, fs_key, T1);
  if (a.Cr > 0) {
    // Candidates of the draw: R minus u_score.  (The Gumbel keys are loaded
    // only now: registers are short while the scores are searched.)
    uint32_t gk[kSelPer];
    load_row(grow, gk);
#pragma unroll
    for (int i = 0; i < kSelPer; ++i)
      if (fk[i] == 0u || ((sel[0] >> i) & 1u)) gk[i] = 0u;
    uint32_t T2;
    sel[1] = top_k(gk, (uint32_t)a.Cr, (uint32_t)(L - a.n_protect - a.Cp), 1,
                   (fs_key != 0u && fs_key < T1) ? g_smp : 0u, T2);
  }
  if (gave_up && tid == 0 && a.health) {
    atomicOr(a.health, 8u);
    atomicOr(a.health + 1, 8u);
  }

  // ---- assembly: this slice's kept tokens, listed in LDS, then copied out
  // with coalesced stores at the slice's offset of the keep list
  uint32_t kept = prot | sel[0] | sel[1];
  if (j0 >= L) kept = 0u;
  if (tid == 0) {
    uint32_t base = 0;
    for (int q = 0; q < part; ++q) base += s.prot[q] + s.taken[0][q] + s.taken[1][q];
    s.shv[12] = base;
    s.shv[13] = s.prot[part] + s.taken[0][part] + s.taken[1][part];
  }
  uint32_t o = block_exclusive_scan((uint32_t)__popc(kept), s.scan);
#pragma unroll
  for (int i = 0; i < kSelPer; ++i)
    if ((kept >> i) & 1u) s.list[o++] = (uint32_t)(j0 + i);
  __syncthreads();
  const uint32_t base = s.shv[12], n_here = min(s.shv[13], (uint32_t)kSelSlice);
  int32_t* out = a.keep + (int64_t)bh * a.C;
  for (uint32_t c = tid; c < n_here; c += kSelThreads)
    if (base + c < (uint32_t)a.C) out[base + c] = (int32_t)s.list[c];
}

// Clears the selection's ticket and round counters (a fill kernel rather
// than a memset, so the sequence can be captured in a graph).
__global__ void select_sync_clear_kernel(uint32_t* w, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) w[i] = 0u;
}

hipError_t launch_select(const SelectLaunch& a, hipStream_t stream) {
  const int BH = a.B * a.H;
  if (a.Cr > 0 && !a.keys_ready) {
    dim3 gk((a.L + 1023) / 1024, BH);
    const uint32_t k0 = (uint32_t)(a.seed & 0xFFFFFFFFu), k1 = (uint32_t)(a.seed >> 32);
    // 16-byte rows: every row start 16-byte aligned (the workspace always is).
    const int vec = (a.L % 4 == 0) && ((uintptr_t)a.scores % 16 == 0) && ((uintptr_t)a.keys2 % 16 == 0);
    if (a.sampling == 0)
      hipLaunchKernelGGL(gumbel_keys_kernel<0>, gk, dim3(256), 0, stream, a.scores, a.H, a.L, k0, k1,
                         a.layer, vec, a.keys2);
    else if (a.sampling == 1)
      hipLaunchKernelGGL(gumbel_keys_kernel<1>, gk, dim3(256), 0, stream, a.scores, a.H, a.L, k0, k1,
                         a.layer, vec, a.keys2);
    else
      hipLaunchKernelGGL(gumbel_keys_kernel<2>, gk, dim3(256), 0, stream, a.scores, a.H, a.L, k0, k1,
                         a.layer, vec, a.keys2);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.L <= 8 * kSelThreads) {
    hipLaunchKernelGGL((select_kernel_regs<kSelThreads, 8>), dim3(BH), dim3(kSelThreads), 0, stream, a);
    return hipGetLastError();
  }
  if (a.L <= 16 * kSelThreads) {
    hipLaunchKernelGGL((select_kernel_regs<kSelThreads, 16>), dim3(BH), dim3(kSelThreads), 0, stream, a);
    return hipGetLastError();
  }
  if (a.L <= kRegMaxL) {
    hipLaunchKernelGGL((select_kernel_regs<kSelThreads, kRegKeys>), dim3(BH), dim3(kSelThreads), 0, stream, a);
    return hipGetLastError();
  }
  if (a.nb < 1 || a.nb > kSelMaxSlices || (int64_t)a.nb * kSelSlice < a.L) return hipErrorInvalidValue;
  if (a.zero_sync) {
    const int n = 64 + BH;
    hipLaunchKernelGGL(select_sync_clear_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a.sync, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(select_kernel, dim3(BH * a.nb), dim3(kSelThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace nacl
