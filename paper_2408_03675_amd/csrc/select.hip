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
// work-group each, every thread holding 32 tokens' keys in registers
// (select_kernel_regs, described with it below).  Longer heads are cut into
// slices of kSelSlice tokens, one work-group each, every thread holding
// kSelPer consecutive tokens in registers; the work-groups of a head exchange
// data through the workspace in rounds (publish, count one arrival on the
// head's counter, wait for the other slices), and every work-group takes the
// same decisions from the same published data.
//
// Sliced heads:
// Top-k of one key set (k-th largest key T, and `need`, how many keys equal
// to T belong to the top k; ties go to the lowest indices):
//   1. pivots: the keys of about kSelSamples sampled tokens (every st-th
//      token of the head) give a window [lo, hi] that holds the k-th largest
//      key with high probability (ranks k*m/n -+ a few standard deviations);
//   2. one counting pass: keys above the window and inside it, per slice;
//      each slice also publishes its keys inside the window with their
//      indices (the window is narrow, typically about 1500 tokens);
//   3. if the window holds the k-th key and all its keys were published, an
//      exact radix select over them in LDS gives T and need; a window of one
//      value gives them from the counts; otherwise the window is halved in
//      key space and counted again (a fallback for degenerate pivots).
// The top k is then "key > T, or key == T with a rank among the T-keys,
// in index order, below need": a block scan gives each slice its ranks, and
// every slice knows how many T-keys the slices before it hold.
//
// Assembly: every work-group knows, from the published counts, how many
// tokens each slice keeps, so it writes its kept indices at the right offset
// of the ascending keep list without another round.

#include <type_traits>

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
// Thread t holds the keys of the 32 consecutive tokens 32 t .. 32 t + 31 in
// registers.  Each key set (scores, then Gumbel keys) is staged in LDS by
// direct buffer->LDS loads (contiguous 16-byte pieces per lane) and read
// back as eight 16-byte pieces per thread in the rotated order (q + t) mod 8,
// under which the eight lanes an LDS cycle serves touch distinct banks; so
// register slot i holds token 32 t + ((i + 4 t) mod 32), and a mask over the
// slots is a mask over the thread's tokens rotated by 4 t.  The Gumbel keys
// are loaded into the staging buffer while the scores are searched.
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

struct RegLds {
  alignas(16) uint32_t hist[kHistBins];  // all zero between passes
  uint32_t fixed[kRegMaxL / 32];         // Pi, one bit per token (word t: tokens 32 t ..)
  uint32_t cand[kRegCand];               // keys of the k-th bin (step 3)
  uint32_t pick[2][4];                   // per rank: found, bin, rank within the bin, bin count
  uint32_t scan[2 * kSelWaves];
  uint32_t shv[8];                       // 0-2 ranked result, 4 gather counter, 5 max key, 6 valid samples
};

struct TopK {
  uint32_t T, need, n_eq;
};

__device__ __forceinline__ uint32_t rotr32(uint32_t x, uint32_t r) { return __builtin_amdgcn_alignbit(x, x, r); }
__device__ __forceinline__ uint32_t rotl32(uint32_t x, uint32_t r) { return __builtin_amdgcn_alignbit(x, x, (32u - r) & 31u); }

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
__device__ __forceinline__ uint32_t reg_block_scan(uint32_t v, uint32_t* scan_buf) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t x = wave_inclusive_scan(v);
  if (lane == kWave - 1) scan_buf[wave] = x;
  lds_barrier();
  if (wave == 0) {
    uint32_t t = lane < kSelWaves ? scan_buf[lane] : 0u;
    t = wave_inclusive_scan(t);
    if (lane < kSelWaves) scan_buf[kSelWaves + lane] = t;
  }
  lds_barrier();
  const uint32_t base = wave ? scan_buf[kSelWaves + wave - 1] : 0u;
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
__device__ __forceinline__ void pick_bins(RegLds& s, const uint32_t (&kr)[NRK]) {
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    uint4* own = reinterpret_cast<uint4*>(s.hist + kHistBins - 64 * (lane + 1));
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
        if (lane == 0) s.pick[r][0] = 0u;
        continue;
      }
      const int l0 = (int)__builtin_ctzll(__ballot(incl >= want));
      const uint32_t above = (uint32_t)__builtin_amdgcn_readlane((int)(incl - sum), l0);
      const int b = kHistBins - 1 - 64 * l0 - lane;  // lane m: the m-th bin of lane l0 from the top
      const uint32_t c = s.hist[b];
      const uint32_t inc2 = above + wave_inclusive_scan(c);
      const int m = (int)__builtin_ctzll(__ballot(inc2 >= want));
      if (lane == m) {
        s.pick[r][0] = 1u;
        s.pick[r][1] = (uint32_t)b;
        s.pick[r][2] = want - (inc2 - c);
        s.pick[r][3] = c;
      }
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) lds_zero16(reinterpret_cast<uint32_t*>(own + ((q + lane) & 15)));
  }
  lds_barrier();
}

// The kr-th largest of the keys whose bits at and above `bits` equal those
// of prefix (its lower bits zero; bits == 32: every key), by radix passes of
// 12 bits (the last one narrower) over the bits below; key 0 never counts.
// At least kr keys must match.
template <int NR>
__device__ __forceinline__ TopK radix_rest(const uint32_t (&key)[NR], RegLds& s, uint32_t prefix, int bits,
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
template <int NR>
__device__ __forceinline__ TopK reg_top_k(const uint32_t (&key)[NR], uint32_t k, uint32_t n_valid, RegLds& s) {
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
template <int NR>
__device__ __forceinline__ uint32_t top_members(const uint32_t (&key)[NR], const TopK& r, uint32_t rot,
                                                RegLds& s) {
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
  uint32_t t_tok = rotl32(tie, rot);  // token order
  const uint32_t n = (uint32_t)__popc(t_tok);
  const uint32_t before = reg_block_scan(n, s.scan);
  uint32_t take = min(r.need - min(r.need, before), n);  // need - before, or 0 past the need-th tie
  uint32_t kept_tok = 0u;
  while (take--) {
    const uint32_t low = t_tok & (0u - t_tok);
    kept_tok |= low;
    t_tok ^= low;
  }
  return in | rotr32(kept_tok, rot);
}

__global__ __launch_bounds__(kSelThreads) void select_kernel_regs(SelectLaunch a) {
  __shared__ RegLds s;
  __shared__ uint32_t stage[kRegMaxL];  // one key set of the head, by buffer->LDS loads
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
      for (int r = 0; r < kRegMaxL / (256 * kSelWaves); ++r) {
        const uint32_t t0 = 256u * (uint32_t)(kSelWaves * r + wave);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(stage + t0), 16,
                                                 (t0 + 4u * (uint32_t)lane) * 4u, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int r = 0; r < kRegMaxL / (64 * kSelWaves); ++r) {
        const uint32_t t0 = 64u * (uint32_t)(kSelWaves * r + wave);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(stage + t0), 4,
                                                 (t0 + (uint32_t)lane) * 4u, 0, 0, 0);
      }
    }
  };
  // Thread t's 32 staged words, slot i = token 32 t + ((i + rot) mod 32).
  const uint32_t rot = (4u * (uint32_t)tid) & 31u;
  uint32_t key[kRegKeys];
  auto read_stage = [&]() {
    const uint4* row = reinterpret_cast<const uint4*>(stage + kRegKeys * tid);
#pragma unroll
    for (int q = 0; q < kRegKeys / 4; ++q) {
      const uint4 v = row[(q + tid) & 7];
      key[4 * q] = v.x;
      key[4 * q + 1] = v.y;
      key[4 * q + 2] = v.z;
      key[4 * q + 3] = v.w;
    }
  };

  stage_keys(fsrc, a.Cp > 0 ? L : 0);
  s.fixed[tid] = 0u;
#pragma unroll
  for (int q = 0; q < kHistBins / kSelThreads; ++q) s.hist[q * kSelThreads + tid] = 0u;
  if (tid < 8) s.shv[tid] = 0u;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's loads
  lds_barrier();                                    // everyone's, and the clears
  if (p0 >= 0) lds_or(&s.fixed[p0 >> 5], 1u << (p0 & 31));
  for (int i = pbase + tid + kSelThreads; i < a.P; i += kSelThreads) {
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
  const int nt = L - kRegKeys * tid;
  const uint32_t live_tok = nt >= kRegKeys ? 0xFFFFFFFFu : (nt > 0 ? (1u << nt) - 1u : 0u);
  const uint32_t live = rotr32(live_tok, rot);
  const uint32_t mp = rotr32(s.fixed[tid], rot);
  uint32_t ms = 0u, mr = 0u;

  // u_score: top-Cp of F over R = [0, L) \ Pi.
  if (a.Cp > 0) {
#pragma unroll
    for (int i = 0; i < kRegKeys; ++i)
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
    for (int i = 0; i < kRegKeys; ++i)
      if (!((cand >> i) & 1u)) key[i] = 0u;
    const TopK r = reg_top_k(key, (uint32_t)a.Cr, (uint32_t)(L - a.n_protect - a.Cp), s);
    mr = top_members(key, r, rot, s);
  }

  // keep = Pi | u_score | u_random in index order: C entries by construction
  // (the bound only guards the write).  The list is assembled in the staging
  // buffer (every thread has read the Gumbel keys from it before the last
  // selection's barriers), then copied out with coalesced stores.
  uint32_t kept = rotl32(mp | ms | mr, rot);
  if (a.Cr == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the zero loads into the buffer
  uint32_t o = reg_block_scan((uint32_t)__popc(kept), s.scan);  // (its barriers: everyone's)
  while (kept) {
    const int b = __builtin_ctz(kept);
    if (o < (uint32_t)a.C) stage[o] = (uint32_t)(kRegKeys * tid + b);
    ++o;
    kept &= kept - 1u;
  }
  lds_barrier();
  int32_t* out = a.keep + (int64_t)bh * a.C;
  for (int c = tid; c < a.C; c += kSelThreads) out[c] = (int32_t)stage[c];
}

// ===========================================================================
// Longer heads: slices of kSelSlice tokens, one work-group each.

// Exclusive prefix of v over the work-group in thread order, and the total.
__device__ uint32_t block_scan_total(uint32_t v, uint32_t* scan_buf, uint32_t& total) {
  const uint32_t ex = block_exclusive_scan(v, scan_buf);
  total = scan_buf[2 * kSelWaves - 1];
  __syncthreads();  // every thread has read the total before the buffer is reused
  return ex;
}

struct SelLds {
  uint32_t a[kSelCapTotal];     // sampled keys, then window keys
  uint32_t b[kSelCapTotal];     // window token indices
  uint32_t smp[2][kSelSamples]; // sampled keys of a head held by one slice
  uint32_t hist[256];
  uint32_t scan[2 * kSelWaves];
  uint32_t shv[16];
  uint32_t cnt_gt[kSelMaxSlices];   // per slice: keys above the window (this round)
  uint32_t cnt_in[kSelMaxSlices];   // per slice: keys inside the window
  uint32_t off_in[kSelMaxSlices];   // prefix of cnt_in
  uint32_t gt_t[kSelMaxSlices];     // per slice: keys above T
  uint32_t ties[kSelMaxSlices];     // per slice: keys equal to T
  uint32_t taken[2][kSelMaxSlices]; // per slice: tokens of u_score / u_random
  uint32_t prot[kSelMaxSlices];     // per slice: protected proxies
};

// hist[bin] += 1 for every lane with `valid`.  The keys cluster (scores
// share a few exponents) and same-address atomics of one instruction are
// serialised, so the most common bins of the wave are counted first with one
// atomic each (up to three of them, the bins of the first pending lanes); the
// lanes left over add one each.
__device__ __forceinline__ void wave_count(uint32_t* hist, uint32_t bin, bool valid) {
  const int lane = threadIdx.x & 63;
  uint64_t todo = __ballot(valid);
#pragma unroll
  for (int r = 0; r < 3; ++r) {
    if (!todo) return;
    const int leader = __builtin_ctzll(todo);
    const uint32_t b0 = __builtin_amdgcn_readlane(bin, leader);
    const uint64_t m = __ballot(valid && bin == b0) & todo;
    if (lane == leader) atomicAdd(&hist[b0], (uint32_t)__popcll(m));
    todo &= ~m;
  }
  if ((todo >> lane) & 1u) atomicAdd(&hist[bin], 1u);
}

// The k-th largest (1 <= k <= n) of the n keys in s.a, by four 8-bit radix
// passes over LDS; returns T and sets need = how many keys equal to T the
// top k holds.
__device__ uint32_t lds_kth(SelLds& s, int n, uint32_t k, uint32_t& need) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint32_t prefix = 0u, pmask = 0u, kr = k;
#pragma unroll 1
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (tid < 256) s.hist[tid] = 0u;
    __syncthreads();
    for (int i0 = 0; i0 < n; i0 += kSelThreads) {
      const int i = i0 + tid;
      const uint32_t v = i < n ? s.a[i] : 0u;
      wave_count(s.hist, (v >> shift) & 255u, i < n && (v & pmask) == prefix);
    }
    __syncthreads();
    if (wave == 0) {
      // lane l holds bins 255 - 4l down to 252 - 4l (descending key order)
      uint32_t c[4], sum = 0u;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c[q] = s.hist[255 - 4 * lane - q];
        sum += c[q];
      }
      const uint32_t incl = wave_inclusive_scan(sum);
      const uint32_t excl = incl - sum;
      if (excl < kr && kr <= incl) {
        uint32_t cum = excl;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (cum < kr && kr <= cum + c[q]) {
            s.shv[0] = (uint32_t)(255 - 4 * lane - q);
            s.shv[1] = kr - cum;
          }
          cum += c[q];
        }
      }
    }
    __syncthreads();
    prefix |= s.shv[0] << shift;
    pmask |= 255u << shift;
    kr = s.shv[1];
    __syncthreads();
  }
  need = kr;
  return prefix;
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectLaunch a) {
  __shared__ SelLds s;
  const int tid = threadIdx.x;
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
  const int b = bh / a.H, h = bh % a.H;
  const int st = select_sample_stride(L);
  const int m_all = (L + st - 1) / st;                 // sampled tokens of the head
  uint32_t* counter = a.sync + 64 + bh;
  uint32_t* samples = a.samples + (int64_t)bh * 2 * a.ms;
  const int j0 = part * kSelSlice + tid * kSelPer;    // this thread's first token
  const int nrem = L - j0;                             // tokens of the head from j0 on
  const int pbase = a.P - a.n_protect;
  int round = 0;

  // Arrival on the head's counter, then wait for every slice of the head.
  auto exchange = [&]() {
    wait_stores();
    __syncthreads();
    if (tid == 0 && nb > 1) {
      atomicAdd(counter, 1u);
      const uint32_t target = (uint32_t)nb * (uint32_t)(round + 1);
      uint32_t spins = 0;
      while (load_coherent(counter) < target) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins > kSelSpinLimit) {
          if (a.health) {
            atomicOr(a.health, 8u);
            atomicOr(a.health + 1, 8u);
          }
          break;
        }
      }
    }
    ++round;
    __syncthreads();
  };

  // ---- this thread's tokens: scores, Gumbel keys, protected marks
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
  const uint32_t* gsrc = a.keys2 + (int64_t)bh * L;
  load_row(reinterpret_cast<const uint32_t*>(a.scores) + (int64_t)bh * L, fk);
  // The protected positions (ascending, at most NACL_MAX_P) staged in LDS.
  const int np = a.n_protect;
  uint32_t* ppos = s.b;
  for (int i = tid; i < np; i += kSelThreads) ppos[i] = (uint32_t)a.pos[pbase + i];
  __syncthreads();
  auto first_at_least = [&](int x) {  // first staged position >= x
    int lo = 0, hi = np;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if ((int)ppos[mid] < x) lo = mid + 1;
      else hi = mid;
    }
    return lo;
  };
  uint32_t prot = 0u;  // bit i: token j0 + i is protected
  if (np > 0 && j0 < L)
    for (int i = first_at_least(j0); i < np && (int)ppos[i] < j0 + kSelPer; ++i) prot |= 1u << (ppos[i] - j0);
#pragma unroll
  for (int i = 0; i < kSelPer; ++i) {
    const bool cand = i < nrem && !((prot >> i) & 1u);
    fk[i] = cand ? float_order_key(__uint_as_float(fk[i])) : 0u;
  }
  // Protected proxies per slice (for the assembly offsets).
  if (tid < nb) s.prot[tid] = (uint32_t)(first_at_least((tid + 1) * kSelSlice) - first_at_least(tid * kSelSlice));
  __syncthreads();  // the staged positions are dead from here on

  // ---- round 0: sampled (score key, Gumbel key) pairs
  {
    int nxt = (j0 + st - 1) / st * st, slot = nxt / st;  // first sampled token >= j0
    int di = nxt - j0;                                    // its offset in this thread's run
#pragma unroll
    for (int i = 0; i < kSelPer; ++i)
      if (i == di && i < nrem) {
        const uint32_t g = a.Cr > 0 && fk[i] != 0u ? gsrc[nxt] : 0u;
        if (nb == 1) {  // one slice: the sample stays in LDS
          s.smp[0][slot] = fk[i];
          s.smp[1][slot] = g;
        } else {
          store_coherent(samples + slot, fk[i]);
          store_coherent(samples + a.ms + slot, g);
        }
        nxt += st;
        di += st;
        ++slot;
      }
  }
  if (nb == 1) __syncthreads();
  else exchange();

  uint32_t sel[2] = {0u, 0u};  // bit i: token j0 + i in u_score / u_random
  // Top-k of key[] (this thread's tokens; 0 = not a candidate) among n
  // candidates of the head; `which` indexes taken[].  samp(x) maps a sampled
  // pair index to its key for this selection (0 = not a candidate).
  auto top_k = [&](const uint32_t (&key)[kSelPer], uint32_t k, uint32_t n, int which, uint32_t& T_out,
                   auto&& samp) -> uint32_t {
    // Pivots: wave 0 sorts the sampled keys (zero past the sample and for
    // tokens that are not candidates) in registers.
    if (tid < kWave) {
      constexpr int R = kSelSamples / kWave;
      uint32_t sv[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int x = tid * R + r;
        sv[r] = x < m_all ? samp(x) : 0u;
      }
      uint32_t nz = 0;
#pragma unroll
      for (int r = 0; r < R; ++r) nz += sv[r] != 0u;
      wave_sort_desc(sv);
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) nz += (uint32_t)__shfl_xor((int)nz, off);
#pragma unroll
      for (int r = 0; r < R; ++r) s.a[tid * R + r] = sv[r];
      if (tid == 0) s.shv[13] = nz;
    }
    __syncthreads();
    const uint32_t m = s.shv[13];
    uint32_t plo = 1u, phi = 0xFFFFFFFFu;
    if (m > 0) {
      // rank of the k-th key among the sampled candidates, give or take
      // three standard deviations, within what the exact step can take
      const double r = (double)k * (double)m / (double)n;
      const double sd = sqrt(r * (1.0 - r / (double)m) + 1.0);
      const double per = (double)n / (double)m;  // candidates per sampled one
      const int delta = (int)fmin(ceil(3.0 * sd) + 2.0, fmax(1.0, floor(0.45 * kSelCapTotal / per)));
      const long hr = (long)floor(r) - delta, lr = (long)ceil(r) + delta;
      if (hr >= 1) phi = s.a[hr - 1];
      if (lr <= (long)m) plo = s.a[lr - 1];
    }
    __syncthreads();
    // Window search: T lies in [lo, hi], `above` keys lie above hi.
    uint32_t lo = 1u, hi = 0xFFFFFFFFu, above = 0u, T = 0u, need = 0u;
    bool done = false;
    for (int it = 0; !done; ++it) {
      const int parity = round & 1;
      uint32_t* rc = a.rounds + ((int64_t)bh * 2 + parity) * nb * 2;
      uint32_t* mid = a.mid + (((int64_t)bh * 2 + parity) * nb + part) * a.cap_b * 2;
      // One scan of both counts packed in 16-bit halves (a slice holds at
      // most kSelSlice = 2^15 tokens).
      uint32_t gt = 0, in = 0;
#pragma unroll
      for (int i = 0; i < kSelPer; ++i) {
        gt += key[i] > phi;
        in += key[i] >= plo && key[i] <= phi;
      }
      uint32_t tot;
      const uint32_t ex = block_scan_total(gt | (in << 16), s.scan, tot);
      const uint32_t gt_tot = tot & 0xFFFFu, in_tot = tot >> 16;
      uint32_t w = ex >> 16;
      if (nb == 1) {
        // One slice: the window's keys go straight to LDS.
        if (in_tot <= (uint32_t)kSelCapTotal) {
#pragma unroll
          for (int i = 0; i < kSelPer; ++i)
            if (key[i] >= plo && key[i] <= phi) {
              s.a[w] = key[i];
              s.b[w] = (uint32_t)(j0 + i);
              ++w;
            }
        }
        if (tid == 0) {
          s.cnt_gt[0] = gt_tot;
          s.cnt_in[0] = in_tot;
        }
      } else {
        if (in_tot <= (uint32_t)a.cap_b) {
#pragma unroll
          for (int i = 0; i < kSelPer; ++i)
            if (key[i] >= plo && key[i] <= phi) {
              store_coherent(mid + 2 * w, key[i]);
              store_coherent(mid + 2 * w + 1, (uint32_t)(j0 + i));
              ++w;
            }
        }
        if (tid == 0) {
          store_coherent(rc + 2 * part, gt_tot);
          store_coherent(rc + 2 * part + 1, in_tot);
        }
        exchange();
        if (tid < nb) {
          s.cnt_gt[tid] = load_coherent(rc + 2 * tid);
          s.cnt_in[tid] = load_coherent(rc + 2 * tid + 1);
        }
      }
      __syncthreads();
      if (tid == 0) {
        uint32_t G = 0, I = 0, full = 1, off = 0;
        for (int q = 0; q < nb; ++q) {
          G += s.cnt_gt[q];
          I += s.cnt_in[q];
          full &= s.cnt_in[q] <= (uint32_t)(nb == 1 ? kSelCapTotal : a.cap_b);
          s.off_in[q] = off;
          off += s.cnt_in[q];
        }
        // state: 0 continue, 1 resolved by one value, 2 resolve from the window's keys
        uint32_t state = 0;
        if (k <= G) {
          lo = phi + 1u;
        } else if (k > G + I) {
          hi = plo - 1u;
          above = G + I;
        } else {
          lo = plo;
          hi = phi;
          above = G;
          if (plo == phi) state = 1;
          else if (full && I <= (uint32_t)kSelCapTotal) state = 2;
        }
        if (state == 0 && it + 1 >= kSelMaxRounds) {
          if (a.health) {
            atomicOr(a.health, 8u);
            atomicOr(a.health + 1, 8u);
          }
          state = 1;  // give up: take the window's low end (never expected)
          plo = phi = lo;
        }
        s.shv[2] = state;
        s.shv[3] = G;
        s.shv[4] = I;
        s.shv[5] = lo;
        s.shv[6] = hi;
        s.shv[7] = above;
        s.shv[8] = plo;
        s.shv[9] = phi;
      }
      __syncthreads();
      const uint32_t state = s.shv[2], G = s.shv[3], I = s.shv[4];
      lo = s.shv[5];
      hi = s.shv[6];
      above = s.shv[7];
      if (state == 1) {
        T = s.shv[8];
        need = k - G;
        if (tid < nb) {
          s.gt_t[tid] = s.cnt_gt[tid];
          s.ties[tid] = s.cnt_in[tid];
        }
        done = true;
      } else if (state == 2) {
        // Every slice's window keys into LDS, then the exact step.
        // (four entries per thread in flight at a time; one slice wrote
        // them to LDS already)
        for (int e0 = 0; nb > 1 && e0 < (int)I; e0 += 4 * kSelThreads) {
          constexpr int kU = 4;
          uint32_t ka[kU], kb[kU];
#pragma unroll
          for (int u = 0; u < kU; ++u) {
            const int e = e0 + tid + u * kSelThreads;
            ka[u] = kb[u] = 0u;
            if (e < (int)I) {
              int q = 0;
              while (q + 1 < nb && s.off_in[q + 1] <= (uint32_t)e) ++q;
              const uint32_t* src = a.mid + (((int64_t)bh * 2 + parity) * nb + q) * a.cap_b * 2 +
                                    2 * (e - (int)s.off_in[q]);
              ka[u] = load_coherent(src);
              kb[u] = load_coherent(src + 1);
            }
          }
#pragma unroll
          for (int u = 0; u < kU; ++u) {
            const int e = e0 + tid + u * kSelThreads;
            if (e < (int)I) {
              s.a[e] = ka[u];
              s.b[e] = kb[u];
            }
          }
        }
        if (tid < nb) {
          s.gt_t[tid] = s.cnt_gt[tid];
          s.ties[tid] = 0u;
        }
        __syncthreads();
        T = lds_kth(s, (int)I, k - G, need);
        for (int e0 = 0; e0 < (int)I; e0 += kSelThreads) {
          const int e = e0 + tid;
          const uint32_t v = e < (int)I ? s.a[e] : 0u;
          const uint32_t q = e < (int)I ? s.b[e] / (uint32_t)kSelSlice : 0u;
          wave_count(s.gt_t, q, e < (int)I && v > T);
          wave_count(s.ties, q, e < (int)I && v == T);
        }
        done = true;
      } else {
        // Halve the window in key space: count [mid, hi] next.
        plo = lo + ((hi - lo) >> 1) + (hi > lo ? 1u : 0u);
        phi = hi;
      }
      __syncthreads();
    }
      // Tokens each slice takes, and this slice's tie offset.
    if (tid == 0) {
      uint32_t toff = 0, mine = 0;
      for (int q = 0; q < nb; ++q) {
        const uint32_t tq = s.ties[q];
        const uint32_t take = need > toff ? min(need - toff, tq) : 0u;
        s.taken[which][q] = s.gt_t[q] + take;
        if (q == part) mine = toff;
        toff += tq;
      }
      s.shv[10] = mine;
    }
    __syncthreads();
    const uint32_t tie_off = s.shv[10];
    T_out = T;
    uint32_t nt = 0;
#pragma unroll
    for (int i = 0; i < kSelPer; ++i) nt += key[i] == T;
    uint32_t tt;
    uint32_t rank = tie_off + block_scan_total(nt, s.scan, tt);
    uint32_t mask = 0u;
#pragma unroll
    for (int i = 0; i < kSelPer; ++i) {
      bool take = key[i] > T;
      if (key[i] == T) {
        take = rank < need;
        ++rank;
      }
      if (take) mask |= 1u << i;
    }
    return mask;
  };

  if (tid < nb) {
    s.taken[0][tid] = 0u;
    s.taken[1][tid] = 0u;
  }
  __syncthreads();
  const uint32_t n1 = (uint32_t)(L - a.n_protect);
  uint32_t T1 = 0xFFFFFFFFu, T2 = 0u;
  if (a.Cp > 0) {
    sel[0] = top_k(fk, (uint32_t)a.Cp, n1, 0, T1,
                   [&](int x) { return nb == 1 ? s.smp[0][x] : load_coherent(samples + x); });
  }
  if (a.Cr > 0) {
    // Candidates of the draw: R minus u_score; their Gumbel keys are loaded
    // only now, when the score keys die.
    uint32_t gk[kSelPer];
    load_row(gsrc, gk);
#pragma unroll
    for (int i = 0; i < kSelPer; ++i)
      if (fk[i] == 0u || ((sel[0] >> i) & 1u)) gk[i] = 0u;
    // Sampled tokens already in u_score are left out of the pivots (ties at
    // the score threshold counted as taken; the pivots are only a guess).
    sel[1] = top_k(gk, (uint32_t)a.Cr, n1 - (uint32_t)a.Cp, 1, T2, [&](int x) {
      const uint32_t f = nb == 1 ? s.smp[0][x] : load_coherent(samples + x);
      const uint32_t g = nb == 1 ? s.smp[1][x] : load_coherent(samples + a.ms + x);
      return (f != 0u && f < T1) ? g : 0u;
    });
  }

  // ---- assembly: this slice's kept tokens at their offset of the keep list
  uint32_t kept = prot | sel[0] | sel[1];
  if (j0 >= L) kept = 0u;
  if (tid == 0) {
    uint32_t base = 0;
    for (int q = 0; q < part; ++q) base += s.prot[q] + s.taken[0][q] + s.taken[1][q];
    s.shv[12] = base;
  }
  __syncthreads();
  uint32_t tot;
  uint32_t o = s.shv[12] + block_scan_total((uint32_t)__popc(kept), s.scan, tot);
  int32_t* out = a.keep + (int64_t)bh * a.C;
#pragma unroll
  for (int i = 0; i < kSelPer; ++i)
    if ((kept >> i) & 1u) {
      if (o < (uint32_t)a.C) out[o] = j0 + i;
      ++o;
    }
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
  if (a.L <= kRegMaxL) {
    hipLaunchKernelGGL(select_kernel_regs, dim3(BH), dim3(kSelThreads), 0, stream, a);
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
