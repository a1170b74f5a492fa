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
// token that is not a candidate).  A head of L tokens is cut into slices of
// kSelSlice tokens, one work-group each, every thread holding kSelPer
// consecutive tokens in registers; the work-groups of a head exchange data
// through the workspace in rounds (publish, count one arrival on the head's
// counter, wait for the other slices), and every work-group takes the same
// decisions from the same published data.
//
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
// Heads of up to kRegMaxL tokens: one work-group per head, keys in registers.
//
// Both top-k searches are exact radix selects over the order-preserving keys
// (12-, 12- and 8-bit digits, most significant first): each digit pass builds
// a histogram of the keys that still match the chosen prefix and picks the
// digit where the count from the top reaches k.  That yields the k-th largest
// key T and how many keys equal to T to take; a block-wide ordered scan then
// hands those to the lowest indices.  Set membership lives in LDS bitmaps, one
// bit per token.

struct SelScratch {
  uint32_t* hist;   // kHistBins, all zero between radix passes
  uint32_t* scan;   // 2 * kSelWaves
  uint32_t* shv;    // 3: radix pick results
};

// Radix select digits, most significant first: 12 + 12 + 8 bits.  The wide
// first digit spreads even tightly clustered keys (scores within a few
// binades) over many counters, so the shared histogram's atomics rarely
// collide; later passes only count keys that match the chosen prefix.
constexpr int kHistBins = 4096;
constexpr int kDigitShift[3] = {20, 8, 0};
constexpr int kDigitBits[3] = {12, 12, 8};

// After a histogram pass over the digit at `shift`: the digit at which the
// count from the top reaches kr, appended to prefix; kr becomes the rank
// within that digit's keys and n_eq their number.  Thread t owns bins
// nbins-1-per*t down to nbins-per-per*t and zeroes them once read, so the
// histogram is all zero again for the next pass.
__device__ void radix_pick(int shift, int nbins, const SelScratch& s, uint32_t& prefix, uint32_t& kr,
                           uint32_t& n_eq) {
  const int tid = threadIdx.x;
  const int per = (nbins + kSelThreads - 1) / kSelThreads;  // 4 or 1
  uint32_t c[4] = {0u, 0u, 0u, 0u}, local = 0u;
#pragma unroll
  for (int qq = 0; qq < 4; ++qq) {
    const int b = nbins - 1 - per * tid - qq;
    if (qq < per && b >= 0) {
      c[qq] = s.hist[b];
      s.hist[b] = 0u;
    }
    local += c[qq];
  }
  const uint32_t excl = block_exclusive_scan(local, s.scan);
  if (excl < kr && kr <= excl + local) {
    uint32_t cum = excl;
    for (int qq = 0; qq < per; ++qq) {
      if (cum + c[qq] >= kr) {
        s.shv[0] = prefix | ((uint32_t)(nbins - 1 - per * tid - qq) << shift);
        s.shv[1] = kr - cum;
        s.shv[2] = c[qq];
        break;
      }
      cum += c[qq];
    }
  }
  // The next write of shv follows the next pass's histogram barrier, which
  // every thread reaches only after reading these values.
  __syncthreads();
  prefix = s.shv[0];
  kr = s.shv[1];
  n_eq = s.shv[2];
}

// k-th largest key T (1 <= k <= number of keys), the number `need` of keys
// equal to T that belong to the top k, and the number n_eq of keys equal to T.
// get(j) reads key j.  A key of 0 marks an excluded token and is never
// counted: the first pass skips it, and later prefixes never match it (an
// order key below 2^20 would be a NaN, so every real key has a nonzero
// first digit).
template <class Get>
__device__ void radix_select(const Get& get, int L, uint32_t k, const SelScratch& s, uint32_t& T,
                             uint32_t& need, uint32_t& n_eq) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0u, kr = k;
#pragma unroll
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = kDigitShift[pass];
    const uint32_t dmask = (1u << kDigitBits[pass]) - 1u;
    const uint32_t hm = pass == 0 ? 0u : (0xFFFFFFFFu << (shift + kDigitBits[pass]));
    // Eight keys per thread in flight before their counter updates.
    for (int j0 = tid; j0 < L; j0 += 8 * kSelThreads) {
      uint32_t kv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u * kSelThreads;
        kv[u] = j < L ? get(j) : 0u;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (pass == 0 ? kv[u] != 0u : ((kv[u] ^ prefix) & hm) == 0u)
          atomicAdd(&s.hist[(kv[u] >> shift) & dmask], 1u);
    }
    __syncthreads();
    radix_pick(shift, 1 << kDigitBits[pass], s, prefix, kr, n_eq);
  }
  T = prefix;
  need = kr;
}

// The same over keys held in registers: key[i] belongs to token
// i * kSelThreads + threadIdx.x (0 past the end of the head or excluded).
template <int NR>
__device__ __forceinline__ void radix_select_regs(const uint32_t (&key)[NR], uint32_t k, const SelScratch& s,
                                                  uint32_t& T, uint32_t& need, uint32_t& n_eq) {
  uint32_t prefix = 0u, kr = k;
#pragma unroll
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = kDigitShift[pass];
    const uint32_t dmask = (1u << kDigitBits[pass]) - 1u;
    const uint32_t hm = pass == 0 ? 0u : (0xFFFFFFFFu << (shift + kDigitBits[pass]));
#pragma unroll
    for (int i = 0; i < NR; ++i)
      if (pass == 0 ? key[i] != 0u : ((key[i] ^ prefix) & hm) == 0u)
        atomicAdd(&s.hist[(key[i] >> shift) & dmask], 1u);
    __syncthreads();
    radix_pick(shift, 1 << kDigitBits[pass], s, prefix, kr, n_eq);
  }
  T = prefix;
  need = kr;
}

// Sets, in out_bits, the bit of every token with key >= T (T > 0): the top k
// when every key equal to T belongs to it.  Each wave covers 64 consecutive
// tokens per step; lanes 0 and 32 OR the two words of the ballot into the
// bitmap with LDS atomics that return nothing (no wait on the old word), and
// the four steps of an iteration keep their loads and updates independent.
template <class Get>
__device__ void mark_at_least(const Get& get, int L, uint32_t T, uint32_t* out_bits) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int b0 = wave * 64; b0 < L; b0 += 4 * kSelThreads) {
    bool take[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = b0 + u * kSelThreads + lane;
      take[u] = j < L && get(j) >= T;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int base = b0 + u * kSelThreads;
      const uint64_t m = __ballot(take[u]);
      const int word = (base >> 5) + (lane >> 5);
      if ((lane & 31) == 0 && base + (lane & 32) < L) {
        const uint32_t bits = (lane & 32) ? (uint32_t)(m >> 32) : (uint32_t)m;
        if (bits) atomicOr(&out_bits[word], bits);
      }
    }
  }
  __syncthreads();
}

// The same over keys in registers (same token mapping as radix_select_regs).
template <int NR>
__device__ __forceinline__ void mark_at_least_regs(const uint32_t (&key)[NR], int L, uint32_t T, uint32_t* out_bits) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    const int base = i * kSelThreads + wave * 64;
    const uint64_t m = __ballot(key[i] >= T);
    if ((lane & 31) == 0 && base + (lane & 32) < L) {
      const uint32_t bits = (lane & 32) ? (uint32_t)(m >> 32) : (uint32_t)m;
      if (bits) atomicOr(&out_bits[(base >> 5) + (lane >> 5)], bits);
    }
  }
  __syncthreads();
}

// Sets, in out_bits, the bit of every token with key > T and of the first
// `need` tokens (in index order) with key == T.  Thread t owns bitmap words
// [t * seg_words, (t + 1) * seg_words).
template <class Get>
__device__ void mark_top(const Get& get, int L, int nwords, int seg_words, uint32_t T, uint32_t need,
                         uint32_t* out_bits, uint32_t* scan_buf) {
  const int w0 = threadIdx.x * seg_words;
  const int w1 = min(w0 + seg_words, nwords);
  uint32_t ties = 0;
  for (int w = w0; w < w1; ++w)
    for (int bit = 0; bit < 32; ++bit) {
      const int j = w * 32 + bit;
      if (j < L && get(j) == T) ++ties;
    }
  uint32_t rank = block_exclusive_scan(ties, scan_buf);
  for (int w = w0; w < w1; ++w) {
    uint32_t word = 0;
    for (int bit = 0; bit < 32; ++bit) {
      const int j = w * 32 + bit;
      if (j < L) {
        const uint32_t key = get(j);
        bool take = key > T;
        if (key == T) {
          take = rank < need;
          ++rank;
        }
        if (take) word |= 1u << bit;
      }
    }
    out_bits[w] |= word;
  }
  __syncthreads();
}

// The top k of get() into out_bits: ballot marking when every key equal to
// the k-th largest is kept, the ordered tie scan otherwise.
template <class Get>
__device__ void select_top(const Get& get, int L, int nwords, int seg_words, uint32_t k,
                           const SelScratch& s, uint32_t* out_bits) {
  uint32_t T, need, n_eq;
  radix_select(get, L, k, s, T, need, n_eq);
  if (need == n_eq) mark_at_least(get, L, T, out_bits);
  else mark_top(get, L, nwords, seg_words, T, need, out_bits, s.scan);
}

// keep = the set bits of a | b in ascending order, C of them: ranks by an
// ordered scan of the bitmap words (thread t owns words [t * seg_words,
// (t + 1) * seg_words)), the list assembled in `list` (LDS, then copied out
// with coalesced stores, or keep itself).
__device__ void assemble_keep(const uint32_t* a_bits, const uint32_t* b_bits, int nwords, int seg_words, int C,
                              const SelScratch& s, int32_t* list, int32_t* keep) {
  const int tid = threadIdx.x;
  const int w0 = tid * seg_words;
  const int w1 = min(w0 + seg_words, nwords);
  uint32_t cnt = 0;
  for (int w = w0; w < w1; ++w) cnt += __popc(a_bits[w] | b_bits[w]);
  uint32_t out = block_exclusive_scan(cnt, s.scan);
  for (int w = w0; w < w1; ++w) {
    uint32_t bits = a_bits[w] | b_bits[w];
    while (bits) {
      const int bit = __ffs(bits) - 1;
      if (out < (uint32_t)C) list[out] = w * 32 + bit;  // |keep| == C by construction
      ++out;
      bits &= bits - 1;
    }
  }
  if (list != keep) {
    __syncthreads();
    for (int c = tid; c < C; c += kSelThreads) keep[c] = list[c];
  }
}

// Heads of up to kRegMaxL tokens: every thread holds the scores and Gumbel
// keys of tokens tid + i * kSelThreads (i < kRegKeys) in registers, both
// loaded at the start so the Gumbel keys arrive while the top-Cp search
// runs.  Radix passes and ballot marking then touch LDS only for the
// histogram and the bitmaps.  LDS: L words (the keys for the ordered tie
// scan, then the keep list), two bitmaps, the histogram.
constexpr int kRegKeys = 32;
constexpr int kRegMaxL = kRegKeys * kSelThreads;
static_assert(kRegMaxL == kSelRegMaxL, "register selection length");

// The top k of the register keys into out_bits; returns the k-th largest
// key T when the top k are exactly the keys >= T (then a token's membership
// is a register compare), else 0 (ties at T split by index).
template <int NR>
__device__ __forceinline__ uint32_t top_regs(const uint32_t (&key)[NR], int L, uint32_t k, const SelScratch& s,
                                             uint32_t* keys_lds, uint32_t* out_bits) {
  uint32_t T, need, n_eq;
  radix_select_regs(key, k, s, T, need, n_eq);
  if (need == n_eq) {
    mark_at_least_regs(key, L, T, out_bits);
    return T;
  } else {
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const int j = i * kSelThreads + (int)threadIdx.x;
      if (j < L) keys_lds[j] = key[i];
    }
    __syncthreads();
    mark_top([&](int j) { return keys_lds[j]; }, L, (L + 31) / 32, 1, T, need, out_bits, s.scan);
    return 0u;
  }
}

__global__ __launch_bounds__(kSelThreads) void select_kernel_regs(SelectLaunch a) {
  extern __shared__ uint32_t smem[];
  const int L = a.L;
  const int nwords = (L + 31) / 32;  // <= kSelThreads
  uint32_t* keys_lds = smem;
  uint32_t* fixed = smem + L;        // Pi, then Pi | u_score
  uint32_t* rnd = fixed + nwords;    // u_random
  SelScratch s;
  s.hist = rnd + nwords;
  s.scan = s.hist + kHistBins;
  s.shv = s.scan + 2 * kSelWaves;

  const int tid = threadIdx.x;
  const int bh = blockIdx.x;
  const uint32_t* fbits = reinterpret_cast<const uint32_t*>(a.scores) + (int64_t)bh * L;
  const uint32_t* gsrc = a.keys2 + (int64_t)bh * L;

  // The first protected position is loaded ahead of the keys, so that using
  // it does not wait for them.
  const int pbase = a.P - a.n_protect;
  const int p0 = pbase + tid < a.P ? a.pos[pbase + tid] : -1;

  // Past the end of the head the loads repeat the last token (masked below),
  // so every load is unconditional and all of them are in flight at once.
  uint32_t fk[kRegKeys], gk[kRegKeys];
  if (a.Cp > 0) {
#pragma unroll
    for (int i = 0; i < kRegKeys; ++i) fk[i] = fbits[min(i * kSelThreads + tid, L - 1)];
  }
  if (a.Cr > 0) {
#pragma unroll
    for (int i = 0; i < kRegKeys; ++i) gk[i] = gsrc[min(i * kSelThreads + tid, L - 1)];
  }

  if (tid < nwords) {
    fixed[tid] = 0u;
    rnd[tid] = 0u;
  }
  for (int i = tid; i < kHistBins; i += kSelThreads) s.hist[i] = 0u;
  __syncthreads();
  if (p0 >= 0) atomicOr(&fixed[p0 >> 5], 1u << (p0 & 31));
  for (int i = pbase + tid + kSelThreads; i < a.P; i += kSelThreads) {
    const int j = a.pos[i];
    atomicOr(&fixed[j >> 5], 1u << (j & 31));
  }
  __syncthreads();
  auto is_fixed = [&](int j) -> bool { return ((fixed[j >> 5] >> (j & 31)) & 1u) != 0u; };

  // u_score: top-Cp of F over R = [0, L) \ Pi, marked into `fixed`.
  uint32_t T1 = 0u;
  if (a.Cp > 0) {
#pragma unroll
    for (int i = 0; i < kRegKeys; ++i) {
      const int j = i * kSelThreads + tid;
      fk[i] = (j < L && !is_fixed(j)) ? float_order_key(__uint_as_float(fk[i])) : 0u;
    }
    T1 = top_regs(fk, L, (uint32_t)a.Cp, s, keys_lds, fixed);
  }

  // u_random: top-Cr of the Gumbel keys over R \ u_score.  Excluded are the
  // tokens past the end, Pi (score key 0) and u_score (score key >= T1)
  // when u_score is exactly the keys >= T1; otherwise the bitmap says.
  if (a.Cr > 0) {
    if (T1) {
#pragma unroll
      for (int i = 0; i < kRegKeys; ++i)
        if (fk[i] == 0u || fk[i] >= T1) gk[i] = 0u;
    } else {
#pragma unroll
      for (int i = 0; i < kRegKeys; ++i) {
        const int j = i * kSelThreads + tid;
        if (j >= L || is_fixed(j)) gk[i] = 0u;
      }
    }
    top_regs(gk, L, (uint32_t)a.Cr, s, keys_lds, rnd);
  }

  assemble_keep(fixed, rnd, nwords, 1, a.C, s, reinterpret_cast<int32_t*>(keys_lds), a.keep + (int64_t)bh * a.C);
}


// LDS bytes of the one-work-group selection for a head of L tokens.
size_t select_lds_bytes(int L) {
  const size_t nwords = ((size_t)L + 31) / 32;
  return ((size_t)L + 2 * nwords + kHistBins + 2 * kSelWaves + 3) * sizeof(uint32_t);
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
    const size_t lds = select_lds_bytes(a.L);
    if (lds > 64 * 1024) {
      hipError_t e = hipFuncSetAttribute((const void*)select_kernel_regs, hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(select_kernel_regs, dim3(BH), dim3(kSelThreads), lds, stream, a);
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
