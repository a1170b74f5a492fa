// Keep-set selection (NaCl Section 5.1 argmax, Section 5.2 random eviction,
// Algorithm 1 union), one work-group per (b, h).
//
//   Pi       the last n_protect proxy tokens, always kept
//   u_score  top-Cp of F over R = [0, L) \ Pi, ties to the lower index
//   u_random top-Cr of the Gumbel-perturbed keys over R \ u_score, ties to the
//            lower index: Gumbel-top-k, a draw of Cr tokens without
//            replacement from the weights (Softmax(F) by default)
//   keep     Pi | u_score | u_random, ascending, exactly C entries
//
// Both top-k searches are exact radix selects over order-preserving uint32
// keys (12-, 12- and 8-bit digits, most significant first): each digit pass
// builds a histogram of the keys that still match the chosen prefix and picks
// the digit where the count from the top reaches k.  That yields the k-th
// largest key T and how many keys equal to T to take; a block-wide ordered
// scan then hands those to the lowest indices.  Set membership lives in LDS
// bitmaps, one bit per token.

#include "device_common.h"
#include "internal.h"
#include "gumbel.h"
#include "philox.h"

namespace nacl {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;

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

// Longer heads: every radix pass re-reads the keys from global memory
// (L2-resident); the bitmaps and the histogram stay in LDS.
__global__ __launch_bounds__(kSelThreads) void select_kernel_global(SelectLaunch a) {
  extern __shared__ uint32_t smem[];
  const int L = a.L;
  const int nwords = (L + 31) / 32;
  const int seg_words = (nwords + kSelThreads - 1) / kSelThreads;
  uint32_t* fixed = smem;            // Pi, then Pi | u_score
  uint32_t* rnd = fixed + nwords;    // u_random
  SelScratch s;
  s.hist = rnd + nwords;
  s.scan = s.hist + kHistBins;
  s.shv = s.scan + 2 * kSelWaves;

  const int tid = threadIdx.x;
  const int bh = blockIdx.x;
  const float* f = a.scores + (int64_t)bh * L;
  const uint32_t* keys = a.keys2 + (int64_t)bh * L;

  for (int w = tid; w < nwords; w += kSelThreads) {
    fixed[w] = 0u;
    rnd[w] = 0u;
  }
  for (int i = tid; i < kHistBins; i += kSelThreads) s.hist[i] = 0u;
  __syncthreads();
  for (int i = a.P - a.n_protect + tid; i < a.P; i += kSelThreads) {
    const int j = a.pos[i];
    atomicOr(&fixed[j >> 5], 1u << (j & 31));
  }
  __syncthreads();

  // u_score.  Reads `fixed` inside its own marking: a token's bit is read
  // before its word is updated, and a pick is never an excluded token.
  if (a.Cp > 0)
    select_top([&](int j) { return ((fixed[j >> 5] >> (j & 31)) & 1u) ? 0u : float_order_key(f[j]); }, L,
               nwords, seg_words, (uint32_t)a.Cp, s, fixed);
  // u_random over R \ u_score.
  if (a.Cr > 0)
    select_top([&](int j) { return ((fixed[j >> 5] >> (j & 31)) & 1u) ? 0u : keys[j]; }, L, nwords,
               seg_words, (uint32_t)a.Cr, s, rnd);

  assemble_keep(fixed, rnd, nwords, seg_words, a.C, s, a.keep + (int64_t)bh * a.C,
                a.keep + (int64_t)bh * a.C);
}

// LDS bytes of the selection for a head of L tokens.
size_t select_lds_bytes(int L) {
  const size_t nwords = ((size_t)L + 31) / 32;
  const size_t keys = L <= kRegMaxL ? (size_t)L : 0;
  return (keys + 2 * nwords + kHistBins + 2 * kSelWaves + 3) * sizeof(uint32_t);
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
  const bool regs = a.L <= kRegMaxL;
  const size_t lds = select_lds_bytes(a.L);
  const void* fn = regs ? (const void*)select_kernel_regs : (const void*)select_kernel_global;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  if (regs) hipLaunchKernelGGL(select_kernel_regs, dim3(BH), dim3(kSelThreads), lds, stream, a);
  else hipLaunchKernelGGL(select_kernel_global, dim3(BH), dim3(kSelThreads), lds, stream, a);
  return hipGetLastError();
}

}  // namespace nacl
