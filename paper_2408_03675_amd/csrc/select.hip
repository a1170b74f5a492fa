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
#include "philox.h"

namespace nacl {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;

// Gumbel keys of every token: key = binary32(logw + g) with
// g = -ln(-ln u) in binary64, u = (word + 1/2) / 2^32, word = Philox4x32-10
// output j mod 4 at counter (j / 4, h, b, layer) under key = seed.
// MODE selects the log-weight: 0 = F (Softmax(F)), 1 = ln F (weights F),
// 2 = none (uniform).  One kernel per mode keeps each straight-line.  One
// thread per token: the two dependent binary64 logarithms are the cost, so
// every token gets its own thread (the four threads of a Philox block each
// evaluate the block and keep their word; the integer rounds are cheap next
// to the logarithms).
template <int MODE>
__global__ __launch_bounds__(256) void gumbel_keys_kernel(const float* __restrict__ F, int H, int L,
                                                          uint32_t k0, uint32_t k1, uint32_t layer,
                                                          uint32_t* __restrict__ keys) {
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= L) return;
  const U32x4 w = philox4x32_10(U32x4{(uint32_t)(j >> 2), (uint32_t)h, (uint32_t)b, layer}, k0, k1);
  const int e = j & 3;
  const uint32_t word = e == 0 ? w.x : (e == 1 ? w.y : (e == 2 ? w.z : w.w));
  const double u = ((double)word + 0.5) * 0x1p-32;
  const double g = -log(-log(u));
  double key = g;
  if constexpr (MODE == 0) key = (double)F[(int64_t)bh * L + j] + g;
  if constexpr (MODE == 1) key = log((double)F[(int64_t)bh * L + j]) + g;
  keys[(int64_t)bh * L + j] = float_order_key((float)key);
}

__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

// Exclusive prefix sum of v over the work-group in thread order.  scan_buf
// holds 2 * kSelWaves words of LDS.
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* scan_buf) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t x = wave_inclusive_scan(v, lane);
  if (lane == kWave - 1) scan_buf[wave] = x;
  __syncthreads();
  if (wave == 0) {
    uint32_t t = lane < kSelWaves ? scan_buf[lane] : 0u;
    t = wave_inclusive_scan(t, lane);
    if (lane < kSelWaves) scan_buf[kSelWaves + lane] = t;
  }
  __syncthreads();
  const uint32_t base = wave ? scan_buf[kSelWaves + wave - 1] : 0u;
  __syncthreads();
  return base + x - v;
}

struct SelScratch {
  uint32_t* hist;   // kHistBins
  uint32_t* scan;   // 2 * kSelWaves
  uint32_t* shv;    // 4
};

// Radix select digits, most significant first: 12 + 12 + 8 bits.  The wide
// first digit spreads even tightly clustered keys (scores within a few
// binades) over many counters, so the shared histogram's atomics rarely
// collide; later passes only count keys that match the chosen prefix.
constexpr int kHistBins = 4096;
constexpr int kDigitShift[3] = {20, 8, 0};
constexpr int kDigitBits[3] = {12, 12, 8};

// k-th largest key T (1 <= k <= number of keys), the number `need` of keys
// equal to T that belong to the top k, and the number n_eq of keys equal to T.
template <class Get>
__device__ void radix_select(const Get& get, int L, uint32_t k, const SelScratch& s, uint32_t& T,
                             uint32_t& need, uint32_t& n_eq) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0u, kr = k;
#pragma unroll
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = kDigitShift[pass];
    const int nbins = 1 << kDigitBits[pass];
    const uint32_t dmask = (uint32_t)nbins - 1u;
    const uint32_t hm = pass == 0 ? 0u : (0xFFFFFFFFu << (shift + kDigitBits[pass]));
    for (int i = tid; i < nbins; i += kSelThreads) s.hist[i] = 0u;
    __syncthreads();
    // Eight keys per thread in flight before their counter updates.
    for (int j0 = tid; j0 < L; j0 += 8 * kSelThreads) {
      uint32_t kv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u * kSelThreads;
        kv[u] = j < L ? get(j) : 0u;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u * kSelThreads;
        if (j < L && ((kv[u] ^ prefix) & hm) == 0u) atomicAdd(&s.hist[(kv[u] >> shift) & dmask], 1u);
      }
    }
    __syncthreads();
    // Counts from the top: thread t owns bins nbins-1-4t down to nbins-4-4t.
    const int per = (nbins + kSelThreads - 1) / kSelThreads;  // 4 or 1
    uint32_t c[4] = {0u, 0u, 0u, 0u}, local = 0u;
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const int b = nbins - 1 - per * tid - qq;
      if (qq < per && b >= 0) c[qq] = s.hist[b];
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
    __syncthreads();
    prefix = s.shv[0];
    kr = s.shv[1];
    n_eq = s.shv[2];
    __syncthreads();
  }
  T = prefix;
  need = kr;
}

// Sets, in out_bits, the bit of every token with key >= T: the top k when
// every key equal to T belongs to it.  Each wave covers 64 consecutive tokens
// per step; lanes 0 and 32 OR the two words of the ballot into the bitmap
// (the words of a step belong to that wave alone, so no atomics are needed),
// and the four steps of an iteration keep their loads and updates independent.
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
        if (bits) out_bits[word] |= bits;
      }
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

// keys_lds[j] = f(j, src[j]) for the whole head: 16-byte loads, eight per
// thread in flight (src is 16-byte aligned when L % 4 == 0; otherwise
// 4-byte loads).
template <class F>
__device__ void stage_keys(int L, const uint32_t* src, uint32_t* keys_lds, const F& f) {
  if ((L & 3) == 0) {
    const u32x4* s4 = reinterpret_cast<const u32x4*>(src);
    const int n4 = L >> 2;
    for (int i0 = threadIdx.x; i0 < n4; i0 += 8 * kSelThreads) {
      u32x4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * kSelThreads;
        v[u] = i < n4 ? s4[i] : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * kSelThreads;
        if (i < n4) {
#pragma unroll
          for (int e = 0; e < 4; ++e) keys_lds[4 * i + e] = f(4 * i + e, v[u][e]);
        }
      }
    }
  } else {
    for (int j = threadIdx.x; j < L; j += kSelThreads) keys_lds[j] = f(j, src[j]);
  }
  __syncthreads();
}

// KEYS_IN_LDS: the head's keys live in LDS (L * 4 bytes), loaded once per
// selection; otherwise every radix pass re-reads them from global memory
// (L2-resident) for heads too long for LDS.
template <bool KEYS_IN_LDS>
__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectLaunch a) {
  extern __shared__ uint32_t smem[];
  const int L = a.L;
  const int nwords = (L + 31) / 32;
  const int seg_words = (nwords + kSelThreads - 1) / kSelThreads;
  uint32_t* keys_lds = smem;
  uint32_t* prot = smem + (KEYS_IN_LDS ? L : 0);
  uint32_t* sel = prot + nwords;
  SelScratch s;
  s.hist = sel + nwords;
  s.scan = s.hist + kHistBins;
  s.shv = s.scan + 2 * kSelWaves;

  const int tid = threadIdx.x;
  const int bh = blockIdx.x;
  const float* f = a.scores + (int64_t)bh * L;
  const uint32_t* keys = a.keys2 + (int64_t)bh * L;

  for (int w = tid; w < nwords; w += kSelThreads) {
    prot[w] = 0u;
    sel[w] = 0u;
  }
  __syncthreads();
  for (int i = a.P - a.n_protect + tid; i < a.P; i += kSelThreads) {
    const int j = a.pos[i];
    atomicOr(&prot[j >> 5], 1u << (j & 31));
  }
  __syncthreads();
  auto excluded = [&](int j) -> bool { return (((prot[j >> 5] | sel[j >> 5]) >> (j & 31)) & 1u) != 0u; };

  // u_score: top-Cp of F over R.
  if (a.Cp > 0) {
    if constexpr (KEYS_IN_LDS) {
      stage_keys(L, reinterpret_cast<const uint32_t*>(f), keys_lds,
                 [&](int j, uint32_t bits) { return excluded(j) ? 0u : float_order_key(__uint_as_float(bits)); });
      select_top([&](int j) { return keys_lds[j]; }, L, nwords, seg_words, (uint32_t)a.Cp, s, sel);
    } else {
      select_top([&](int j) { return ((prot[j >> 5] >> (j & 31)) & 1u) ? 0u : float_order_key(f[j]); }, L,
                 nwords, seg_words, (uint32_t)a.Cp, s, sel);
    }
  }

  // u_random: top-Cr of the Gumbel keys over R \ u_score.
  if (a.Cr > 0) {
    if constexpr (KEYS_IN_LDS) {
      stage_keys(L, keys, keys_lds, [&](int j, uint32_t key) { return excluded(j) ? 0u : key; });
      select_top([&](int j) { return keys_lds[j]; }, L, nwords, seg_words, (uint32_t)a.Cr, s, sel);
    } else {
      // Reads sel inside the marking of sel: a token's own bit is read before
      // its word is updated, and random picks are never excluded tokens.
      select_top([&](int j) { return excluded(j) ? 0u : keys[j]; }, L, nwords, seg_words, (uint32_t)a.Cr, s,
                 sel);
    }
  }

  // keep = Pi | u_score | u_random, in ascending order: ranks by an ordered
  // scan of the bitmap words, the list assembled in LDS (over the keys when
  // they live there), then copied out with coalesced stores.
  const int w0 = tid * seg_words;
  const int w1 = min(w0 + seg_words, nwords);
  uint32_t cnt = 0;
  for (int w = w0; w < w1; ++w) cnt += __popc(sel[w] | prot[w]);
  uint32_t out = block_exclusive_scan(cnt, s.scan);
  int32_t* keep = a.keep + (int64_t)bh * a.C;
  int32_t* list = KEYS_IN_LDS ? reinterpret_cast<int32_t*>(keys_lds) : keep;
  for (int w = w0; w < w1; ++w) {
    uint32_t bits = sel[w] | prot[w];
    while (bits) {
      const int bit = __ffs(bits) - 1;
      if (out < (uint32_t)a.C) list[out] = w * 32 + bit;  // |keep| == C by construction
      ++out;
      bits &= bits - 1;
    }
  }
  if constexpr (KEYS_IN_LDS) {
    __syncthreads();
    for (int c = tid; c < a.C; c += kSelThreads) keep[c] = list[c];
  }
}

// LDS bytes of select_kernel: bitmaps + histograms (+ keys when in LDS).
size_t select_lds_bytes(int L, bool keys_in_lds) {
  const size_t nwords = ((size_t)L + 31) / 32;
  return ((keys_in_lds ? (size_t)L : 0) + 2 * nwords + kHistBins + 2 * kSelWaves + 4) * sizeof(uint32_t);
}

constexpr size_t kMaxLds = 160 * 1024;

hipError_t launch_select(const SelectLaunch& a, hipStream_t stream) {
  const int BH = a.B * a.H;
  if (a.Cr > 0) {
    dim3 gk((a.L + 255) / 256, BH);
    const uint32_t k0 = (uint32_t)(a.seed & 0xFFFFFFFFu), k1 = (uint32_t)(a.seed >> 32);
    if (a.sampling == 0)
      hipLaunchKernelGGL(gumbel_keys_kernel<0>, gk, dim3(256), 0, stream, a.scores, a.H, a.L, k0, k1,
                         a.layer, a.keys2);
    else if (a.sampling == 1)
      hipLaunchKernelGGL(gumbel_keys_kernel<1>, gk, dim3(256), 0, stream, a.scores, a.H, a.L, k0, k1,
                         a.layer, a.keys2);
    else
      hipLaunchKernelGGL(gumbel_keys_kernel<2>, gk, dim3(256), 0, stream, a.scores, a.H, a.L, k0, k1,
                         a.layer, a.keys2);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const bool in_lds = select_lds_bytes(a.L, true) <= kMaxLds;
  const size_t lds = select_lds_bytes(a.L, in_lds);
  const void* fn = in_lds ? (const void*)select_kernel<true> : (const void*)select_kernel<false>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  if (in_lds) hipLaunchKernelGGL(select_kernel<true>, dim3(BH), dim3(kSelThreads), lds, stream, a);
  else hipLaunchKernelGGL(select_kernel<false>, dim3(BH), dim3(kSelThreads), lds, stream, a);
  return hipGetLastError();
}

}  // namespace nacl
