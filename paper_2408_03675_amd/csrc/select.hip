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
// keys (four 8-bit digits, most significant first): each digit pass builds a
// 256-bin histogram of the keys that still match the chosen prefix and picks
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
// 2 = none (uniform).  One kernel per mode keeps each straight-line.
template <int MODE>
__global__ __launch_bounds__(256) void gumbel_keys_kernel(const float* __restrict__ F, int H, int L,
                                                          uint32_t k0, uint32_t k1, uint32_t layer,
                                                          uint32_t* __restrict__ keys) {
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int qd = blockIdx.x * 256 + threadIdx.x;
  const int j0 = qd * 4;
  if (j0 >= L) return;
  const U32x4 w = philox4x32_10(U32x4{(uint32_t)qd, (uint32_t)h, (uint32_t)b, layer}, k0, k1);
  const uint32_t words[4] = {w.x, w.y, w.z, w.w};
  const float* f = F + (int64_t)bh * L;
  uint32_t* out = keys + (int64_t)bh * L;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int j = j0 + e;
    if (j < L) {
      const double u = ((double)words[e] + 0.5) * 0x1p-32;
      const double g = -log(-log(u));
      double key = g;
      if constexpr (MODE == 0) key = (double)f[j] + g;
      if constexpr (MODE == 1) key = log((double)f[j]) + g;
      out[j] = float_order_key((float)key);
    }
  }
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
  uint32_t* hist;   // kSelWaves * 256
  uint32_t* tot;    // 256
  uint32_t* scan;   // 2 * kSelWaves
  uint32_t* shv;    // 4
};

// k-th largest key (1 <= k <= number of keys) and the number of keys equal to
// it that belong to the top k.
template <class Get>
__device__ void radix_select(const Get& get, int L, uint32_t k, const SelScratch& s, uint32_t& T,
                             uint32_t& need) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint32_t prefix = 0u, kr = k;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const uint32_t hm = pass == 0 ? 0u : (0xFFFFFFFFu << (shift + 8));
    for (int i = tid; i < kSelWaves * 256; i += kSelThreads) s.hist[i] = 0u;
    __syncthreads();
    uint32_t* hw = s.hist + wave * 256;
    int run_bin = -1;
    uint32_t run = 0;
    for (int j = tid; j < L; j += kSelThreads) {
      const uint32_t key = get(j);
      if (((key ^ prefix) & hm) == 0u) {
        const int bin = (key >> shift) & 255;
        if (bin != run_bin) {
          if (run) atomicAdd(&hw[run_bin], run);
          run_bin = bin;
          run = 0;
        }
        ++run;
      }
    }
    if (run) atomicAdd(&hw[run_bin], run);
    __syncthreads();
    if (tid < 256) {
      uint32_t t = 0;
#pragma unroll
      for (int w = 0; w < kSelWaves; ++w) t += s.hist[w * 256 + tid];
      s.tot[tid] = t;
    }
    __syncthreads();
    if (wave == 0) {
      uint32_t c[4], local = 0;
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        c[qq] = s.tot[255 - 4 * lane - qq];
        local += c[qq];
      }
      const uint32_t incl = wave_inclusive_scan(local, lane);
      const uint32_t excl = incl - local;
      if (excl < kr && kr <= incl) {
        uint32_t cum = excl;
        for (int qq = 0; qq < 4; ++qq) {
          if (cum + c[qq] >= kr) {
            s.shv[0] = prefix | ((uint32_t)(255 - 4 * lane - qq) << shift);
            s.shv[1] = kr - cum;
            break;
          }
          cum += c[qq];
        }
      }
    }
    __syncthreads();
    prefix = s.shv[0];
    kr = s.shv[1];
    __syncthreads();
  }
  T = prefix;
  need = kr;
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

__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectLaunch a) {
  extern __shared__ uint32_t smem[];
  const int L = a.L;
  const int nwords = (L + 31) / 32;
  const int seg_words = (nwords + kSelThreads - 1) / kSelThreads;
  uint32_t* prot = smem;
  uint32_t* sel = prot + nwords;
  SelScratch s;
  s.hist = sel + nwords;
  s.tot = s.hist + kSelWaves * 256;
  s.scan = s.tot + 256;
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

  // u_score: top-Cp of F over R.
  if (a.Cp > 0) {
    auto key1 = [&](int j) -> uint32_t {
      return ((prot[j >> 5] >> (j & 31)) & 1u) ? 0u : float_order_key(f[j]);
    };
    uint32_t T1, need1;
    radix_select(key1, L, (uint32_t)a.Cp, s, T1, need1);
    mark_top(key1, L, nwords, seg_words, T1, need1, sel, s.scan);
  }

  // u_random: top-Cr of the Gumbel keys over R \ u_score.
  if (a.Cr > 0) {
    auto key2 = [&](int j) -> uint32_t {
      return (((prot[j >> 5] | sel[j >> 5]) >> (j & 31)) & 1u) ? 0u : keys[j];
    };
    uint32_t T2, need2;
    radix_select(key2, L, (uint32_t)a.Cr, s, T2, need2);
    mark_top(key2, L, nwords, seg_words, T2, need2, sel, s.scan);
  }

  // keep = Pi | u_score | u_random, written in ascending order.
  const int w0 = tid * seg_words;
  const int w1 = min(w0 + seg_words, nwords);
  uint32_t cnt = 0;
  for (int w = w0; w < w1; ++w) cnt += __popc(sel[w] | prot[w]);
  uint32_t out = block_exclusive_scan(cnt, s.scan);
  int32_t* keep = a.keep + (int64_t)bh * a.C;
  for (int w = w0; w < w1; ++w) {
    uint32_t bits = sel[w] | prot[w];
    while (bits) {
      const int bit = __ffs(bits) - 1;
      if (out < (uint32_t)a.C) keep[out] = w * 32 + bit;  // |keep| == C by construction
      ++out;
      bits &= bits - 1;
    }
  }
}

size_t select_lds_bytes(int L) {
  const size_t nwords = ((size_t)L + 31) / 32;
  return (2 * nwords + kSelWaves * 256 + 256 + 2 * kSelWaves + 4) * sizeof(uint32_t);
}

hipError_t launch_select(const SelectLaunch& a, hipStream_t stream) {
  const int BH = a.B * a.H;
  if (a.Cr > 0) {
    dim3 gk(((a.L + 3) / 4 + 255) / 256, BH);
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
  const size_t lds = select_lds_bytes(a.L);
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)select_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(select_kernel, dim3(BH), dim3(kSelThreads), lds, stream, a);
  return hipGetLastError();
}

}  // namespace nacl
