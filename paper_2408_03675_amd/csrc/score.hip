// Proxy-token scores F (NaCl, Section 5.1 F_score; Appendix A.7): for each
// (b, h), F[j] = sum_i exp(s * <Q[p_i], K[j]> - LSE_i) over proxies with
// p_i >= j, where LSE_i is the natural log-sum-exp of proxy row i over its
// causal keys 0..p_i.
//
// Three kernels, all on MFMA (v_mfma_f32_16x16x32_bf16 for bf16 inputs,
// v_mfma_f32_16x16x4_f32 for fp32 inputs):
//   pass1   per (b, h, key chunk): online base-2 (max, sum) of every proxy
//           row over the chunk's keys -> partials
//   combine per (b, h, proxy): merge the chunk partials -> LSE (base 2)
//   pass2   per (b, h, key chunk): exp2(logit - LSE) column sums over the
//           proxy rows -> F; the reduction of Appendix A.7's Algorithm 2,
//           with each key tile owned by one wave, so there are no atomics and
//           results are bit-reproducible.
//
// Fragment layout.  A 16x16 MFMA tile is indexed by (lane % 16) along M/N and
// by the lane group g = lane / 16 along the contraction.  Lane group g holds
// the contiguous d-slice [g*D/4, (g+1)*D/4) of its row, for Q and K alike;
// contraction step s uses elements [s*E, (s+1)*E) of that slice (E = 8 for
// bf16, 1 for fp32).  Any permutation of the contraction index is harmless as
// long as both operands use the same one, and this one lets every lane fetch
// its slice with 16-byte loads.  The 16x16 accumulator holds rows
// 4*g + e (e = 0..3) and column lane % 16.
//   pass1 computes K_tile * Q_P^T: rows = keys, columns = proxies, so each lane
//         keeps running statistics for one proxy.
//   pass2 computes Q_P * K_tile^T: rows = proxies, columns = keys, so each
//         lane sums one key's column in registers and two cross-lane adds
//         finish it.

#include "device_common.h"
#include "internal.h"

namespace nacl {

template <typename T, int D> struct Mma;

template <int D> struct Mma<__bf16, D> {
  static constexpr int kSteps = D / 32;
  typedef bf16x8 frag_t;
  __device__ static void load(const __bf16* row, int g, frag_t (&f)[kSteps]) {
    const u32x4* p = reinterpret_cast<const u32x4*>(row + g * (D / 4));
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
      u32x4 v = __builtin_nontemporal_load(p + s);
      f[s] = __builtin_bit_cast(frag_t, v);
    }
  }
  __device__ static void zero(frag_t (&f)[kSteps]) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s) f[s] = __builtin_bit_cast(frag_t, u32x4{0u, 0u, 0u, 0u});
  }
  __device__ static f32x4 mma(frag_t a, frag_t b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

template <int D> struct Mma<float, D> {
  static constexpr int kSteps = D / 4;
  typedef float frag_t;
  __device__ static void load(const float* row, int g, frag_t (&f)[kSteps]) {
    const float4* p = reinterpret_cast<const float4*>(row + g * (D / 4));
#pragma unroll
    for (int s = 0; s < kSteps / 4; ++s) {
      float4 v = p[s];
      f[4 * s + 0] = v.x;
      f[4 * s + 1] = v.y;
      f[4 * s + 2] = v.z;
      f[4 * s + 3] = v.w;
    }
  }
  __device__ static void zero(frag_t (&f)[kSteps]) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s) f[s] = 0.f;
  }
  __device__ static f32x4 mma(frag_t a, frag_t b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

constexpr int kScoreThreads = 256;  // 4 waves

// Loads the proxy positions of group [g0, g0 + 16*PB) into LDS (-1 pads).
template <int PB>
__device__ __forceinline__ void load_group_positions(const int* __restrict__ pos, int g0, int gn,
                                                     int* pos_g) {
  __syncthreads();
  if (threadIdx.x < 16 * PB) pos_g[threadIdx.x] = threadIdx.x < gn ? pos[g0 + threadIdx.x] : -1;
  __syncthreads();
}

template <typename T, int D, int PB, int TPW>
__global__ __launch_bounds__(kScoreThreads) void score_pass1_kernel(const T* __restrict__ q,
                                                                    const T* __restrict__ k,
                                                                    ScoreArgs a,
                                                                    float2* __restrict__ partials) {
  using M = Mma<T, D>;
  constexpr int kS = M::kSteps;
  __shared__ int pos_g[16 * PB];
  __shared__ float2 red[4][16 * PB];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const int chunk = blockIdx.x;
  const T* qb = q + b * a.qs[0] + h * a.qs[1];
  const T* kb = k + b * a.ks[0] + h * a.ks[1];
  const int key_base = chunk * (TPW * 4 * 16);
  const float c2 = a.c2;

  for (int g0 = 0; g0 < a.P; g0 += 16 * PB) {
    const int gn = min(16 * PB, a.P - g0);
    load_group_positions<PB>(a.pos, g0, gn, pos_g);
    const int first = pos_g[0], last = pos_g[gn - 1];

    typename M::frag_t qf[PB][kS];
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int i = 16 * pb + r16;
      if (i < gn) M::load(qb + (int64_t)pos_g[i] * a.qs[2], g, qf[pb]);
      else M::zero(qf[pb]);
    }

    float m[PB], s[PB];
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) { m[pb] = -INFINITY; s[pb] = 0.f; }

#pragma unroll 1
    for (int it = 0; it < TPW; ++it) {
      const int key0 = key_base + (it * 4 + wave) * 16;
      if (key0 > last) break;
      typename M::frag_t kf[kS];
      M::load(kb + (int64_t)min(key0 + r16, a.L - 1) * a.ks[2], g, kf);
      const bool full = key0 + 15 <= first;
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < kS; ++ks) acc = M::mma(kf[ks], qf[pb][ks], acc);
        if (full) {
          const float mx = fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3]));
          const float mn = fmaxf(m[pb], mx);
          const float sc = fast_exp2((m[pb] - mn) * c2);
          const float mc = mn * c2;
          float sum = fast_exp2(fmaf(acc[0], c2, -mc)) + fast_exp2(fmaf(acc[1], c2, -mc));
          sum += fast_exp2(fmaf(acc[2], c2, -mc)) + fast_exp2(fmaf(acc[3], c2, -mc));
          s[pb] = fmaf(s[pb], sc, sum);
          m[pb] = mn;
        } else {
          const int pi = pos_g[16 * pb + r16];
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = (key0 + 4 * g + e <= pi) ? acc[e] : -INFINITY;
          const float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
          const float mn = fmaxf(m[pb], mx);
          if (mn != -INFINITY) {
            const float sc = (m[pb] == -INFINITY) ? 0.f : fast_exp2((m[pb] - mn) * c2);
            const float mc = mn * c2;
            float sum = 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) sum += (v[e] == -INFINITY) ? 0.f : fast_exp2(fmaf(v[e], c2, -mc));
            s[pb] = fmaf(s[pb], sc, sum);
            m[pb] = mn;
          }
        }
      }
    }

    // Merge the four lane groups (different keys, same proxy), then the waves.
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      float mm = m[pb] * c2, ss = s[pb];
      lse_merge(mm, ss, __shfl_xor(mm, 16), __shfl_xor(ss, 16));
      lse_merge(mm, ss, __shfl_xor(mm, 32), __shfl_xor(ss, 32));
      if (g == 0) red[wave][16 * pb + r16] = make_float2(mm, ss);
    }
    __syncthreads();
    if (threadIdx.x < gn) {
      float2 r = red[0][threadIdx.x];
#pragma unroll
      for (int w = 1; w < 4; ++w) lse_merge(r.x, r.y, red[w][threadIdx.x].x, red[w][threadIdx.x].y);
      partials[((int64_t)bh * gridDim.x + chunk) * a.P + g0 + threadIdx.x] = r;
    }
  }
}

__global__ __launch_bounds__(256) void lse_combine_kernel(const float2* __restrict__ partials,
                                                          int n_chunks, int P,
                                                          float* __restrict__ lse2) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  const int bh = blockIdx.y;
  if (i >= P) return;
  float m = -INFINITY, s = 0.f;
  const float2* p = partials + (int64_t)bh * n_chunks * P + i;
  for (int c = 0; c < n_chunks; ++c) {
    float2 v = p[(int64_t)c * P];
    lse_merge(m, s, v.x, v.y);
  }
  lse2[(int64_t)bh * P + i] = m + __log2f(s);
}

template <typename T, int D, int PB, int TPW>
__global__ __launch_bounds__(kScoreThreads) void score_pass2_kernel(const T* __restrict__ q,
                                                                    const T* __restrict__ k,
                                                                    ScoreArgs a,
                                                                    const float* __restrict__ lse,
                                                                    float lse_mul,
                                                                    float* __restrict__ F) {
  using M = Mma<T, D>;
  constexpr int kS = M::kSteps;
  __shared__ int pos_g[16 * PB];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const T* qb = q + b * a.qs[0] + h * a.qs[1];
  const T* kb = k + b * a.ks[0] + h * a.ks[1];
  const int key_base = blockIdx.x * (TPW * 4 * 16);
  const float c2 = a.c2;

  float colsum[TPW];
#pragma unroll
  for (int it = 0; it < TPW; ++it) colsum[it] = 0.f;

  for (int g0 = 0; g0 < a.P; g0 += 16 * PB) {
    const int gn = min(16 * PB, a.P - g0);
    load_group_positions<PB>(a.pos, g0, gn, pos_g);
    const int first = pos_g[0], last = pos_g[gn - 1];

    typename M::frag_t qf[PB][kS];
    float lr[PB][4];
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int i = 16 * pb + r16;
      if (i < gn) M::load(qb + (int64_t)pos_g[i] * a.qs[2], g, qf[pb]);
      else M::zero(qf[pb]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int ir = 16 * pb + 4 * g + e;
        lr[pb][e] = ir < gn ? lse[(int64_t)bh * a.P + g0 + ir] * lse_mul : INFINITY;
      }
    }

#pragma unroll
    for (int it = 0; it < TPW; ++it) {
      const int key0 = key_base + (it * 4 + wave) * 16;
      if (key0 > last) break;
      typename M::frag_t kf[kS];
      M::load(kb + (int64_t)min(key0 + r16, a.L - 1) * a.ks[2], g, kf);
      const bool full = key0 + 15 <= first;
      float cs = 0.f;
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < kS; ++ks) acc = M::mma(qf[pb][ks], kf[ks], acc);
        if (full) {
#pragma unroll
          for (int e = 0; e < 4; ++e) cs += fast_exp2(fmaf(acc[e], c2, -lr[pb][e]));
        } else {
          const int key = key0 + r16;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int pi = pos_g[16 * pb + 4 * g + e];
            cs += (key <= pi) ? fast_exp2(fmaf(acc[e], c2, -lr[pb][e])) : 0.f;
          }
        }
      }
      colsum[it] += cs;
    }
  }

#pragma unroll
  for (int it = 0; it < TPW; ++it) {
    const int key0 = key_base + (it * 4 + wave) * 16;
    float v = colsum[it];
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    if (g == 0 && key0 + r16 < a.L) F[(int64_t)bh * a.L + key0 + r16] = v;
  }
}

// ---------------------------------------------------------------------------
// Host-side launchers.

namespace {

template <typename T, int D, int PB>
hipError_t launch_score_t(const ScoreLaunch& L, hipStream_t stream) {
  constexpr int TPW = kScoreTilesPerWave;
  const T* q = static_cast<const T*>(L.q);
  const T* k = static_cast<const T*>(L.k);
  const int BH = L.args.B * L.args.H;
  if (L.run_pass1) {
    dim3 g1(L.n_chunks1, BH);
    hipLaunchKernelGGL((score_pass1_kernel<T, D, PB, TPW>), g1, dim3(kScoreThreads), 0, stream, q, k,
                       L.args, L.partials);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 gc((L.args.P + 255) / 256, BH);
    hipLaunchKernelGGL(lse_combine_kernel, gc, dim3(256), 0, stream, L.partials, L.n_chunks1, L.args.P,
                       L.lse2_ws);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  dim3 g2(L.n_chunks2, BH);
  hipLaunchKernelGGL((score_pass2_kernel<T, D, PB, TPW>), g2, dim3(kScoreThreads), 0, stream, q, k,
                     L.args, L.lse_in, L.lse_mul, L.scores);
  return hipGetLastError();
}

template <typename T, int D, int PBMAX>
hipError_t dispatch_pb(const ScoreLaunch& L, hipStream_t stream) {
  const int need = std::min((L.args.P + 15) / 16, PBMAX);
  if (need <= 1) return launch_score_t<T, D, 1>(L, stream);
  if (need <= 2) return launch_score_t<T, D, 2>(L, stream);
  if constexpr (PBMAX >= 8) {
    if (need > 4) return launch_score_t<T, D, 8>(L, stream);
  }
  return launch_score_t<T, D, 4>(L, stream);
}

}  // namespace

hipError_t launch_score(const ScoreLaunch& L, hipStream_t stream) {
  if (L.dtype == 1) {
    if (L.D == 128) return dispatch_pb<__bf16, 128, 8>(L, stream);
    return dispatch_pb<__bf16, 64, 8>(L, stream);
  }
  if (L.D == 128) return dispatch_pb<float, 128, 4>(L, stream);
  return dispatch_pb<float, 64, 8>(L, stream);
}

}  // namespace nacl
