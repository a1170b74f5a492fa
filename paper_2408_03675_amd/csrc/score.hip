// Proxy-token scores F (NaCl, Section 5.1 F_score; Appendix A.7): for each
// (b, h), F[j] = sum_i exp(s * <Q[p_i], K[j]> - LSE_i) over proxies with
// p_i >= j, where LSE_i is the natural log-sum-exp of proxy row i over its
// causal keys 0..p_i.
//
// One persistent kernel runs two kinds of work items over key chunks of
// sched.chunk_keys keys, all on MFMA (v_mfma_f32_16x16x32_bf16 for bf16
// inputs, v_mfma_f32_16x16x4_f32 for fp32 inputs):
//   pass 1  online base-2 (max, sum) of every proxy row over the chunk's keys
//           -> per-chunk partials; the last chunk of a head to finish merges
//           the head's partials into its log-sum-exp
//   pass 2  exp2(logit - LSE) summed over the proxy rows for each key of the
//           chunk -> F (the column reduction of Appendix A.7's Algorithm 2).
//           Each key tile is owned by one wave: no atomics on F, so results
//           are bit-reproducible.
//
// Work-groups take items from a queue counter in a fixed order: the pass-1
// items of head group g + lag come before the pass-2 items of head group g.
// A pass-2 item therefore re-reads keys that pass 1 streamed from HBM shortly
// before, which the 256 MB memory-side Infinity Cache still holds, so K
// crosses HBM about once.  A pass-2 item waits (bounded spin) until its
// head's log-sum-exp is published; every item it waits on was taken from the
// queue earlier by a running work-group and never waits itself, so the wait
// always ends, whatever the number of resident work-groups.
//
// Fragment layout.  A 16x16 MFMA tile is indexed by (lane % 16) along M/N and
// by the lane group g = lane / 16 along the contraction.  Lane group g holds
// the contiguous d-slice [g*D/4, (g+1)*D/4) of its row, for Q and K alike;
// contraction step s uses elements [s*E, (s+1)*E) of that slice (E = 8 for
// bf16, 1 for fp32).  Any permutation of the contraction index is harmless as
// long as both operands use the same one, and this one lets every lane fetch
// its slice with 16-byte loads.  The 16x16 accumulator holds rows
// 4*g + e (e = 0..3) and column lane % 16.
//   pass 1 computes K_tile * Q_P^T: rows = keys, columns = proxies, so each
//          lane keeps running statistics for one proxy.
//   pass 2 computes Q_P * K_tile^T: rows = proxies, columns = keys, so each
//          lane sums one key's column in registers and two cross-lane adds
//          finish it.

#include <type_traits>

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
    for (int s = 0; s < kSteps; ++s) f[s] = __builtin_bit_cast(frag_t, p[s]);
  }
  __device__ static void zero(frag_t (&f)[kSteps]) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s) f[s] = __builtin_bit_cast(frag_t, u32x4{0u, 0u, 0u, 0u});
  }
  __device__ static f32x4 mma(frag_t a, frag_t b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  // Fragment of row r16 from a staged K tile (see KStage); one 16-byte chunk
  // per contraction step.
  template <int kChunks, int kSwz>
  __device__ static void from_lds(const unsigned char* tile, int r16, int g, frag_t (&f)[kSteps]) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
      const int x = (g * kSteps + s) ^ (r16 & kSwz);
      f[s] = __builtin_bit_cast(frag_t, *reinterpret_cast<const u32x4*>(tile + (r16 * kChunks + x) * 16));
    }
  }
};

template <int D> struct Mma<float, D> {
  static constexpr int kSteps = D / 4;
  typedef float frag_t;
  __device__ static void load(const float* row, int g, frag_t (&f)[kSteps]) {
    const float4* p = reinterpret_cast<const float4*>(row + g * (D / 4));
#pragma unroll
    for (int s = 0; s < kSteps / 4; ++s) {
      const float4 v = p[s];
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
  // Four contraction steps per 16-byte chunk.
  template <int kChunks, int kSwz>
  __device__ static void from_lds(const unsigned char* tile, int r16, int g, frag_t (&f)[kSteps]) {
#pragma unroll
    for (int cc = 0; cc < kSteps / 4; ++cc) {
      const int x = (g * (kSteps / 4) + cc) ^ (r16 & kSwz);
      const f32x4 v = *reinterpret_cast<const f32x4*>(tile + (r16 * kChunks + x) * 16);
      f[4 * cc + 0] = v[0];
      f[4 * cc + 1] = v[1];
      f[4 * cc + 2] = v[2];
      f[4 * cc + 3] = v[3];
    }
  }
};

// Cache policy of the K tile loads: 2 = nt (streaming).  Each pass reads K
// once; on a plain LDS-DMA ring the streaming hint raised the rate from 5.6
// to 6.2 TB/s (the score kernel itself times the same either way).
#ifndef NACL_SCORE_DMA_AUX
#define NACL_SCORE_DMA_AUX 2
#endif
constexpr int kScoreDmaAux = NACL_SCORE_DMA_AUX;

// A 16-key tile of K staged in LDS by direct buffer->LDS loads
// (buffer_load_dwordx4 ... lds: each lane moves 16 bytes, and one
// instruction fills 1 KB of LDS in lane order).  Row r of the tile occupies
// kChunks consecutive 16-byte slots; slot x holds the row's chunk
// x ^ (r & kSwz), an XOR swizzle that spreads the fragment reads of 16 rows
// over the LDS banks.  Addressing goes through a buffer descriptor of the
// head's K rows: rows at or past L fall outside it and read as zeros (their
// keys are masked), and the tile position is a scalar offset.
template <typename T, int D>
struct KStage {
  static constexpr int kRowBytes = D * (int)sizeof(T);
  static constexpr int kChunks = kRowBytes / 16;
  static constexpr int kRowsPerInstr = 64 / kChunks;
  static constexpr int kInstr = 16 / kRowsPerInstr;  // DMA instructions per tile
  static constexpr int kTileBytes = 16 * kRowBytes;
  static constexpr int kSwz = (kChunks < 8 ? kChunks : 8) - 1;
  // Ring depth in tiles (one __shared__ array per slot, see score_kernel):
  // kScoreRingBytes of LDS per key group, at least double buffering, at most 8.
  static constexpr int kDepth =
      kScoreRingBytes / kTileBytes < 2 ? 2 : (kScoreRingBytes / kTileBytes > 8 ? 8 : kScoreRingBytes / kTileBytes);

  // Lane byte offsets inside a tile, one per DMA instruction.
  __device__ static void offsets(uint32_t row_bytes, int lane, uint32_t (&vo)[kInstr]) {
#pragma unroll
    for (int i = 0; i < kInstr; ++i) {
      const int row = i * kRowsPerInstr + lane / kChunks;
      const int c = (lane % kChunks) ^ (row & kSwz);
      vo[i] = (uint32_t)row * row_bytes + (uint32_t)c * 16u;
    }
  }
  // The DMA instructions i = half, half + 2, ... of one tile.
  __device__ static void issue_half(__amdgpu_buffer_rsrc_t rsrc, const uint32_t (&vo)[kInstr],
                                    uint32_t tile_byte, unsigned char* dst, int half) {
#pragma unroll
    for (int j = 0; j < kInstr / 2; ++j) {
      const int i = 2 * j + half;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(dst + i * 1024),
                                               16, vo[i], tile_byte, 0, kScoreDmaAux);
    }
  }
};

// Waits until at most `remaining` tiles of DMA loads (kInstr instructions
// each) are outstanding for this wave.  The tile loops issue no other vector
// memory operations, so the count is exact.  The memory clobber keeps LDS
// reads of the awaited tile below the wait.
template <int kInstr, int K>
__device__ __forceinline__ void wait_dma_tiles(int remaining) {
  if constexpr (K <= 0) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  } else {
    if (remaining >= K) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kInstr * K) : "memory");
    else wait_dma_tiles<kInstr, K - 1>(remaining);
  }
}

constexpr int kScoreThreads = 128 * kScoreKeyGroups;  // 2 waves per key group
// Word 3 of a raw buffer descriptor on gfx9-family parts (32-bit data format).
constexpr int kBufferRsrcWord3 = 0x00020000;

// Calls f(std::integral_constant<int, i>) for i = 0 .. N-1.
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}
constexpr uint32_t kSpinLimit = 1u << 24;

struct ItemRef {
  int kind;   // 1 = pass 1, 2 = pass 2
  int bh;
  int chunk;
};

// Item i of the queue order described at the top of the file.
__device__ __forceinline__ ItemRef decode_item(const ScoreSched& s, int i) {
  const int S = s.heads_per_group * s.n_chunks;  // items per group and pass
  int kind, group, r;
  if (s.lse_given) {
    kind = 2;
    group = i / S;
    r = i % S;
  } else if (i < s.lag * S) {
    kind = 1;
    group = i / S;
    r = i % S;
  } else {
    const int i2 = i - s.lag * S;
    const int mid = (s.n_groups - s.lag) * 2 * S;
    if (i2 < mid) {
      const int step = s.lag + i2 / (2 * S);
      r = i2 % (2 * S);
      if (r < S) {
        kind = 1;
        group = step;
      } else {
        kind = 2;
        group = step - s.lag;
        r -= S;
      }
    } else {
      kind = 2;
      group = s.n_groups - s.lag + (i2 - mid) / S;
      r = (i2 - mid) % S;
    }
  }
  return ItemRef{kind, group * s.heads_per_group + r / s.n_chunks, r % s.n_chunks};
}

// Pass 1 over one tile of 16 keys: folds the tile's logits into the running
// base-2 (max, sum) of the 16*PB proxies (m in raw logit units, the sum
// relative to exp2(m * c2)).  Proxy blocks go in batches of kHalf so at most
// kHalf accumulators are live.
//
// Tiles where every key is visible to every proxy of the group (the common
// case) keep the reference max lazily: terms may exceed exp2(m * c2) by up to
// 2^kLazyLog2, and only a tile whose max passes that threshold in some lane
// rescales, on a wave-uniform branch.  Tiles that straddle a proxy position
// mask keys past each proxy and update the max exactly.
constexpr float kLazyLog2 = 8.f;

template <typename M, int PB>
__device__ __forceinline__ void pass1_tile_full(const typename M::frag_t (&kf)[M::kSteps],
                                                const typename M::frag_t (&qf)[PB][M::kSteps], float c2,
                                                float lazy_raw, float (&m)[PB], float (&sm)[PB]) {
  constexpr int kHalf = PB > 4 ? 4 : PB;
#pragma unroll
  for (int p0 = 0; p0 < PB; p0 += kHalf) {
    f32x4 acc[kHalf];
#pragma unroll
    for (int j = 0; j < kHalf; ++j) {
      acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < M::kSteps; ++ks) acc[j] = M::mma(kf[ks], qf[p0 + j][ks], acc[j]);
    }
    bool over = false;
#pragma unroll
    for (int j = 0; j < kHalf; ++j)
      over |= fmaxf(fmaxf(fmaxf(acc[j][0], acc[j][1]), acc[j][2]), acc[j][3]) > m[p0 + j] + lazy_raw;
    if (__builtin_amdgcn_ballot_w64(over)) {
#pragma unroll
      for (int j = 0; j < kHalf; ++j) {
        const int pb = p0 + j;
        const float mx = fmaxf(fmaxf(fmaxf(acc[j][0], acc[j][1]), acc[j][2]), acc[j][3]);
        const float mn = fmaxf(m[pb], mx);
        sm[pb] = (m[pb] == -INFINITY) ? 0.f : sm[pb] * fast_exp2((m[pb] - mn) * c2);
        m[pb] = mn;
      }
    }
#pragma unroll
    for (int j = 0; j < kHalf; ++j) {
      const int pb = p0 + j;
      const float mc = m[pb] * c2;
      float sum = fast_exp2(fmaf(acc[j][0], c2, -mc)) + fast_exp2(fmaf(acc[j][1], c2, -mc));
      sum += fast_exp2(fmaf(acc[j][2], c2, -mc)) + fast_exp2(fmaf(acc[j][3], c2, -mc));
      sm[pb] += sum;
    }
  }
}

template <typename M, int PB>
__device__ __forceinline__ void pass1_tile_masked(const typename M::frag_t (&kf)[M::kSteps],
                                                  const typename M::frag_t (&qf)[PB][M::kSteps], int key0,
                                                  const int* pos_g, int g, int r16, float c2, float (&m)[PB],
                                                  float (&sm)[PB]) {
  constexpr int kHalf = PB > 4 ? 4 : PB;
#pragma unroll
  for (int p0 = 0; p0 < PB; p0 += kHalf) {
    f32x4 acc_h[kHalf];
#pragma unroll
    for (int j = 0; j < kHalf; ++j) {
      acc_h[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < M::kSteps; ++ks) acc_h[j] = M::mma(kf[ks], qf[p0 + j][ks], acc_h[j]);
    }
#pragma unroll
    for (int j = 0; j < kHalf; ++j) {
      const int pb = p0 + j;
      const f32x4 acc = acc_h[j];
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
        sm[pb] = fmaf(sm[pb], sc, sum);
        m[pb] = mn;
      }
    }
  }
}

// Pass 2 over one tile of 16 keys: this lane's share of its key's column sum
// of exp2(logit - LSE) over the 16*PB proxies (lse_g: base-2 LSE per row).
template <typename M, int PB, bool FULL>
__device__ __forceinline__ float pass2_tile(const typename M::frag_t (&kf)[M::kSteps],
                                            const typename M::frag_t (&qf)[PB][M::kSteps], int key0,
                                            const int* pos_g, int g, int r16, float c2,
                                            const float* lse_g) {
  // Proxy blocks in batches of kHalf so at most kHalf accumulators are live.
  constexpr int kHalf = PB > 4 ? 4 : PB;
  float cs = 0.f;
#pragma unroll
  for (int p0 = 0; p0 < PB; p0 += kHalf) {
    f32x4 acc[kHalf];
#pragma unroll
    for (int j = 0; j < kHalf; ++j) {
      acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < M::kSteps; ++ks) acc[j] = M::mma(qf[p0 + j][ks], kf[ks], acc[j]);
    }
#pragma unroll
    for (int j = 0; j < kHalf; ++j) {
      const int pb = p0 + j;
      const f32x4 lr = *reinterpret_cast<const f32x4*>(lse_g + 16 * pb + 4 * g);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = fast_exp2(fmaf(acc[j][e], c2, -lr[e]));
        if constexpr (FULL) cs += x;
        else cs += (key0 + r16 <= pos_g[16 * pb + 4 * g + e]) ? x : 0.f;
      }
    }
  }
  return cs;
}

// Column sums of four consecutive tiles: x[t] holds, in lane (g, r16), the
// sum over lane group g's proxy rows for key r16 of tile t.  Two
// v_permlane32_swap and one v_permlane16_swap transpose the four lane groups
// so that lane group g returns the full column sum of tile g.
__device__ __forceinline__ float colsum4(float x0, float x1, float x2, float x3) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x0), __float_as_uint(x2), false, false);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x1), __float_as_uint(x3), false, false);
  const float y0 = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const float y1 = __uint_as_float(b[0]) + __uint_as_float(b[1]);
  auto c = __builtin_amdgcn_permlane16_swap(__float_as_uint(y0), __float_as_uint(y1), false, false);
  return __uint_as_float(c[0]) + __uint_as_float(c[1]);
}

// Work-group layout: kScoreKeyGroups key groups x 2 proxy halves, one wave
// each.  The two waves of a key group share one LDS ring of K tiles and each
// holds the Q fragments of half of the proxy group, which keeps registers low
// enough for two waves per SIMD.  Each key group covers s.tpw consecutive
// tiles (at most TPWMAX), so an item spans kScoreKeyGroups * s.tpw * 16 keys.
template <typename T, int D, int PB, int TPWMAX>
__global__ __launch_bounds__(kScoreThreads)
__attribute__((amdgpu_waves_per_eu(kScoreWavesPerSimd, kScoreWavesPerSimd))) void score_kernel(
    const T* __restrict__ q, const T* __restrict__ k, ScoreArgs a, ScoreSched s) {
  using M = Mma<T, D>;
  using KS = KStage<T, D>;
  constexpr int kS = M::kSteps;
  constexpr int kGroup = 16 * PB;        // proxies per group
  constexpr int PBW = PB / 2;            // proxy blocks per wave
  constexpr int kHalfRows = 16 * PBW;    // proxies per wave
  constexpr int kMaxKeysPerPair = TPWMAX * 16;
  constexpr int kDmaPerWave = KS::kInstr / 2;
  static_assert(PB % 2 == 0, "proxy groups split over two waves");
  static_assert(KS::kInstr % 2 == 0, "tile DMA split over two waves");
  constexpr int kUnroll = KS::kDepth > 4 ? KS::kDepth : 4;  // tiles per unrolled step
  static_assert(kUnroll % KS::kDepth == 0 && kScoreTpwMin % kUnroll == 0, "tiles per key group vs ring depth");
  constexpr int NK = kScoreKeyGroups;
  __shared__ int item_s, last_s;
  __shared__ int pos_g[kGroup];
  __shared__ float2 red[NK][kGroup];
  __shared__ float2 mrg[kScoreThreads];
  __shared__ float col_lds[2 * NK][kMaxKeysPerPair];
  __shared__ __attribute__((aligned(16))) float lse_g[kGroup];
  // One array per ring slot: distinct objects let the compiler see that a
  // DMA into one slot does not alias reads of another, so it does not wait
  // for outstanding DMA before every LDS read.
#define NACL_KSLOT(i) \
  __shared__ __attribute__((aligned(16))) unsigned char kslot##i[NK][KS::kDepth > i ? KS::kTileBytes : 16];
  NACL_KSLOT(0) NACL_KSLOT(1) NACL_KSLOT(2) NACL_KSLOT(3) NACL_KSLOT(4) NACL_KSLOT(5) NACL_KSLOT(6) NACL_KSLOT(7)
#undef NACL_KSLOT

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int kp = wave >> 1, ph = wave & 1;  // key group, proxy half
  const int r16 = lane & 15, g = lane >> 4;
  const float c2 = a.c2;
  float* my_cols = col_lds[wave];

  for (;;) {
    __syncthreads();
    if (threadIdx.x == 0) item_s = (int)atomicAdd(s.queue, 1u);
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(item_s);
    if (item >= s.total_items) break;
    const ItemRef it = decode_item(s, item);
    const int bh = it.bh, b = bh / a.H, h = bh % a.H;
    const T* qb = q + b * a.qs[0] + h * a.qs[1];
    const T* kb = k + b * a.ks[0] + h * a.ks[1];
    const int TPW = s.tpw;  // multiple of kUnroll, at most TPWMAX
    const int kKeysPerPair = TPW * 16;
    const int chunk_key0 = it.chunk * s.chunk_keys;
    const int key_base = chunk_key0 + kp * kKeysPerPair;
    const bool beyond = chunk_key0 > a.p_last;  // no proxy sees these keys

    auto slot = [&](auto u_c) -> unsigned char* {
      constexpr int u = decltype(u_c)::value;
      if constexpr (u == 0) return kslot0[kp];
      else if constexpr (u == 1) return kslot1[kp];
      else if constexpr (u == 2) return kslot2[kp];
      else if constexpr (u == 3) return kslot3[kp];
      else if constexpr (u == 4) return kslot4[kp];
      else if constexpr (u == 5) return kslot5[kp];
      else if constexpr (u == 6) return kslot6[kp];
      else return kslot7[kp];
    };
    // Runs step(t, tile) over the key group's TPW tiles.  Tiles stream
    // through the pair's LDS ring of kDepth slots: tile t + kDepth - 1 is in
    // flight while tile t is read into registers and computed.  Each wave of
    // the pair issues half of a tile's DMA and waits for its own half; the
    // barrier then publishes the whole tile (and retires every read of the
    // slot the next DMA overwrites).
    auto k_stream = [&](auto&& step) {
      const uint32_t row_bytes = (uint32_t)(a.ks[2] * (int64_t)sizeof(T));
      const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<T*>(kb), (short)0, (int)((uint32_t)(a.L - 1) * row_bytes + KS::kRowBytes),
          kBufferRsrcWord3);
      uint32_t vo[KS::kInstr];
      KS::offsets(row_bytes, lane, vo);
      auto issue_tile = [&](int t, unsigned char* dst) {
        KS::issue_half(rsrc, vo, (uint32_t)(key_base + 16 * t) * row_bytes, dst, ph);
      };
      static_for<KS::kDepth - 1>([&](auto u_c) {
        constexpr int u = decltype(u_c)::value;
        if (u < TPW) issue_tile(u, slot(u_c));
      });
#pragma unroll 1
      for (int t = 0; t < TPW; t += kUnroll) {
        static_for<kUnroll>([&](auto u_c) {
          constexpr int u = decltype(u_c)::value;
          const int tt = t + u;
          wait_dma_tiles<kDmaPerWave, KS::kDepth - 2>(min(KS::kDepth - 2, TPW - 1 - tt));
          __syncthreads();
          typename M::frag_t kf[kS];
          M::template from_lds<KS::kChunks, KS::kSwz>(slot(std::integral_constant<int, u % KS::kDepth>{}), r16, g,
                                                      kf);
          const int tn = tt + KS::kDepth - 1;
          if (tn < TPW) issue_tile(tn, slot(std::integral_constant<int, (u + KS::kDepth - 1) % KS::kDepth>{}));
          step(tt, kf, u_c);
        });
      }
    };
    // Positions of the proxy group [g0, g0 + gn), -1 past its end.
    auto load_group = [&](int g0, int gn) {
      __syncthreads();
      for (int i = threadIdx.x; i < kGroup; i += kScoreThreads) pos_g[i] = i < gn ? a.pos[g0 + i] : -1;
      __syncthreads();
    };
    // This wave's Q fragments: proxies kHalfRows * ph + [0, kHalfRows) of the group.
    auto load_q = [&](int gn, typename M::frag_t (&qf)[PBW][kS]) {
#pragma unroll
      for (int pb = 0; pb < PBW; ++pb) {
        const int i = ph * kHalfRows + 16 * pb + r16;
        if (i < gn) M::load(qb + (int64_t)pos_g[i] * a.qs[2], g, qf[pb]);
        else M::zero(qf[pb]);
      }
    };
    const int* my_pos = pos_g + ph * kHalfRows;

    if (it.kind == 1) {
      // ---------------- pass 1: per-chunk (max, sum) of every proxy row ----
      float2* part = s.partials + ((int64_t)bh * s.n_chunks + it.chunk) * a.P;
      if (beyond)
        for (int i = threadIdx.x; i < a.P; i += kScoreThreads)
          store_coherent(part + i, make_float2(-INFINITY, 0.f));
      for (int g0 = 0; g0 < (beyond ? 0 : a.P); g0 += kGroup) {
        const int gn = min(kGroup, a.P - g0);
        load_group(g0, gn);
        const int first = pos_g[0], last = pos_g[gn - 1];
        typename M::frag_t qf[PBW][kS];
        load_q(gn, qf);
        float m[PBW], sm[PBW];
#pragma unroll
        for (int pb = 0; pb < PBW; ++pb) {
          m[pb] = -INFINITY;
          sm[pb] = 0.f;
        }
        const float lazy_raw = kLazyLog2 / c2;
        auto step1 = [&](int t, const typename M::frag_t (&kf)[kS], auto) {
          const int key0 = key_base + t * 16;
          if (key0 + 15 <= first) pass1_tile_full<M, PBW>(kf, qf, c2, lazy_raw, m, sm);
          else if (key0 <= last) pass1_tile_masked<M, PBW>(kf, qf, key0, my_pos, g, r16, c2, m, sm);
        };
        k_stream(step1);
        // Merge the four lane groups (different keys, same proxy), then the key groups.
#pragma unroll
        for (int pb = 0; pb < PBW; ++pb) {
          float mm = m[pb] * c2, ss = sm[pb];
          lse_merge(mm, ss, __shfl_xor(mm, 16), __shfl_xor(ss, 16));
          lse_merge(mm, ss, __shfl_xor(mm, 32), __shfl_xor(ss, 32));
          if (g == 0) red[kp][ph * kHalfRows + 16 * pb + r16] = make_float2(mm, ss);
        }
        __syncthreads();
        for (int i = threadIdx.x; i < gn; i += kScoreThreads) {
          float2 r = red[0][i];
#pragma unroll
          for (int kk = 1; kk < NK; ++kk) lse_merge(r.x, r.y, red[kk][i].x, red[kk][i].y);
          store_coherent(part + g0 + i, r);
        }
      }
      // Publish the partials; the last chunk of the head merges them.
      wait_stores();
      __syncthreads();
      if (threadIdx.x == 0) last_s = atomicAdd(&s.head_cnt[bh], 1u) == (unsigned)(s.n_chunks - 1);
      __syncthreads();
      if (last_s) {
        // Merge the head's n_chunks partials per proxy: `split` threads share
        // a proxy, each taking every split-th chunk with kBatch loads in
        // flight, and combine through LDS.
        const float2* hp = s.partials + (int64_t)bh * s.n_chunks * a.P;
        const int split = a.P >= kScoreThreads ? 1 : kScoreThreads / a.P;
        const int part = threadIdx.x / a.P;  // >= split for idle threads when P does not divide
        constexpr int kBatch = 8;
        for (int i0 = 0; i0 < a.P; i0 += kScoreThreads) {
          const int i = i0 + (split == 1 ? (int)threadIdx.x : (int)threadIdx.x % a.P);
          float mm = -INFINITY, ss = 0.f;
          if (i < a.P && part < split) {
            for (int c0 = part; c0 < s.n_chunks; c0 += kBatch * split) {
              float2 v[kBatch];
#pragma unroll
              for (int u = 0; u < kBatch; ++u) {
                const int c = c0 + u * split;
                v[u] = c < s.n_chunks ? load_coherent(hp + (int64_t)c * a.P + i) : make_float2(-INFINITY, 0.f);
              }
#pragma unroll
              for (int u = 0; u < kBatch; ++u) lse_merge(mm, ss, v[u].x, v[u].y);
            }
          }
          if (split > 1) {
            mrg[threadIdx.x] = make_float2(mm, ss);
            __syncthreads();
            if (part == 0 && i < a.P)
              for (int pp = 1; pp < split; ++pp) {
                const float2 r = mrg[threadIdx.x + pp * a.P];
                lse_merge(mm, ss, r.x, r.y);
              }
          }
          if (part == 0 && i < a.P) store_coherent(s.lse2 + (int64_t)bh * a.P + i, mm + __log2f(ss));
        }
        wait_stores();
        __syncthreads();
        if (threadIdx.x == 0) atomicAdd(&s.head_cnt[bh], 1u);
      }
    } else if (beyond) {
      float* F = s.scores + (int64_t)bh * a.L;
      const int end = min(chunk_key0 + s.chunk_keys, a.L);
      for (int j = chunk_key0 + threadIdx.x; j < end; j += kScoreThreads) F[j] = 0.f;
    } else {
      // ---------------- pass 2: column sums of exp2(logit - LSE) ----------
      if (!s.lse_given) {
        if (threadIdx.x == 0) {
          uint32_t spins = 0;
          while (load_coherent(&s.head_cnt[bh]) < (unsigned)(s.n_chunks + 1)) {
            __builtin_amdgcn_s_sleep(2);
            if (++spins > kSpinLimit) {
              atomicOr(s.status, 1u);
              break;
            }
          }
        }
        __syncthreads();
      }
      const float* lse = s.lse_given ? s.lse_in : s.lse2;
      const float lse_mul = s.lse_given ? s.lse_mul : 1.0f;
      for (int g0 = 0; g0 < a.P; g0 += kGroup) {
        const int gn = min(kGroup, a.P - g0);
        load_group(g0, gn);
        const int first = pos_g[0], last = pos_g[gn - 1];
        typename M::frag_t qf[PBW][kS];
        load_q(gn, qf);
        for (int i = threadIdx.x; i < kGroup; i += kScoreThreads)
          lse_g[i] = i < gn ? load_coherent(lse + (int64_t)bh * a.P + g0 + i) * lse_mul : INFINITY;
        __syncthreads();
        const float* my_lse = lse_g + ph * kHalfRows;
        // Column sums over this wave's proxies, accumulated across proxy
        // groups in the wave's own LDS row (same-wave LDS accesses are ordered).
        // This lane's partial column sums of the last four tiles; every
        // fourth tile they are reduced across lane groups and lane group g
        // stores tile t - 3 + g.
        float cs4[4];
        auto step2 = [&](int t, const typename M::frag_t (&kf)[kS], auto u_c) {
          constexpr int u = decltype(u_c)::value;
          const int key0 = key_base + t * 16;
          float cs = 0.f;
          if (key0 + 15 <= first) cs = pass2_tile<M, PBW, true>(kf, qf, key0, my_pos, g, r16, c2, my_lse);
          else if (key0 <= last) cs = pass2_tile<M, PBW, false>(kf, qf, key0, my_pos, g, r16, c2, my_lse);
          cs4[u % 4] = cs;
          if constexpr (u % 4 == 3) {
            const float z = colsum4(cs4[0], cs4[1], cs4[2], cs4[3]);
            const int idx = (t - 3) * 16 + lane;
            my_cols[idx] = (g0 == 0 ? 0.f : my_cols[idx]) + z;
          }
        };
        k_stream(step2);
      }
      __syncthreads();
      float* F = s.scores + (int64_t)bh * a.L;
      for (int idx = threadIdx.x; idx < s.chunk_keys; idx += kScoreThreads) {
        const int pair = idx / kKeysPerPair, j = idx % kKeysPerPair;
        const int key = chunk_key0 + idx;
        if (key < a.L) F[key] = col_lds[2 * pair][j] + col_lds[2 * pair + 1][j];
      }
    }
  }
}

// Zeroes the queue counter, the per-head counters and the status word.
__global__ void score_init_kernel(uint32_t* words, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) words[i] = 0u;
}

// ---------------------------------------------------------------------------
// Host-side launchers.

namespace {

template <typename T, int D, int PB>
hipError_t launch_score_t(const ScoreLaunch& L, hipStream_t stream) {
  auto kern = score_kernel<T, D, PB, kScoreTpwMax>;
  int per_cu = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kScoreThreads, 0);
  if (e != hipSuccess) return e;
  int dev = 0, cus = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  const int grid = std::max(1, std::min(L.sched.total_items, std::max(1, per_cu) * cus));
  const int init_blocks = std::max(1, std::min(64, (L.n_counter_words + 255) / 256));
  hipLaunchKernelGGL(score_init_kernel, dim3(init_blocks), dim3(256), 0, stream, L.sched.queue,
                     L.n_counter_words);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kScoreThreads), 0, stream, static_cast<const T*>(L.q),
                     static_cast<const T*>(L.k), L.args, L.sched);
  return hipGetLastError();
}

template <typename T, int D, int PBMAX>
hipError_t dispatch_pb(const ScoreLaunch& L, hipStream_t stream) {
  const int need = std::min((L.args.P + 15) / 16, PBMAX);
  if (need <= 2 || PBMAX == 2) return launch_score_t<T, D, 2>(L, stream);
  if constexpr (PBMAX >= 4) {
    if (need <= 4 || PBMAX == 4) return launch_score_t<T, D, 4>(L, stream);
  }
  if constexpr (PBMAX >= 8) return launch_score_t<T, D, 8>(L, stream);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_score(const ScoreLaunch& L, hipStream_t stream) {
  if (L.dtype == 1) {
    if (L.D == 128) return dispatch_pb<__bf16, 128, 8>(L, stream);
    return dispatch_pb<__bf16, 64, 8>(L, stream);
  }
  if (L.D == 128) return dispatch_pb<float, 128, 2>(L, stream);
  return dispatch_pb<float, 64, 4>(L, stream);
}

}  // namespace nacl
