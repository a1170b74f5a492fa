// Proxy-token scores F (NaCl, Section 5.1 F_score; Appendix A.7): for each
// (b, h), F[j] = sum_i exp(s * <Q[p_i], K[j]> - LSE_i) over proxies with
// p_i >= j, where LSE_i is the natural log-sum-exp of proxy row i over its
// causal keys 0..p_i.
//
// One persistent kernel runs two kinds of work items over key chunks of
// sched.chunk_keys keys, all on MFMA (v_mfma_f32_16x16x32_bf16 for bf16
// inputs, v_mfma_f32_16x16x4_f32 for fp32 inputs):
//   pass 1  base-2 (reference, sum) of every proxy row over the chunk's keys
//           -> per-chunk partials; the last chunk of a head to finish merges
//           the head's partials into its log-sum-exp
//   pass 2  exp2(logit - LSE) summed over the proxy rows for each key of the
//           chunk -> F (the column reduction of Appendix A.7's Algorithm 2).
//           Each key is owned by one wave: no atomics on F, so results are
//           bit-reproducible.
//
// The kernel streams K from HBM through a small LDS ring per wave: the
// chunk's 16-key tiles are dealt round-robin to the block's waves, and each
// wave works on its own tiles with all proxies of the current proxy group, so
// a K tile is used by exactly one wave and the waves of a block read
// neighbouring pieces of K at any moment.  Tiles are fetched by non-temporal
// buffer loads that write the wave's LDS slots directly, several tiles ahead
// of the MFMAs that consume them.  Pass 2 reads K a second time; a
// memory-side cache does not serve that re-read faster than HBM on this part,
// so K crosses HBM twice and the kernel is bound by 2 x |K| / HBM bandwidth.
//
// For bf16 inputs with D = 128 and at least 128 proxies, score_split_kernel
// (below) replaces this layout: the waves of a block share the tile ring and
// split the proxy group instead, which frees registers for four blocks per
// CU.  Everything else (queue, passes, merge, reproducibility) is the same.
//
// Work-groups take items from a queue counter in a fixed order: the pass-1
// items of head group g + lag come before the pass-2 items of head group g,
// so a pass-2 item rarely finds its head's log-sum-exp unpublished.  A
// pass-2 item waits (bounded spin) until its head's log-sum-exp is published;
// every item it waits on was taken from the queue earlier by a running
// work-group and never waits itself, so the wait always ends, whatever the
// number of resident work-groups.
//
// Fragment layout.  A 16x16 MFMA tile is indexed by (lane % 16) along M/N and
// by the lane group g = lane / 16 along the contraction.  The head dimension
// is cut into 64-byte pieces; piece c of a row holds d in [c*P, (c+1)*P)
// (P = 32 bf16 or 16 fp32 elements) and lane group g takes its 16-byte part
// [c*P + g*P/4, c*P + (g+1)*P/4).  For bf16 piece c is contraction step c (a
// 16x16x32 step consumes 8 elements per lane); for fp32 element i of the
// lane's part is step 4c + i (a 16x16x4 step consumes one).  Q and K use the
// same map, so the permutation of the contraction index cancels, and one
// 16-byte load instruction reads 64 contiguous bytes of each of 16 rows.  The
// 16x16 accumulator holds rows 4*g + e (e = 0..3) and column lane % 16.
//   pass 1 computes K_tile * Q_P^T: rows = keys, columns = proxies, so each
//          lane keeps the running statistics of one proxy per block.
//   pass 2 computes Q_P * K_tile^T: rows = proxies, columns = keys, so each
//          lane sums one key's column in registers and cross-lane moves
//          finish it.

#include <type_traits>

#include "device_common.h"
#include "gumbel.h"
#include "internal.h"

namespace nacl {

// Cache policy of the K tile loads: 2 = nt (streaming).  Each pass reads K
// once per proxy group and nothing re-reads it soon after.
#ifndef NACL_SCORE_K_AUX
#define NACL_SCORE_K_AUX 2
#endif
constexpr int kScoreKAux = NACL_SCORE_K_AUX;

// Word 3 of a raw buffer descriptor on gfx9-family parts (32-bit data format).
constexpr int kBufferRsrcWord3 = 0x00020000;
// A byte offset beyond every descriptor's range (num_records < 2^31) that
// cannot wrap when a lane offset below 2^30 is added.
constexpr uint32_t kOutOfRange = 0xC0000000u;

template <typename T, int D> struct Mma;

// Proxy blocks whose accumulators are live at once.
#ifndef NACL_SCORE_HALF
#define NACL_SCORE_HALF 4
#endif

template <int D> struct Mma<__bf16, D> {
  static constexpr int kSteps = D / 32;
  typedef bf16x8 frag_t;
  __device__ static void load(const __bf16* row, int g, frag_t (&f)[kSteps]) {
    const u32x4* p = reinterpret_cast<const u32x4*>(row + 8 * g);
#pragma unroll
    for (int s = 0; s < kSteps; ++s) f[s] = __builtin_bit_cast(frag_t, p[4 * s]);
  }
  __device__ static void zero(frag_t (&f)[kSteps]) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s) f[s] = __builtin_bit_cast(frag_t, u32x4{0u, 0u, 0u, 0u});
  }
  __device__ static f32x4 mma(frag_t a, frag_t b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  // This lane's fragment of one K row read directly through the head's
  // buffer descriptor at byte offset off (the whole offset is range-checked:
  // rows past the descriptor's end read as zeros).  Used by the exact path.
  __device__ static void load_k(__amdgpu_buffer_rsrc_t r, uint32_t off, frag_t (&f)[kSteps]) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s)
      f[s] = __builtin_bit_cast(frag_t, __builtin_amdgcn_raw_buffer_load_b128(r, off + 64u * s, 0, kScoreKAux));
  }
};

template <int D> struct Mma<float, D> {
  static constexpr int kSteps = D / 4;
  typedef float frag_t;
  __device__ static void load(const float* row, int g, frag_t (&f)[kSteps]) {
    const float4* p = reinterpret_cast<const float4*>(row + 4 * g);
#pragma unroll
    for (int s = 0; s < kSteps / 4; ++s) {
      const float4 v = p[4 * s];
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
  __device__ static void load_k(__amdgpu_buffer_rsrc_t r, uint32_t off, frag_t (&f)[kSteps]) {
#pragma unroll
    for (int c = 0; c < kSteps / 4; ++c) {
      const f32x4 v = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off + 64u * c, 0, kScoreKAux));
      f[4 * c + 0] = v[0];
      f[4 * c + 1] = v[1];
      f[4 * c + 2] = v[2];
      f[4 * c + 3] = v[3];
    }
  }
};

// One wave's 16-key tile of K staged in LDS by direct buffer->LDS loads
// (buffer_load_dwordx4 ... lds: each lane moves 16 bytes and one instruction
// fills 1 KB of LDS in lane order).  An instruction reads kRowsPerInstr whole
// rows, so its global accesses are contiguous.  Row r of the tile occupies
// kChunks consecutive 16-byte slots; slot x holds the row's chunk
// x ^ (r & kSwz), an XOR swizzle under which the 16 rows of a fragment read
// fall on distinct LDS banks.  Offsets go through the head's buffer
// descriptor (whole offset range-checked: rows at or past L read as zeros).
template <typename T, int D>
struct KStage {
  static constexpr int kRowBytes = D * (int)sizeof(T);
  static constexpr int kChunks = kRowBytes / 16;
  static constexpr int kRowsPerInstr = 64 / kChunks;
  static constexpr int kInstr = 16 / kRowsPerInstr;  // DMA instructions per tile
  static constexpr int kTileBytes = 16 * kRowBytes;
  static constexpr int kSwz = (kChunks < 16 ? kChunks : 16) - 1;
  // Ring depth per wave: 16 KB of tiles (two work-groups share a CU's LDS),
  // at least 2 and at most 8.
  static constexpr int kDepth = 16384 / kTileBytes < 2 ? 2 : (16384 / kTileBytes > 8 ? 8 : 16384 / kTileBytes);

  // Lane byte offsets inside a tile, one per DMA instruction.
  __device__ static void offsets(uint32_t row_bytes, int lane, uint32_t (&vo)[kInstr]) {
#pragma unroll
    for (int i = 0; i < kInstr; ++i) {
      const int row = i * kRowsPerInstr + lane / kChunks;
      const int c = (lane % kChunks) ^ (row & kSwz);
      vo[i] = (uint32_t)row * row_bytes + (uint32_t)c * 16u;
    }
  }
  __device__ static void issue(__amdgpu_buffer_rsrc_t rsrc, const uint32_t (&vo)[kInstr], uint32_t tile_byte,
                               unsigned char* dst) {
#pragma unroll
    for (int i = 0; i < kInstr; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(dst + i * 1024), 16,
                                               vo[i] + tile_byte, 0, 0, kScoreKAux);
  }
  // Fragment of row r16 (lane group g): 16-byte chunk 4*c + g of piece c.
  template <typename M>
  __device__ static void frag(const unsigned char* tile, int r16, int g, typename M::frag_t (&f)[M::kSteps]) {
    if constexpr (std::is_same_v<T, __bf16>) {
#pragma unroll
      for (int c = 0; c < M::kSteps; ++c) {
        const int x = (4 * c + g) ^ (r16 & kSwz);
        f[c] = __builtin_bit_cast(typename M::frag_t, *reinterpret_cast<const u32x4*>(tile + (r16 * kChunks + x) * 16));
      }
    } else {
#pragma unroll
      for (int c = 0; c < M::kSteps / 4; ++c) {
        const int x = (4 * c + g) ^ (r16 & kSwz);
        const f32x4 v = *reinterpret_cast<const f32x4*>(tile + (r16 * kChunks + x) * 16);
        f[4 * c + 0] = v[0];
        f[4 * c + 1] = v[1];
        f[4 * c + 2] = v[2];
        f[4 * c + 3] = v[3];
      }
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

constexpr int kScoreThreads = 64 * kScoreWaves;

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
  int psl;    // group of proxy rows (0 unless the items are split along the rows)
};

// Item i of the queue order described at the top of the file.
__device__ __forceinline__ ItemRef decode_item(const ScoreSched& s, int i) {
  const int U = s.n_chunks * s.n_psplit;         // items per head and pass
  const int S = s.heads_per_group * U;           // items per group and pass
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
  const int u = r % U;
  return ItemRef{kind, group * s.heads_per_group + r / U, u / s.n_psplit, u % s.n_psplit};
}

// Proxy row r of a K/V head is proxy r / qg of query head r % qg of its
// group (rows sorted by position, so positions never decrease along the
// rows).  Returns the row's position and sets qrow to the element offset of
// its query from the group's first query head.
__device__ __forceinline__ int row_position(const ScoreArgs& a, int r, int64_t& qrow) {
  const int ip = r / a.qg, e = r - ip * a.qg;
  const int p = a.pos[ip];
  qrow = (int64_t)e * a.qs[1] + (int64_t)p * a.qs[2];
  return p;
}

// Index of row r's log-sum-exp: the library's own [B*H, P] rows, or the
// caller's [B, H * qg, P] per query head.
__device__ __forceinline__ int64_t lse_index(const ScoreArgs& a, const ScoreSched& s, int bh, int r) {
  if (!s.lse_given) return (int64_t)bh * a.P + r;
  const int ip = r / a.qg, e = r - ip * a.qg;
  return ((int64_t)bh * a.qg + e) * a.P0 + ip;
}

// Logits of one 16-key tile for proxy blocks [P0, P0 + N) into acc[0 .. N):
// pass-1 orientation (rows = keys) when KROWS, pass-2 orientation (rows =
// proxies) otherwise.
template <typename M, int PB, int P0, int N, bool KROWS, int NA>
__device__ __forceinline__ void tile_logits(const typename M::frag_t (&kf)[M::kSteps],
                                            const typename M::frag_t (&qf)[PB][M::kSteps], f32x4 (&acc)[NA]) {
#pragma unroll
  for (int j = 0; j < N; ++j) {
    acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < M::kSteps; ++ks)
      acc[j] = KROWS ? M::mma(kf[ks], qf[P0 + j][ks], acc[j]) : M::mma(qf[P0 + j][ks], kf[ks], acc[j]);
  }
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

// An integer the compiler cannot see through: LDS reads indexed with it are
// re-issued where they stand instead of being hoisted out of the tile loop
// into (scarce) registers.
__device__ __forceinline__ int opaque(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Maximum over the 4 lane groups (same r16) of a per-lane value.
__device__ __forceinline__ float max_over_groups(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float sum_over_groups(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}

// Work-group layout: kScoreWaves waves, each owning s.tpw consecutive tiles
// of 16 keys (at most TPWMAX) and the Q fragments of the whole proxy group of
// 16*PB proxies.  An item spans kScoreWaves * s.tpw * 16 keys.
template <typename T, int D, int PB, int TPWMAX>
__global__ __launch_bounds__(kScoreThreads)
__attribute__((amdgpu_waves_per_eu(kScoreWavesPerSimd, kScoreWavesPerSimd))) void score_kernel(
    const T* __restrict__ q, const T* __restrict__ k, ScoreArgs a, ScoreSched s) {
  using M = Mma<T, D>;
  using frag_t = typename M::frag_t;
  constexpr int kS = M::kSteps;
  constexpr int kGroup = 16 * PB;        // proxies per group
  constexpr int kMaxKeysPerWave = TPWMAX * 16;
  constexpr int kHalf = PB > NACL_SCORE_HALF ? NACL_SCORE_HALF : PB;  // live accumulators (exact path)
  constexpr int kUnroll = KStage<T, D>::kDepth > 4 ? KStage<T, D>::kDepth : 4;  // tiles per unrolled step
  static_assert(kUnroll % KStage<T, D>::kDepth == 0 && kScoreTpwMin % kUnroll == 0, "tiles per wave vs ring");
  __shared__ int item_s, last_s;
  __shared__ int pos_g[kGroup];
  __shared__ int64_t qrow_g[kGroup];  // element offset of each row's query from qb
  __shared__ float2 red[kScoreWaves][kGroup];
  __shared__ float2 mrg[kScoreThreads];
  __shared__ float col_lds[kScoreWaves][kMaxKeysPerWave];
  __shared__ __attribute__((aligned(16))) float lse_g[kGroup];
  using KS = KStage<T, D>;
  constexpr int kDepth = KS::kDepth;
  // One array per ring slot: distinct objects let the compiler see that a
  // DMA into one slot does not alias reads of another, so it does not wait
  // for outstanding DMA before every LDS read.
#define NACL_KSLOT(i) \
  __shared__ __attribute__((aligned(16))) unsigned char kslot##i[kScoreWaves][kDepth > i ? KS::kTileBytes : 16];
  NACL_KSLOT(0) NACL_KSLOT(1) NACL_KSLOT(2) NACL_KSLOT(3) NACL_KSLOT(4) NACL_KSLOT(5) NACL_KSLOT(6) NACL_KSLOT(7)
#undef NACL_KSLOT

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const float c2 = a.c2;
  float* my_cols = col_lds[wave];
  const uint32_t row_bytes = (uint32_t)(a.ks[2] * (int64_t)sizeof(T));
  uint32_t vo[KStage<T, D>::kInstr];
  KStage<T, D>::offsets(row_bytes, lane, vo);
  const uint32_t voff = (uint32_t)r16 * row_bytes + 16u * (uint32_t)g;  // direct fragment loads (exact path)

  for (;;) {
    __syncthreads();
    if (threadIdx.x == 0) item_s = (int)atomicAdd(s.queue, 1u);
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(item_s);
    if (item >= s.total_items) break;
    const ItemRef it = decode_item(s, item);
    const int bh = it.bh, b = bh / a.H, h = bh % a.H;
    const T* qb = q + b * a.qs[0] + (int64_t)h * a.qg * a.qs[1];  // first query head of the group
    const T* kb = k + b * a.ks[0] + h * a.ks[1];
    const int TPW = s.tpw;  // multiple of kUnroll, at most TPWMAX
    const int chunk_key0 = it.chunk * s.chunk_keys;
    // The chunk's 16-key tiles are dealt round-robin to the waves: tile t of
    // this wave holds keys tile_key(t) .. tile_key(t) + 15, so the waves of a
    // block stream neighbouring 4 KB pieces of K at any moment (better DRAM
    // page locality than one contiguous range per wave).
    auto tile_key = [&](int t) -> int { return chunk_key0 + (t * kScoreWaves + wave) * 16; };
    const bool beyond = chunk_key0 > a.p_last;  // no proxy sees these keys
    // Inside a whole eviction the column reduction also draws the chunk's
    // Gumbel keys for the selection that follows, from the chunk's scores
    // f_of(idx) (the values just written to F): one Philox block of four
    // keys per thread and step.
    auto chunk_gumbel_keys = [&](auto&& f_of) {
      uint32_t* gk = s.gkeys + (int64_t)bh * a.L;
      for (int q4 = 4 * (int)threadIdx.x; q4 < s.chunk_keys; q4 += 4 * kScoreThreads) {
        const int j0 = chunk_key0 + q4;
        if (j0 >= a.L) break;
        const int n = min(4, a.L - j0);
        float fv[4] = {0.f, 0.f, 0.f, 0.f};
        for (int e = 0; e < n; ++e) fv[e] = f_of(q4 + e);
        uint32_t kv[4];
        gumbel_block_keys(s.g_mode, j0, n, b, h, s.g_layer, s.g_k0, s.g_k1, fv, kv);
        for (int e = 0; e < n; ++e) gk[j0 + e] = kv[e];
      }
    };
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<T*>(kb), (short)0, (int)((uint32_t)(a.L - 1) * row_bytes + (uint32_t)(D * sizeof(T))),
        kBufferRsrcWord3);

    // Streams the wave's TPW tiles through its own LDS ring of kDepth slots:
    // tiles t + 1 .. t + kDepth - 1 are in flight while tile t is used.  Proxy blocks go
    // in batches of kHalf (MFMAs, then their VALU work) so at most kHalf
    // accumulators are live; the other wave on the SIMD fills the MFMA and
    // VALU gaps.  Only this wave touches its ring, so no barrier is involved.
    // The DMA is unconditional (a tile past the wave's range gets an offset
    // beyond the descriptor and reads zeros without touching memory), so
    // every wait count is static.
    auto tile_byte = [&](int t) -> uint32_t {
      return t < TPW ? (uint32_t)tile_key(t) * row_bytes : kOutOfRange;
    };
    auto slot = [&](auto u_c) -> unsigned char* {
      constexpr int u = decltype(u_c)::value % kDepth;
      if constexpr (u == 0) return kslot0[wave];
      else if constexpr (u == 1) return kslot1[wave];
      else if constexpr (u == 2) return kslot2[wave];
      else if constexpr (u == 3) return kslot3[wave];
      else if constexpr (u == 4) return kslot4[wave];
      else if constexpr (u == 5) return kslot5[wave];
      else if constexpr (u == 6) return kslot6[wave];
      else return kslot7[wave];
    };
    auto k_stream = [&](auto&& mfma, auto&& valu) {
      f32x4 acc[kHalf];
      static_for<kDepth - 1>([&](auto u_c) { KS::issue(rsrc, vo, tile_byte(decltype(u_c)::value), slot(u_c)); });
#pragma unroll 1
      for (int t = 0; t < TPW; t += kUnroll) {
        static_for<kUnroll>([&](auto u_c) {
          constexpr int u = decltype(u_c)::value;
          const int tt = t + u;
          // The slot of tile tt - 1 was read in the previous step: refill it
          // before waiting, so kDepth - 1 tiles stay in flight across the
          // wait.  The LDS wait first makes those reads complete (the
          // compiler may otherwise issue the refill while some are queued).
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          KS::issue(rsrc, vo, tile_byte(tt + kDepth - 1), slot(std::integral_constant<int, u + kDepth - 1>{}));
          asm volatile("s_waitcnt vmcnt(%0)" ::"n"(KS::kInstr * (kDepth - 1)) : "memory");
          frag_t kf[kS];
          KS::template frag<M>(slot(u_c), r16, g, kf);
          static_for<PB / kHalf>([&](auto h_c) {
            using P0 = std::integral_constant<int, decltype(h_c)::value * kHalf>;
            using N = std::integral_constant<int, kHalf>;
            mfma(tt, kf, acc, P0{}, N{});
            valu(tt, acc, u_c, P0{}, N{});
          });
        });
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    };
    // Positions of the proxy group [g0, g0 + gn), -1 past its end.
    auto load_group = [&](int g0, int gn) {
      __syncthreads();
      for (int i = threadIdx.x; i < kGroup; i += kScoreThreads) pos_g[i] = i < gn ? row_position(a, g0 + i, qrow_g[i]) : -1;
      __syncthreads();
    };
    // The Q fragments of the whole group (zeros past its end).
    auto load_q = [&](int gn, frag_t (&qf)[PB][kS]) {
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        const int i = 16 * pb + r16;
        if (i < gn) M::load(qb + qrow_g[i], g, qf[pb]);
        else M::zero(qf[pb]);
      }
    };

    if (it.kind == 1) {
      // ---------------- pass 1: per-chunk (reference, sum) of every proxy row
      float2* part = s.partials + ((int64_t)bh * s.n_chunks + it.chunk) * a.P;
      if (beyond)
        for (int i = threadIdx.x; i < a.P; i += kScoreThreads)
          store_coherent(part + i, make_float2(-INFINITY, 0.f));
      for (int g0 = 0; g0 < (beyond ? 0 : a.P); g0 += kGroup) {
        const int gn = min(kGroup, a.P - g0);
        load_group(g0, gn);
        const int first = pos_g[0], last = pos_g[gn - 1];
        frag_t qf[PB][kS];
        load_q(gn, qf);
        // Per proxy block: base-2 reference (the scaled maximum of the wave's
        // first tile, 0 if that tile shows the proxy nothing) and the running
        // sum of exp2(logit * c2 - ref) over this lane's keys.  Visibility is a
        // prefix of the keys, so a proxy that sees nothing of the first tile
        // sees nothing of the wave's keys; one that sees something has a sum of
        // at least 1 (its reference key contributes exp2(0)).
        float ref[PB], sm[PB];
#pragma unroll
        for (int pb = 0; pb < PB; ++pb) {
          ref[pb] = 0.f;
          sm[pb] = 0.f;
        }
        auto mfma1 = [&](int t, const frag_t (&kf)[kS], auto& acc, auto p0_c, auto n_c) {
          if (tile_key(t) > last) return;  // no proxy of the group sees this tile
          tile_logits<M, PB, decltype(p0_c)::value, decltype(n_c)::value, true>(kf, qf, acc);
        };
        // VALU work of one tile; FULL tiles (every key visible to every proxy
        // of the group, the common case) carry no masking at all.
        auto valu1_body = [&](int t, const auto& acc, auto p0_c, auto n_c, auto full_c) {
          constexpr int P0 = decltype(p0_c)::value, N = decltype(n_c)::value;
          constexpr bool FULL = decltype(full_c)::value;
          const int key0 = tile_key(t);
          const int* pos_l = pos_g + opaque(r16);
#pragma unroll
          for (int pb = P0; pb < P0 + N; ++pb) {
            bool vis[4];
            if constexpr (!FULL) {
              const int pi = pos_l[16 * pb];
#pragma unroll
              for (int e = 0; e < 4; ++e) vis[e] = key0 + 4 * g + e <= pi;
            }
            if (t == 0) {
              float mx = -INFINITY;
#pragma unroll
              for (int e = 0; e < 4; ++e) mx = (FULL || vis[e]) ? fmaxf(mx, acc[pb - P0][e]) : mx;
              mx = max_over_groups(mx);
              ref[pb] = mx != -INFINITY ? mx * c2 : 0.f;
            }
            float x[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = fast_exp2(fmaf(acc[pb - P0][e], c2, -ref[pb]));
            if constexpr (!FULL) {
#pragma unroll
              for (int e = 0; e < 4; ++e) x[e] = vis[e] ? x[e] : 0.f;
            }
            sm[pb] += (x[0] + x[1]) + (x[2] + x[3]);
          }
        };
        auto valu1 = [&](int t, const auto& acc, auto, auto p0_c, auto n_c) {
          const int key0 = tile_key(t);
          if (key0 > last) return;
          if (key0 + 15 <= first) valu1_body(t, acc, p0_c, n_c, std::true_type{});
          else valu1_body(t, acc, p0_c, n_c, std::false_type{});
        };
        k_stream(mfma1, valu1);
        // Row sums over the four lane groups; a sum that overflowed (a key far
        // above the first tile's maximum) is recomputed with the exact maximum.
        bool bad = false;
#pragma unroll
        for (int pb = 0; pb < PB; ++pb) {
          sm[pb] = sum_over_groups(sm[pb]);
          bad |= !(sm[pb] <= 3.0e38f);
        }
        if (__builtin_amdgcn_ballot_w64(bad)) {
          // Exact path: maximum over every visible key of the wave, then the sums.
          float mx[PB];
#pragma unroll
          for (int pb = 0; pb < PB; ++pb) mx[pb] = -INFINITY;
          for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
            for (int pb = 0; pb < PB; ++pb) sm[pb] = 0.f;
            for (int t = 0; t < TPW; ++t) {
              const int key0 = tile_key(t);
              if (key0 > last) break;
              frag_t kf[kS];
              M::load_k(rsrc, voff + (uint32_t)key0 * row_bytes, kf);  // direct loads: rare path
              static_for<PB / kHalf>([&](auto h_c) {
                constexpr int P0 = decltype(h_c)::value * kHalf;
                f32x4 acc[kHalf];
                tile_logits<M, PB, P0, kHalf, true>(kf, qf, acc);
#pragma unroll
                for (int pb = P0; pb < P0 + kHalf; ++pb) {
                  const int pi = pos_g[16 * pb + r16];
#pragma unroll
                  for (int e = 0; e < 4; ++e) {
                    const bool v = key0 + 4 * g + e <= pi;
                    if (pass == 0) mx[pb] = v ? fmaxf(mx[pb], acc[pb - P0][e]) : mx[pb];
                    else sm[pb] += v ? fast_exp2(fmaf(acc[pb - P0][e], c2, -ref[pb])) : 0.f;
                  }
                }
              });
            }
            if (pass == 0) {
#pragma unroll
              for (int pb = 0; pb < PB; ++pb) {
                mx[pb] = max_over_groups(mx[pb]);
                ref[pb] = mx[pb] != -INFINITY ? mx[pb] * c2 : 0.f;
              }
            }
          }
#pragma unroll
          for (int pb = 0; pb < PB; ++pb) sm[pb] = sum_over_groups(sm[pb]);
        }
        if (g == 0) {
#pragma unroll
          for (int pb = 0; pb < PB; ++pb)
            red[wave][16 * pb + r16] = sm[pb] > 0.f ? make_float2(ref[pb], sm[pb]) : make_float2(-INFINITY, 0.f);
        }
        __syncthreads();
        for (int i = threadIdx.x; i < gn; i += kScoreThreads) {
          float2 r = red[0][i];
#pragma unroll
          for (int w = 1; w < kScoreWaves; ++w) lse_merge(r.x, r.y, red[w][i].x, red[w][i].y);
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
      if (s.gkeys) chunk_gumbel_keys([](int) { return 0.f; });
    } else {
      // ---------------- pass 2: column sums of exp2(logit - LSE) ----------
      if (!s.lse_given) {
        if (threadIdx.x == 0) {
          uint32_t spins = 0;
          while (load_coherent(&s.head_cnt[bh]) < (unsigned)(s.n_chunks + 1)) {
            __builtin_amdgcn_s_sleep(2);
            if (++spins > kSpinLimit) {
              atomicOr(s.status, 1u);
              atomicOr(s.status + 1, 1u);
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
        frag_t qf[PB][kS];
        load_q(gn, qf);
        for (int i = threadIdx.x; i < kGroup; i += kScoreThreads)
          lse_g[i] = i < gn ? load_coherent(lse + lse_index(a, s, bh, g0 + i)) * lse_mul : INFINITY;
        __syncthreads();
        // This lane's partial column sums of the last four tiles; every
        // fourth tile they are reduced across lane groups and lane group g
        // stores tile t - 3 + g (accumulated across proxy groups in the
        // wave's own LDS row; same-wave LDS accesses are ordered).
        float cs4[4];
        auto mfma2 = [&](int t, const frag_t (&kf)[kS], auto& acc, auto p0_c, auto n_c) {
          if (tile_key(t) > last) return;
          tile_logits<M, PB, decltype(p0_c)::value, decltype(n_c)::value, false>(kf, qf, acc);
        };
        // This lane's share of its key's column sum over blocks [P0, P0 + N);
        // FULL tiles carry no masking.
        auto valu2_body = [&](int key0, const auto& acc, auto p0_c, auto n_c, auto full_c) -> float {
          constexpr int P0 = decltype(p0_c)::value, N = decltype(n_c)::value;
          constexpr bool FULL = decltype(full_c)::value;
          const int o = opaque(4 * g);
          const float* lse_l = lse_g + o;
          const int* pos_l = pos_g + o;
          float cs = 0.f;
          f32x4 lrs[N];
#pragma unroll
          for (int pb = P0; pb < P0 + N; ++pb) lrs[pb - P0] = *reinterpret_cast<const f32x4*>(lse_l + 16 * pb);
#pragma unroll
          for (int pb = P0; pb < P0 + N; ++pb) {
            const f32x4 lr = lrs[pb - P0];
            float x[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = fast_exp2(fmaf(acc[pb - P0][e], c2, -lr[e]));
            if constexpr (!FULL) {
#pragma unroll
              for (int e = 0; e < 4; ++e) x[e] = key0 + r16 <= pos_l[16 * pb + e] ? x[e] : 0.f;
            }
            cs += (x[0] + x[1]) + (x[2] + x[3]);
          }
          return cs;
        };
        auto valu2 = [&](int t, const auto& acc, auto u_c, auto p0_c, auto n_c) {
          constexpr int u = decltype(u_c)::value;
          constexpr int P0 = decltype(p0_c)::value, N = decltype(n_c)::value;
          const int key0 = tile_key(t);
          float cs = P0 == 0 ? 0.f : cs4[u % 4];
          if (key0 <= last) {
            if (key0 + 15 <= first) cs += valu2_body(key0, acc, p0_c, n_c, std::true_type{});
            else cs += valu2_body(key0, acc, p0_c, n_c, std::false_type{});
          }
          cs4[u % 4] = cs;
          if constexpr (u % 4 == 3 && P0 + N == PB) {
            const float z = colsum4(cs4[0], cs4[1], cs4[2], cs4[3]);
            const int idx = (t - 3) * 16 + lane;
            my_cols[idx] = (g0 == 0 ? 0.f : my_cols[idx]) + z;
          }
        };
        k_stream(mfma2, valu2);
      }
      __syncthreads();
      float* F = s.scores + (int64_t)bh * a.L;
      // Key chunk_key0 + idx sits in tile idx / 16 of the chunk: wave
      // (idx / 16) % kScoreWaves, that wave's tile (idx / 16) / kScoreWaves.
      auto col_of = [&](int idx) -> float {
        const int tile = idx >> 4;
        return col_lds[tile % kScoreWaves][(tile / kScoreWaves) * 16 + (idx & 15)];
      };
      for (int idx = threadIdx.x; idx < s.chunk_keys; idx += kScoreThreads) {
        const int key = chunk_key0 + idx;
        if (key < a.L) F[key] = col_of(idx);
      }
      if (s.gkeys) chunk_gumbel_keys(col_of);
    }
  }
}

// Zeroes the queue counter, the call's health word and the per-head
// counters; the sticky health word (word 2) is left as it is.
__global__ void score_init_kernel(uint32_t* words, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    if (i != 2) words[i] = 0u;
}

// ---------------------------------------------------------------------------
// Few proxy rows (at most score_rows_max rows per K/V head, log-sum-exp
// computed here).  With one to sixteen rows a key's logits take 4 to 64
// bytes, less than its K row, so they are stored instead of reading K again:
//   score_rows_logits_kernel  one work-group per chunk of a head (64 to
//     kRowsChunkMax keys, sized so that the work-groups fill whole rounds of
//     the resident ones); each wave streams a quarter of it through its own LDS
//     ring (buffer loads that write LDS, as in the kernels above), computes
//     their logits (16 keys per MFMA tile, rows = keys, columns = the proxy
//     rows) and keeps them in registers; then it stores them and the
//     chunk's base-2 (maximum, sum) per row, taken against the chunk's exact
//     maximum, so no term exceeds 1;
//   score_rows_column_kernel  merges a head's partials into its log-sum-exp
//     (each work-group of the head for itself), then F[j] = sum over the
//     rows that see key j of exp2(logit * c2 - LSE) from the stored logits
//     (rows in order), and inside a whole eviction the Gumbel keys of the
//     four keys a thread owns.
// No work-group waits for another: no queue, no counter, no spin.

template <typename T, int D>
__global__ __launch_bounds__(kScoreThreads) void score_rows_logits_kernel(const T* __restrict__ q,
                                                                         const T* __restrict__ k, ScoreArgs a,
                                                                         ScoreSched s) {
  using M = Mma<T, D>;
  using frag_t = typename M::frag_t;
  using KS = KStage<T, D>;
  constexpr int kS = M::kSteps;
  constexpr int kTiles = kRowsChunkMax / 16 / kScoreWaves;  // most tiles of 16 keys per wave
  // Ring slots per wave: 12 KB of tiles (at least two), so that three
  // work-groups share a CU's LDS.
  constexpr int kDepth = 12288 / KS::kTileBytes < 2 ? 2 : (12288 / KS::kTileBytes > 8 ? 8 : 12288 / KS::kTileBytes);
  __shared__ float red[kScoreWaves][16];
  // One array per ring slot, so that the compiler sees a DMA into one slot
  // does not alias reads of another.
#define NACL_RSLOT(i) \
  __shared__ __attribute__((aligned(16))) unsigned char rslot##i[kScoreWaves][kDepth > i ? KS::kTileBytes : 16];
  NACL_RSLOT(0) NACL_RSLOT(1) NACL_RSLOT(2) NACL_RSLOT(3) NACL_RSLOT(4) NACL_RSLOT(5) NACL_RSLOT(6) NACL_RSLOT(7)
#undef NACL_RSLOT
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int chunk = blockIdx.x, bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const int tpw = s.chunk_keys / (16 * kScoreWaves);  // this launch's tiles per wave, 1 .. kTiles
  // The first work-group zeroes the workspace's counter words (the call's
  // health word, the selection's synchronisation words), all but the sticky
  // health word (word 2); nothing in this launch reads them.
  if (chunk == 0 && bh == 0)
    for (int i = threadIdx.x; i < s.n_clear; i += kScoreThreads)
      if (i != 2) s.queue[i] = 0u;
  const int key_c0 = chunk * s.chunk_keys;
  float2* part = s.partials + ((int64_t)bh * s.n_chunks + chunk) * a.P;
  const float c2 = a.c2;
  if (key_c0 > a.p_last) {
    // No row sees these keys: an empty partial, no logits.
    for (int i = threadIdx.x; i < a.P; i += kScoreThreads) part[i] = make_float2(-INFINITY, 0.f);
  } else {
    // This lane's proxy row r16 (none past the last row: position -1, so no
    // key is visible to it; positions come with the launch) and its query
    // fragments, loaded before the K stream (vector memory loads complete in
    // order, so the stream's waits cover them).
    const bool row_ok = r16 < a.P;
    const int pr = row_ok ? s.row_pos[r16] : -1;
    frag_t qf[kS];
    const T* qb = q + b * a.qs[0] + (int64_t)h * a.qg * a.qs[1];
    if (row_ok) M::load(qb + (int64_t)(r16 % a.qg) * a.qs[1] + (int64_t)pr * a.qs[2], g, qf);
    else M::zero(qf);
    const T* kb = k + b * a.ks[0] + h * a.ks[1];
    const uint32_t row_bytes = (uint32_t)(a.ks[2] * (int64_t)sizeof(T));
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<T*>(kb), (short)0, (int)((uint32_t)(a.L - 1) * row_bytes + (uint32_t)(D * sizeof(T))),
        kBufferRsrcWord3);
    uint32_t vo[KS::kInstr];
    KS::offsets(row_bytes, lane, vo);
    const int key_w0 = key_c0 + wave * tpw * 16;  // the wave's tpw * 16 consecutive keys
    // Tiles past the wave's range or past L get an offset beyond the
    // descriptor: the DMA reads zeros without touching memory, so every
    // wait count below is static.
    auto tile_byte = [&](int t) -> uint32_t {
      const int key0 = key_w0 + 16 * t;
      return t < tpw && key0 < a.L ? (uint32_t)key0 * row_bytes : kOutOfRange;
    };
    auto slot = [&](auto u_c) -> unsigned char* {
      constexpr int u = decltype(u_c)::value % kDepth;
      if constexpr (u == 0) return rslot0[wave];
      else if constexpr (u == 1) return rslot1[wave];
      else if constexpr (u == 2) return rslot2[wave];
      else if constexpr (u == 3) return rslot3[wave];
      else if constexpr (u == 4) return rslot4[wave];
      else if constexpr (u == 5) return rslot5[wave];
      else if constexpr (u == 6) return rslot6[wave];
      else return rslot7[wave];
    };
    // The wave's logits stay in registers (lg[t][e]: key key_w0 + 16 t +
    // 4 g + e, row r16) until the stream ends; the stream issues no other
    // vector memory operation, so its wait counts are exact.
    f32x4 lg[kTiles];
    static_for<kDepth - 1>([&](auto u_c) { KS::issue(rsrc, vo, tile_byte(decltype(u_c)::value), slot(u_c)); });
    static_for<kTiles>([&](auto t_c) {
      constexpr int t = decltype(t_c)::value;
      // The slot of tile t - 1 was read in the previous step: refill it
      // before waiting, so kDepth - 1 tiles stay in flight.  The LDS wait
      // first makes those reads complete (the compiler may otherwise issue
      // the refill while the last of them are still queued).
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      KS::issue(rsrc, vo, tile_byte(t + kDepth - 1), slot(std::integral_constant<int, t + kDepth - 1>{}));
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(KS::kInstr * (kDepth - 1)) : "memory");
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      if (t < tpw) {
        frag_t kf[kS];
        KS::template frag<M>(slot(t_c), r16, g, kf);
#pragma unroll
        for (int ks = 0; ks < kS; ++ks) acc = M::mma(kf[ks], qf[ks], acc);
      }
      lg[t] = acc;
    });
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    // Store the logits (the row stride is a multiple of 4, so a group of four
    // keys reaching past L stays in the row's padding).
    if (row_ok) {
      float* lrow = s.logits + ((int64_t)bh * a.P + r16) * s.logits_stride;
#pragma unroll
      for (int t = 0; t < kTiles; ++t) {
        const int key = key_w0 + 16 * t + 4 * g;
        if (t < tpw && key < a.L) *reinterpret_cast<f32x4*>(lrow + key) = lg[t];
      }
    }
    // The chunk's maximum per row over the keys the row sees (a prefix of
    // the keys), then the sum of exp2(logit * c2 - maximum * c2).
    // Keys of tiles past tpw belong to the next wave: none counts here.
    const int pw = min(pr, key_w0 + 16 * tpw - 1);
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < kTiles; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) mx = key_w0 + 16 * t + 4 * g + e <= pw ? fmaxf(mx, lg[t][e]) : mx;
    mx = max_over_groups(mx);
    if (g == 0) red[wave][r16] = mx;
    __syncthreads();
    float bm = red[0][r16];
#pragma unroll
    for (int w = 1; w < kScoreWaves; ++w) bm = fmaxf(bm, red[w][r16]);
    const float ref = bm != -INFINITY ? bm * c2 : 0.f;
    float sm = 0.f;
#pragma unroll
    for (int t = 0; t < kTiles; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        sm += key_w0 + 16 * t + 4 * g + e <= pw ? fast_exp2(fmaf(lg[t][e], c2, -ref)) : 0.f;
    sm = sum_over_groups(sm);
    __syncthreads();  // every wave has read red
    if (g == 0) red[wave][r16] = sm;
    __syncthreads();
    // Thread r < P (lane r of wave 0) holds row r's reference.
    if (threadIdx.x < a.P) {
      const int r = threadIdx.x;
      const float tot = ((red[0][r] + red[1][r]) + red[2][r]) + red[3][r];
      part[r] = tot > 0.f ? make_float2(ref, tot) : make_float2(-INFINITY, 0.f);
    }
  }
}

__global__ __launch_bounds__(kScoreThreads) void score_rows_column_kernel(ScoreArgs a, ScoreSched s) {
  __shared__ float lse_s[16];
  __shared__ int pos_s[16];
  __shared__ float2 mrg[kScoreThreads];
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  {
    // The head's log-sum-exp per row from the chunks' partials (every
    // work-group of the head merges them itself): `split` threads share a
    // row, each taking every split-th chunk with kMB loads in flight, and
    // they combine through LDS in thread order.
    const float2* hp = s.partials + (int64_t)bh * s.n_chunks * a.P;
    constexpr int kMB = 8;
    // Enough threads per row for one batch of kMB loads each, at most
    // kScoreThreads / P (the combine below is serial in split).
    const int split = min(kScoreThreads / a.P, (s.n_chunks + kMB - 1) / kMB);
    const int i = (int)threadIdx.x % a.P, pi = (int)threadIdx.x / a.P;
    float mm = -INFINITY, ss = 0.f;
    if (pi < split) {
      for (int c0 = pi; c0 < s.n_chunks; c0 += kMB * split) {
        float2 v[kMB];
#pragma unroll
        for (int u = 0; u < kMB; ++u) {
          const int c = c0 + u * split;
          v[u] = c < s.n_chunks ? hp[(int64_t)c * a.P + i] : make_float2(-INFINITY, 0.f);
        }
#pragma unroll
        for (int u = 0; u < kMB; ++u) lse_merge(mm, ss, v[u].x, v[u].y);
      }
    }
    mrg[threadIdx.x] = make_float2(mm, ss);
    __syncthreads();
    if (threadIdx.x < a.P) {
      for (int pp = 1; pp < split; ++pp) {
        const float2 r = mrg[threadIdx.x + pp * a.P];
        lse_merge(mm, ss, r.x, r.y);
      }
      const float l2 = mm + __log2f(ss);
      lse_s[threadIdx.x] = l2;
      pos_s[threadIdx.x] = s.row_pos[threadIdx.x];
      if (blockIdx.x == 0) s.lse2[(int64_t)bh * a.P + threadIdx.x] = l2;
    }
    __syncthreads();
  }
  const int j0 = 4 * (blockIdx.x * kScoreThreads + (int)threadIdx.x);
  if (j0 >= a.L) return;
  const int n = min(4, a.L - j0);
  float fv[4] = {0.f, 0.f, 0.f, 0.f};
  if (j0 <= a.p_last) {
    for (int r = 0; r < a.P; ++r) {
      const int pr = pos_s[r];
      if (j0 > pr) continue;  // the row sees none of the four keys
      const f32x4 x = *reinterpret_cast<const f32x4*>(s.logits + ((int64_t)bh * a.P + r) * s.logits_stride + j0);
      const float l2 = lse_s[r];
#pragma unroll
      for (int e = 0; e < 4; ++e) fv[e] += j0 + e <= pr ? fast_exp2(fmaf(x[e], a.c2, -l2)) : 0.f;
    }
  }
  float* F = s.scores + (int64_t)bh * a.L + j0;
  for (int e = 0; e < n; ++e) F[e] = fv[e];
  if (s.gkeys) {
    uint32_t kv[4];
    gumbel_block_keys(s.g_mode, j0, n, b, h, s.g_layer, s.g_k0, s.g_k1, fv, kv);
    uint32_t* gk = s.gkeys + (int64_t)bh * a.L + j0;
    for (int e = 0; e < n; ++e) gk[e] = kv[e];
  }
}

// ---------------------------------------------------------------------------
// Proxy-split variant: bf16, D = 128, groups of 128 proxies.  The four waves
// of a block share one LDS ring of K tiles and split the proxy group: wave w
// takes proxies [32w, 32w + 32) of every tile, so it holds a quarter of the
// group's Q fragments and four blocks fit on a CU (more waves to hide the
// MFMA, exponential and LDS latencies behind the K stream).  Each wave issues
// one of a tile's four DMA instructions; one block barrier per tile makes the
// whole tile visible and guarantees that the slot refilled next was read by
// every wave one step earlier.  An item is kSplitChunkKeys keys; pass 1 needs
// no merge across waves (each wave owns its proxies' sums over all the
// item's keys), pass 2 adds the four waves' partial column sums every four
// tiles through a small stage.
#ifndef NACL_SPLIT_DEPTH
#define NACL_SPLIT_DEPTH 4
#endif
#ifndef NACL_SPLIT_OCC
#define NACL_SPLIT_OCC 4
#endif
// Proxy lists at least this long use groups of 512 (eight blocks per wave).
constexpr int kSplitWideP = kSplitWideRows;
constexpr int kSplitDepth = NACL_SPLIT_DEPTH;                // ring slots per block (at most 8)
constexpr int kSplitTiles = kSplitChunkKeys / 16;            // tiles per item
static_assert(kSplitTiles % kSplitDepth == 0 && kSplitDepth % 4 == 0, "tiles per item vs ring");

__device__ __forceinline__ void block_barrier() {
  // A barrier without the full fence of __syncthreads(): it waits for this
  // wave's LDS operations (so LDS writes before it are seen by every wave
  // after it) but not for its vector memory operations, so the DMA of later
  // tiles stays in flight across it.
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// WB proxy blocks of 16 per wave, so proxy groups of 64 * WB: WB = 2 (groups
// of 128, four blocks per CU) or WB = 8 (groups of 512 for long proxy lists,
// so that K is streamed once per pass instead of once per 128 proxies; two
// blocks per CU).
template <int WB>
__device__ __forceinline__ void score_split_body(const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                                                 const ScoreArgs& a, const ScoreSched& s) {
  using T = __bf16;
  constexpr int D = 128;
  using M = Mma<T, D>;
  using KS = KStage<T, D>;
  using frag_t = typename M::frag_t;
  constexpr int kS = M::kSteps;
  constexpr int kSplitGroup = 16 * WB * kScoreWaves;  // proxies per group
  constexpr int kNB = WB < 4 ? WB : 4;                // proxy blocks per MFMA batch
  static_assert(KS::kInstr == kScoreWaves, "one DMA instruction per wave and tile");
  static_assert(WB != 8 || kSplitGroup == kSplitWideRows, "row groups of split items are the wide kernel's groups");
  __shared__ int item_s, last_s;
  __shared__ int pos_g[kSplitGroup];
  __shared__ int64_t qrow_g[kSplitGroup];  // element offset of each row's query from qb
  __shared__ float2 mrg[kScoreThreads];
  __shared__ __attribute__((aligned(16))) float col_lds[kSplitChunkKeys];
  __shared__ float stage[kScoreWaves][64];
  __shared__ __attribute__((aligned(16))) float lse_g[kSplitGroup];
#define NACL_SSLOT(i) __shared__ __attribute__((aligned(16))) unsigned char sslot##i[KS::kTileBytes];
  NACL_SSLOT(0) NACL_SSLOT(1) NACL_SSLOT(2) NACL_SSLOT(3) NACL_SSLOT(4) NACL_SSLOT(5) NACL_SSLOT(6) NACL_SSLOT(7)
#undef NACL_SSLOT

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const float c2 = a.c2;
  const uint32_t row_bytes = (uint32_t)(a.ks[2] * (int64_t)sizeof(T));
  // This wave's DMA instruction of a tile: rows kRowsPerInstr * wave ...
  uint32_t vo_all[KS::kInstr];
  KS::offsets(row_bytes, lane, vo_all);
  uint32_t vo = vo_all[0];
#pragma unroll
  for (int i = 1; i < KS::kInstr; ++i) vo = wave == i ? vo_all[i] : vo;
  const uint32_t voff = (uint32_t)r16 * row_bytes + 16u * (uint32_t)g;  // direct fragment loads (exact path)
  const int w0 = 16 * WB * wave;  // this wave's first proxy within the group

  for (;;) {
    __syncthreads();
    if (threadIdx.x == 0) item_s = (int)atomicAdd(s.queue, 1u);
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(item_s);
    if (item >= s.total_items) break;
    const ItemRef it = decode_item(s, item);
    const int bh = it.bh, b = bh / a.H, h = bh % a.H;
    const T* qb = q + b * a.qs[0] + (int64_t)h * a.qg * a.qs[1];  // first query head of the group
    const T* kb = k + b * a.ks[0] + h * a.ks[1];
    const int chunk_key0 = it.chunk * kSplitChunkKeys;
    const bool beyond = chunk_key0 > a.p_last;
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<T*>(kb), (short)0, (int)((uint32_t)(a.L - 1) * row_bytes + (uint32_t)(D * sizeof(T))),
        kBufferRsrcWord3);
    auto tile_byte = [&](int t) -> uint32_t {
      return t < kSplitTiles ? (uint32_t)(chunk_key0 + 16 * t) * row_bytes : kOutOfRange;
    };
    auto slot = [&](auto u_c) -> unsigned char* {
      constexpr int u = decltype(u_c)::value % kSplitDepth;
      if constexpr (u == 0) return sslot0;
      else if constexpr (u == 1) return sslot1;
      else if constexpr (u == 2) return sslot2;
      else if constexpr (u == 3) return sslot3;
      else if constexpr (u == 4) return sslot4;
      else if constexpr (u == 5) return sslot5;
      else if constexpr (u == 6) return sslot6;
      else return sslot7;
    };
    auto issue = [&](int t, unsigned char* dst) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(dst + wave * 1024), 16,
                                               vo + tile_byte(t), 0, 0, kScoreKAux);
    };
    // Streams the item's tiles through the shared ring and calls
    // tile_fn(t, kf, u_c) with tile t's fragments.  Step t: wait for this
    // wave's part of tile t, barrier (every part landed; every wave is done
    // with tile t - 1), refill tile t - 1's slot with tile t + kSplitDepth - 1,
    // read tile t.  The DMA is unconditional (tiles past the item read
    // nothing), so every wait count is static.
    auto k_tiles = [&](auto&& tile_fn) {
      static_for<kSplitDepth - 1>([&](auto u_c) { issue(decltype(u_c)::value, slot(u_c)); });
#pragma unroll 1
      for (int t = 0; t < kSplitTiles; t += kSplitDepth) {
        static_for<kSplitDepth>([&](auto u_c) {
          constexpr int u = decltype(u_c)::value;
          const int tt = t + u;
          asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kSplitDepth - 2) : "memory");
          block_barrier();
          issue(tt + kSplitDepth - 1, slot(std::integral_constant<int, u + kSplitDepth - 1>{}));
          frag_t kf[kS];
          KS::template frag<M>(slot(u_c), r16, g, kf);
          tile_fn(tt, kf, u_c);
        });
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    };
    auto load_group = [&](int g0, int gn) {
      __syncthreads();
      for (int i = threadIdx.x; i < kSplitGroup; i += kScoreThreads) pos_g[i] = i < gn ? row_position(a, g0 + i, qrow_g[i]) : -1;
      __syncthreads();
    };
    // This wave's Q fragments (zeros past the group's end) and the positions
    // of its first and last proxy (no proxy: first = INT_MAX, last = -1).
    auto load_wave_q = [&](int gn, frag_t (&qf)[WB][kS], int& first, int& last) {
#pragma unroll
      for (int pb = 0; pb < WB; ++pb) {
        const int i = w0 + 16 * pb + r16;
        if (i < gn) M::load(qb + qrow_g[i], g, qf[pb]);
        else M::zero(qf[pb]);
      }
      const int wn = min(max(gn - w0, 0), 16 * WB);
      first = wn > 0 ? pos_g[w0] : 0x7FFFFFFF;
      last = wn > 0 ? pos_g[w0 + wn - 1] : -1;
    };
    auto chunk_gumbel_keys = [&](auto&& f_of) {
      uint32_t* gk = s.gkeys + (int64_t)bh * a.L;
      for (int q4 = 4 * (int)threadIdx.x; q4 < kSplitChunkKeys; q4 += 4 * kScoreThreads) {
        const int j0 = chunk_key0 + q4;
        if (j0 >= a.L) break;
        const int n = min(4, a.L - j0);
        float fv[4] = {0.f, 0.f, 0.f, 0.f};
        for (int e = 0; e < n; ++e) fv[e] = f_of(q4 + e);
        uint32_t kv[4];
        gumbel_block_keys(s.g_mode, j0, n, b, h, s.g_layer, s.g_k0, s.g_k1, fv, kv);
        for (int e = 0; e < n; ++e) gk[j0 + e] = kv[e];
      }
    };

    // The item's proxy rows [gb, ge): every row, or one group of them.
    const int gb = s.n_psplit > 1 ? it.psl * kSplitGroup : 0;
    const int ge = s.n_psplit > 1 ? min(a.P, gb + kSplitGroup) : a.P;
    if (it.kind == 1) {
      // ---------------- pass 1: per-chunk (reference, sum) of every proxy row
      float2* part = s.partials + ((int64_t)bh * s.n_chunks + it.chunk) * a.P;
      if (beyond)
        for (int i = gb + threadIdx.x; i < ge; i += kScoreThreads)
          store_coherent(part + i, make_float2(-INFINITY, 0.f));
      for (int g0 = gb; g0 < (beyond ? gb : ge); g0 += kSplitGroup) {
        const int gn = min(kSplitGroup, a.P - g0);
        load_group(g0, gn);
        if (pos_g[gn - 1] < chunk_key0) {
          // No row of the group sees this chunk (rows are sorted by
          // position): nothing to stream or compute.
          for (int i = threadIdx.x; i < gn; i += kScoreThreads)
            store_coherent(part + g0 + i, make_float2(-INFINITY, 0.f));
          continue;
        }
        frag_t qf[WB][kS];
        int first, last;
        load_wave_q(gn, qf, first, last);
        // Per proxy block: base-2 reference (the scaled maximum of the item's
        // first tile, 0 if that tile shows the proxy nothing) and the running
        // sum of exp2(logit * c2 - ref) over this lane's keys (visibility is a
        // prefix of the keys: see the main kernel).
        float ref[WB], sm[WB];
#pragma unroll
        for (int pb = 0; pb < WB; ++pb) {
          ref[pb] = 0.f;
          sm[pb] = 0.f;
        }
        // Blocks [P0, P0 + kNB) of one tile (acc[pb - P0]).
        auto body1 = [&](int t, const f32x4 (&acc)[kNB], auto p0_c, auto full_c) {
          constexpr int P0 = decltype(p0_c)::value;
          constexpr bool FULL = decltype(full_c)::value;
          const int key0 = chunk_key0 + 16 * t;
          const int* pos_l = pos_g + w0 + opaque(r16);
#pragma unroll
          for (int pb = P0; pb < P0 + kNB; ++pb) {
            bool vis[4];
            if constexpr (!FULL) {
              const int pi = pos_l[16 * pb];
#pragma unroll
              for (int e = 0; e < 4; ++e) vis[e] = key0 + 4 * g + e <= pi;
            }
            if (t == 0) {
              float mx = -INFINITY;
#pragma unroll
              for (int e = 0; e < 4; ++e) mx = (FULL || vis[e]) ? fmaxf(mx, acc[pb - P0][e]) : mx;
              mx = max_over_groups(mx);
              ref[pb] = mx != -INFINITY ? mx * c2 : 0.f;
            }
            float x[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = fast_exp2(fmaf(acc[pb - P0][e], c2, -ref[pb]));
            if constexpr (!FULL) {
#pragma unroll
              for (int e = 0; e < 4; ++e) x[e] = vis[e] ? x[e] : 0.f;
            }
            sm[pb] += (x[0] + x[1]) + (x[2] + x[3]);
          }
        };
        k_tiles([&](int t, const frag_t (&kf)[kS], auto) {
          const int key0 = chunk_key0 + 16 * t;
          if (key0 > last) return;
          static_for<WB / kNB>([&](auto h_c) {
            using P0 = std::integral_constant<int, decltype(h_c)::value * kNB>;
            f32x4 acc[kNB];
            tile_logits<M, WB, P0::value, kNB, true>(kf, qf, acc);
            if (key0 + 15 <= first) body1(t, acc, P0{}, std::true_type{});
            else body1(t, acc, P0{}, std::false_type{});
          });
        });
        bool bad = false;
#pragma unroll
        for (int pb = 0; pb < WB; ++pb) {
          sm[pb] = sum_over_groups(sm[pb]);
          bad |= !(sm[pb] <= 3.0e38f);
        }
        if (__builtin_amdgcn_ballot_w64(bad)) {
          // Exact path (this wave only): the maximum over every visible key,
          // then the sums, with direct loads.
          float mx[WB];
#pragma unroll
          for (int pb = 0; pb < WB; ++pb) mx[pb] = -INFINITY;
          for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
            for (int pb = 0; pb < WB; ++pb) sm[pb] = 0.f;
            for (int t = 0; t < kSplitTiles; ++t) {
              const int key0 = chunk_key0 + 16 * t;
              if (key0 > last) break;
              frag_t kf[kS];
              M::load_k(rsrc, voff + (uint32_t)key0 * row_bytes, kf);
              static_for<WB / kNB>([&](auto h_c) {
                constexpr int P0 = decltype(h_c)::value * kNB;
                f32x4 acc[kNB];
                tile_logits<M, WB, P0, kNB, true>(kf, qf, acc);
#pragma unroll
                for (int pb = P0; pb < P0 + kNB; ++pb) {
                  const int pi = pos_g[w0 + 16 * pb + r16];
#pragma unroll
                  for (int e = 0; e < 4; ++e) {
                    const bool v = key0 + 4 * g + e <= pi;
                    if (pass == 0) mx[pb] = v ? fmaxf(mx[pb], acc[pb - P0][e]) : mx[pb];
                    else sm[pb] += v ? fast_exp2(fmaf(acc[pb - P0][e], c2, -ref[pb])) : 0.f;
                  }
                }
              });
            }
            if (pass == 0) {
#pragma unroll
              for (int pb = 0; pb < WB; ++pb) {
                mx[pb] = max_over_groups(mx[pb]);
                ref[pb] = mx[pb] != -INFINITY ? mx[pb] * c2 : 0.f;
              }
            }
          }
#pragma unroll
          for (int pb = 0; pb < WB; ++pb) sm[pb] = sum_over_groups(sm[pb]);
        }
        if (g == 0) {
#pragma unroll
          for (int pb = 0; pb < WB; ++pb) {
            const int i = w0 + 16 * pb + r16;
            if (i < gn)
              store_coherent(part + g0 + i, sm[pb] > 0.f ? make_float2(ref[pb], sm[pb]) : make_float2(-INFINITY, 0.f));
          }
        }
      }
      // Publish the partials; the last chunk of the head merges them.
      wait_stores();
      __syncthreads();
      if (threadIdx.x == 0) last_s = atomicAdd(&s.head_cnt[bh], 1u) == (unsigned)(s.n_chunks * s.n_psplit - 1);
      __syncthreads();
      if (last_s) {
        const float2* hp = s.partials + (int64_t)bh * s.n_chunks * a.P;
        const int split = a.P >= kScoreThreads ? 1 : kScoreThreads / a.P;
        const int part_i = threadIdx.x / a.P;
        constexpr int kBatch = 8;
        for (int i0 = 0; i0 < a.P; i0 += kScoreThreads) {
          const int i = i0 + (split == 1 ? (int)threadIdx.x : (int)threadIdx.x % a.P);
          float mm = -INFINITY, ss = 0.f;
          if (i < a.P && part_i < split) {
            for (int c0 = part_i; c0 < s.n_chunks; c0 += kBatch * split) {
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
            if (part_i == 0 && i < a.P)
              for (int pp = 1; pp < split; ++pp) {
                const float2 r = mrg[threadIdx.x + pp * a.P];
                lse_merge(mm, ss, r.x, r.y);
              }
          }
          if (part_i == 0 && i < a.P) store_coherent(s.lse2 + (int64_t)bh * a.P + i, mm + __log2f(ss));
        }
        wait_stores();
        __syncthreads();
        if (threadIdx.x == 0) atomicAdd(&s.head_cnt[bh], 1u);
      }
    } else if (beyond) {
      if (it.psl == 0) {
        float* F = s.scores + (int64_t)bh * a.L;
        const int end = min(chunk_key0 + kSplitChunkKeys, a.L);
        for (int j = chunk_key0 + threadIdx.x; j < end; j += kScoreThreads) F[j] = 0.f;
        if (s.gkeys) chunk_gumbel_keys([](int) { return 0.f; });
      }
    } else {
      // ---------------- pass 2: column sums of exp2(logit - LSE) ----------
      if (!s.lse_given) {
        if (threadIdx.x == 0) {
          uint32_t spins = 0;
          while (load_coherent(&s.head_cnt[bh]) < (unsigned)(s.n_chunks * s.n_psplit + 1)) {
            __builtin_amdgcn_s_sleep(2);
            if (++spins > kSpinLimit) {
              atomicOr(s.status, 1u);
              atomicOr(s.status + 1, 1u);
              break;
            }
          }
        }
        __syncthreads();
      }
      const float* lse = s.lse_given ? s.lse_in : s.lse2;
      const float lse_mul = s.lse_given ? s.lse_mul : 1.0f;
      bool fresh = true;  // the item's columns are not yet written
      for (int g0 = gb; g0 < ge; g0 += kSplitGroup) {
        const int gn = min(kSplitGroup, a.P - g0);
        load_group(g0, gn);
        if (pos_g[gn - 1] < chunk_key0) continue;  // no row of the group sees this chunk
        frag_t qf[WB][kS];
        int first, last;
        load_wave_q(gn, qf, first, last);
        for (int i = threadIdx.x; i < kSplitGroup; i += kScoreThreads)
          lse_g[i] = i < gn ? load_coherent(lse + lse_index(a, s, bh, g0 + i)) * lse_mul : INFINITY;
        __syncthreads();
        // With groups of 128 proxies this lane's eight log-sum-exps (rows
        // 4 g + e of its two proxy blocks) stay in registers for the whole
        // item; wider groups read them from LDS at every tile.
        constexpr int kLR = WB == 2 ? WB : 1;
        f32x4 lse_r[kLR];
        if constexpr (WB == 2) {
#pragma unroll
          for (int pb = 0; pb < kLR; ++pb) lse_r[pb] = *reinterpret_cast<const f32x4*>(lse_g + w0 + 4 * g + 16 * pb);
        }
        // This lane's share of its key's column sum over the wave's proxies;
        // FULL tiles carry no masking.
        auto body2 = [&](int key0, const f32x4 (&acc)[kNB], auto p0_c, auto full_c) -> float {
          constexpr int P0 = decltype(p0_c)::value;
          constexpr bool FULL = decltype(full_c)::value;
          const int o = w0 + opaque(4 * g);
          const float* lse_l = lse_g + o;
          const int* pos_l = pos_g + o;
          f32x4 lrs[kNB];
          if constexpr (WB == 2) {
#pragma unroll
            for (int pb = P0; pb < P0 + kNB; ++pb) lrs[pb - P0] = lse_r[pb < kLR ? pb : 0];
          } else {
#pragma unroll
            for (int pb = P0; pb < P0 + kNB; ++pb) lrs[pb - P0] = *reinterpret_cast<const f32x4*>(lse_l + 16 * pb);
          }
          float cs = 0.f;
#pragma unroll
          for (int pb = P0; pb < P0 + kNB; ++pb) {
            float x[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = fast_exp2(fmaf(acc[pb - P0][e], c2, -lrs[pb - P0][e]));
            if constexpr (!FULL) {
#pragma unroll
              for (int e = 0; e < 4; ++e) x[e] = key0 + r16 <= pos_l[16 * pb + e] ? x[e] : 0.f;
            }
            cs += (x[0] + x[1]) + (x[2] + x[3]);
          }
          return cs;
        };
        // Partial column sums of the last four tiles; every fourth tile they
        // are reduced across lane groups (lane group g holds tile t - 3 + g)
        // and staged per wave; one step later, after the barrier, wave 0 adds
        // the four waves' stages in a fixed order into the item's columns.
        float cs4[4];
        auto reduce_stage = [&](int t0) {  // tiles t0 .. t0 + 3
          if (wave == 0) {
            const float z = ((stage[0][lane] + stage[1][lane]) + stage[2][lane]) + stage[3][lane];
            const int idx = t0 * 16 + lane;
            col_lds[idx] = (fresh ? 0.f : col_lds[idx]) + z;
          }
        };
        k_tiles([&](int t, const frag_t (&kf)[kS], auto u_c) {
          constexpr int u = decltype(u_c)::value;
          if constexpr (u % 4 == 0) {
            if (t >= 4) reduce_stage(t - 4);
          }
          const int key0 = chunk_key0 + 16 * t;
          float cs = 0.f;
          if (key0 <= last) {
            static_for<WB / kNB>([&](auto h_c) {
              using P0 = std::integral_constant<int, decltype(h_c)::value * kNB>;
              f32x4 acc[kNB];
              tile_logits<M, WB, P0::value, kNB, false>(kf, qf, acc);
              if (key0 + 15 <= first) cs += body2(key0, acc, P0{}, std::true_type{});
              else cs += body2(key0, acc, P0{}, std::false_type{});
            });
          }
          cs4[u % 4] = cs;
          if constexpr (u % 4 == 3) stage[wave][lane] = colsum4(cs4[0], cs4[1], cs4[2], cs4[3]);
        });
        __syncthreads();
        reduce_stage(kSplitTiles - 4);
        fresh = false;
      }
      __syncthreads();
      bool write = true;
      if (s.n_psplit > 1) {
        // Publish this group's column sums (none if no row of it sees the
        // chunk); the chunk's last item adds the groups' sums in group order,
        // as one item over every group would, and writes the scores.
        const int64_t cidx = (int64_t)bh * s.n_chunks + it.chunk;
        float* cp = s.colpart + cidx * s.n_psplit * kSplitChunkKeys;
        if (!fresh)
          for (int q4 = 4 * (int)threadIdx.x; q4 < kSplitChunkKeys; q4 += 4 * kScoreThreads)
            store_coherent16(cp + it.psl * kSplitChunkKeys + q4,
                             __builtin_bit_cast(u32x4, *reinterpret_cast<const f32x4*>(col_lds + q4)));
        wait_stores();
        __syncthreads();
        if (threadIdx.x == 0) last_s = atomicAdd(&s.chunk_cnt[cidx], 1u) == (unsigned)(s.n_psplit - 1);
        __syncthreads();
        write = last_s != 0;
        if (write) {
          for (int idx = threadIdx.x; idx < kSplitChunkKeys; idx += kScoreThreads) {
            float acc = 0.f;
            for (int pg = 0; pg < s.n_psplit; ++pg) {
              int64_t unused;
              const int lr = min(a.P, (pg + 1) * kSplitGroup) - 1;  // the group's last row
              if (row_position(a, lr, unused) >= chunk_key0) acc += load_coherent(cp + pg * kSplitChunkKeys + idx);
            }
            col_lds[idx] = acc;
          }
          __syncthreads();
        }
      }
      if (write) {
        float* F = s.scores + (int64_t)bh * a.L;
        auto col_of = [&](int idx) -> float { return col_lds[idx]; };
        for (int idx = threadIdx.x; idx < kSplitChunkKeys; idx += kScoreThreads) {
          const int key = chunk_key0 + idx;
          if (key < a.L) F[key] = col_of(idx);
        }
        if (s.gkeys) chunk_gumbel_keys(col_of);
      }
    }
  }
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

// Proxy blocks of 16 per group (every wave holds all of them).
int proxy_blocks(int dtype, int D, int P) {
  const int need = (P + 15) / 16;
  if (dtype == 1) return need <= 2 ? 2 : (need <= 4 ? 4 : 8);
  if (D == 128) return 2;
  return need <= 2 ? 2 : 4;
}

}  // namespace

// The two kernels (the launch bound, which sets the register budget, has to
// be a constant of the kernel itself).
__global__ __launch_bounds__(kScoreThreads, NACL_SPLIT_OCC) void score_split_kernel(const __bf16* __restrict__ q,
                                                                                    const __bf16* __restrict__ k,
                                                                                    ScoreArgs a, ScoreSched s) {
  score_split_body<2>(q, k, a, s);
}
__global__ __launch_bounds__(kScoreThreads, 2) void score_split_wide_kernel(const __bf16* __restrict__ q,
                                                                           const __bf16* __restrict__ k,
                                                                           ScoreArgs a, ScoreSched s) {
  score_split_body<8>(q, k, a, s);
}

template <class K>
hipError_t launch_score_split_t(K kern, const ScoreLaunch& L, hipStream_t stream) {
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
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kScoreThreads), 0, stream, static_cast<const __bf16*>(L.q),
                     static_cast<const __bf16*>(L.k), L.args, L.sched);
  return hipGetLastError();
}

hipError_t launch_score_split(const ScoreLaunch& L, hipStream_t stream) {
  if (L.args.P >= kSplitWideP) return launch_score_split_t(score_split_wide_kernel, L, stream);
  return launch_score_split_t(score_split_kernel, L, stream);
}

template <typename T, int D>
hipError_t launch_score_rows_t(const ScoreLaunch& L, hipStream_t stream) {
  ScoreSched s = L.sched;
  s.n_clear = L.n_counter_words;  // cleared by the logit kernel: no separate clearing launch
  const int BH = L.args.B * L.args.H;
  hipLaunchKernelGGL((score_rows_logits_kernel<T, D>), dim3(s.n_chunks, BH), dim3(kScoreThreads), 0, stream,
                     static_cast<const T*>(L.q), static_cast<const T*>(L.k), L.args, s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int col_blocks = (L.args.L + 4 * kScoreThreads - 1) / (4 * kScoreThreads);
  hipLaunchKernelGGL(score_rows_column_kernel, dim3(col_blocks, BH), dim3(kScoreThreads), 0, stream, L.args, s);
  return hipGetLastError();
}

int score_rows_chunk(int dtype, int D, int L, int BH, int cus) {
  int per_cu = 0;
  hipError_t e;
  if (dtype == 1)
    e = D == 128 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, score_rows_logits_kernel<__bf16, 128>, kScoreThreads, 0)
                 : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, score_rows_logits_kernel<__bf16, 64>, kScoreThreads, 0);
  else
    e = D == 128 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, score_rows_logits_kernel<float, 128>, kScoreThreads, 0)
                 : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, score_rows_logits_kernel<float, 64>, kScoreThreads, 0);
  if (e != hipSuccess || per_cu < 1) per_cu = 1;
  const int64_t slots = (int64_t)per_cu * std::max(1, cus);
  // Fewest chunks per head (longest chunks), the rounds of resident
  // work-groups they take, then as many chunks as fill those rounds.
  const int64_t n_min = (L + kRowsChunkMax - 1) / kRowsChunkMax;
  const int64_t rounds = (BH * n_min + slots - 1) / slots;
  const int64_t n_fill = std::max(n_min, rounds * slots / BH);
  int ck = (int)(((L + n_fill - 1) / n_fill + 63) / 64 * 64);
  ck = std::max(ck, std::min(kRowsChunkMin, (L + 63) / 64 * 64));
  return std::min(ck, kRowsChunkMax);
}

hipError_t launch_score(const ScoreLaunch& L, hipStream_t stream) {
  if (L.sched.logits) {
    // The few-row path: every row in one 16-column MFMA tile, one partial
    // per chunk, no caller log-sum-exp.
    const int ck = L.sched.chunk_keys;
    if (!score_uses_rows(L.dtype, L.D, L.args.P) || L.args.P > 16 || L.sched.lse_given || ck < 64 ||
        ck > kRowsChunkMax || ck % 64 != 0 || L.sched.n_chunks != (L.args.L + ck - 1) / ck ||
        L.sched.logits_stride < L.args.L || L.sched.logits_stride % 4 != 0)
      return hipErrorInvalidValue;
    if (L.dtype == 1) return L.D == 128 ? launch_score_rows_t<__bf16, 128>(L, stream) : launch_score_rows_t<__bf16, 64>(L, stream);
    return L.D == 128 ? launch_score_rows_t<float, 128>(L, stream) : launch_score_rows_t<float, 64>(L, stream);
  }
  if (score_uses_split(L.dtype, L.D, L.args.P)) {
    if (L.sched.chunk_keys != kSplitChunkKeys) return hipErrorInvalidValue;
    if (L.sched.n_psplit != score_psplit(L.dtype, L.D, L.args.P)) return hipErrorInvalidValue;
    return launch_score_split(L, stream);
  }
  if (L.sched.n_psplit != 1) return hipErrorInvalidValue;
  const int pb = proxy_blocks(L.dtype, L.D, L.args.P);
  if (L.dtype == 1) {
    if (L.D == 128) {
      if (pb == 2) return launch_score_t<__bf16, 128, 2>(L, stream);
      if (pb == 4) return launch_score_t<__bf16, 128, 4>(L, stream);
      return launch_score_t<__bf16, 128, 8>(L, stream);
    }
    if (pb == 2) return launch_score_t<__bf16, 64, 2>(L, stream);
    if (pb == 4) return launch_score_t<__bf16, 64, 4>(L, stream);
    return launch_score_t<__bf16, 64, 8>(L, stream);
  }
  if (L.D == 128) return launch_score_t<float, 128, 2>(L, stream);
  if (pb == 2) return launch_score_t<float, 64, 2>(L, stream);
  return launch_score_t<float, 64, 4>(L, stream);
}

}  // namespace nacl
