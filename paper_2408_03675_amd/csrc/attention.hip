// Causal attention of the prefill with each query row's log-sum-exp: the
// forward pass of FlashAttention-2 that Appendix A.7 reuses, whose
// log-sum-exp lets the proxy-token score run as the single column reduction
// of Algorithm 2 (nacl_score's lse argument).  bf16 Q, K, V and output,
// fp32 accumulation, head dim 64 or 128, grouped query heads.
//
// One work-group of 4 waves takes 128 consecutive query rows of one query
// head; wave w holds rows 32w .. 32w + 31 (two 16-row MFMA tiles) in
// registers and streams the head's keys in tiles of 64:
//   S^T = K Q^T      v_mfma_f32_16x16x32_bf16, keys as MFMA rows, so lane
//                    (g, r) holds keys 4g .. 4g + 3 of each 16-key block for
//                    query r: every lane owns one query per MFMA tile, and
//                    the running maximum, sum and output rescale are
//                    per-lane scalars (the four lane groups agree on the
//                    maximum through two permlane swaps)
//   O^T += V^T P^T   the exponentials P in bf16 as the B operand straight
//                    from the S^T registers (lane (g, r) supplies keys
//                    4g .. 4g + 3 of two 16-key blocks, a permutation of the
//                    contraction that the A operand repeats), V^T from LDS.
// K and V tiles are loaded into registers one tile ahead and written into
// the other half of a double buffer in LDS after the tile in hand is done,
// so one barrier per tile separates the stages: K rows with their 16-byte
// chunks XOR-swizzled (the 16 rows of a fragment read hit distinct banks),
// V transposed (V^T[d][key], each lane's 8 keys of a fragment in one
// XOR-swizzled 16-byte chunk).
// (Buffer->LDS loads for K would save the registers, but the compiler makes
// every LDS read wait for all of them in flight, the next tile's included.)
// Work-groups are dealt to the 8 XCDs in turn; each XCD takes a contiguous
// range of (head, 128-row tile) work, a head's tiles in decreasing length,
// so the tiles in flight on an XCD share their K/V through its L2.

#include <type_traits>

#include "device_common.h"
#include "internal.h"

namespace nacl {

namespace {

constexpr int kAttnThreads = 256;
constexpr int kAttnRows = 128;  // query rows per work-group
constexpr int kAttnKeys = 64;   // keys per tile
constexpr int kRsrcWord3 = 0x00020000;

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void attn_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
// s_waitcnt vmcnt(0) (expcnt and lgkmcnt fields at their maxima), as an
// instruction the compiler's own wait counting sees.
__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Maximum / sum over the four lane groups (lanes r, r + 16, r + 32, r + 48).
__device__ __forceinline__ float group_max(float x) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float group_sum(float x) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

template <int D>
__global__ __launch_bounds__(kAttnThreads, 2) void attn_fwd_kernel(AttnLaunch a) {
  constexpr int kRowBytes = D * 2;         // one K or V row
  constexpr int kChunks = kRowBytes / 16;  // 16-byte chunks per row
  constexpr int kSwz = kChunks - 1;
  constexpr int kKb = D / 32;              // contraction steps of S^T
  constexpr int kDt = D / 16;              // 16-wide d tiles of O^T
  constexpr int kTileBytes = kAttnKeys * kRowBytes;
  constexpr int kKUnits = kAttnKeys * kChunks / kAttnThreads;        // 16-byte K chunks per thread
  constexpr int kVUnits = (kAttnKeys / 2) * kChunks / kAttnThreads;  // (key pair, chunk) per thread
  static_assert(kKUnits >= 1 && kVUnits >= 1, "tile shape");

  __shared__ __attribute__((aligned(16))) unsigned char kbuf[2][kTileBytes];  // K rows, chunks swizzled
  __shared__ __attribute__((aligned(16))) unsigned char vbuf[2][kTileBytes];  // V^T[d][64 keys]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, r = lane & 15;

  // Work index: XCD x = id mod 8 takes the x-th contiguous eighth.
  const int id = blockIdx.x, n = gridDim.x;
  const int xcd = id & 7, slot = id >> 3, q8 = n >> 3, r8 = n & 7;
  const int w = (xcd < r8 ? xcd * (q8 + 1) : r8 * (q8 + 1) + (xcd - r8) * q8) + slot;
  const int bhq = w / a.n_tiles;
  const int tile = a.n_tiles - 1 - (w - bhq * a.n_tiles);
  const int Hq = a.H * a.G;
  const int b = bhq / Hq, hq = bhq - b * Hq, h = hq / a.G;
  const int L = a.L;
  const int q0 = tile * kAttnRows;
  const int qw0 = q0 + 32 * wave;
  const int n_kv = (min(q0 + kAttnRows, L) + kAttnKeys - 1) / kAttnKeys;

  const __bf16* qh = a.q + (int64_t)b * a.qs[0] + (int64_t)hq * a.qs[1];
  const __bf16* kh = a.k + (int64_t)b * a.ks[0] + (int64_t)h * a.ks[1];
  const __bf16* vh = a.v + (int64_t)b * a.vs[0] + (int64_t)h * a.vs[1];
  const uint32_t qrow = (uint32_t)a.qs[2] * 2u, krow = (uint32_t)a.ks[2] * 2u, vrow = (uint32_t)a.vs[2] * 2u;
  // Rows at or past L read as zeros through the descriptors' ranges.
  const __amdgpu_buffer_rsrc_t qr = __builtin_amdgcn_make_buffer_rsrc(const_cast<__bf16*>(qh), (short)0,
                                                                      (int)((uint32_t)L * qrow), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(const_cast<__bf16*>(kh), (short)0,
                                                                      (int)((uint32_t)L * krow), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(const_cast<__bf16*>(vh), (short)0,
                                                                      (int)((uint32_t)L * vrow), kRsrcWord3);

  // Q fragments (B operand of S^T): query row qw0 + 16 qt + r, d = 32 kb + 8 g .. + 7.
  bf16x8 qf[2][kKb];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt)
#pragma unroll
    for (int kb = 0; kb < kKb; ++kb)
      qf[qt][kb] = __builtin_bit_cast(
          bf16x8, __builtin_amdgcn_raw_buffer_load_b128(qr, (uint32_t)(qw0 + 16 * qt + r) * qrow + (uint32_t)(64 * kb + 16 * g),
                                                        0, 0));

  // K units: (row u / kChunks, chunk u mod kChunks) for u = tid + 256 s:
  // 16 lanes read one row's 256 contiguous bytes (D = 128); the chunk goes
  // to position chunk ^ (row & kSwz) of its LDS row.
  u32x4 kreg[kKUnits];
  auto load_k = [&](int j) {
#pragma unroll
    for (int s = 0; s < kKUnits; ++s) {
      const int u = tid + kAttnThreads * s;
      kreg[s] = __builtin_amdgcn_raw_buffer_load_b128(
          kr, (uint32_t)(j * kAttnKeys + u / kChunks) * krow + (uint32_t)(u % kChunks) * 16u, 0, 0);
    }
  };
  auto write_k = [&](int buf) {
#pragma unroll
    for (int s = 0; s < kKUnits; ++s) {
      const int u = tid + kAttnThreads * s;
      const int row = u / kChunks;
      *reinterpret_cast<u32x4*>(kbuf[buf] + row * kRowBytes + (((u % kChunks) ^ (row & kSwz)) * 16)) = kreg[s];
    }
  };
  // V units: (key pair kp = tid mod 32, chunk c = tid / 32 + 8 u): rows 2 kp
  // and 2 kp + 1, d = 8 c .. 8 c + 7.
  const int kp = tid & 31;
  u32x4 vreg[kVUnits][2];
  auto load_v = [&](int j) {
#pragma unroll
    for (int u = 0; u < kVUnits; ++u) {
      const int c = (tid >> 5) + 8 * u;
#pragma unroll
      for (int e = 0; e < 2; ++e)
        vreg[u][e] = __builtin_amdgcn_raw_buffer_load_b128(
            vr, (uint32_t)(j * kAttnKeys + 2 * kp + e) * vrow + (uint32_t)c * 16u, 0, 0);
    }
  };
  // V^T row d (128 bytes) holds the tile's 64 keys permuted so that the 8
  // keys lane group g contributes to contraction block kb2 (keys 32 kb2 +
  // 4 g .. + 3 and 32 kb2 + 16 + 4 g .. + 3) form 16-byte chunk 4 kb2 + g,
  // stored at chunk position (4 kb2 + g) ^ ((d >> 1) & 7): the 16 rows one
  // fragment read touches then cover every bank once per row parity.
  // Per V unit: the byte offset of d = 8 c + 2 h (h = 0..3) in its V^T row
  // pair, chunk swizzle included; d = 8 c + 2 h + 1 is the next row.
  uint32_t vto[kVUnits][4];
  {
    // keys 2 kp, 2 kp + 1: block kp >> 4, half (kp >> 3) & 1, group (kp >> 1) & 3,
    // the first of them at 2 (kp & 1) within its 4 keys
    const int c16 = 4 * (kp >> 4) + ((kp >> 1) & 3);
    const int dw = 2 * ((kp >> 3) & 1) + (kp & 1);  // dword within the chunk
#pragma unroll
    for (int u = 0; u < kVUnits; ++u) {
      const int c = (tid >> 5) + 8 * u;
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const int d = 8 * c + 2 * h;
        vto[u][h] = (uint32_t)(d * 128 + ((c16 ^ ((d >> 1) & 7)) * 16) + dw * 4);
      }
    }
  }
  auto write_vt = [&](int buf) {
#pragma unroll
    for (int u = 0; u < kVUnits; ++u) {
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        // bf16 jj of rows 2 kp (low half) and 2 kp + 1 (high half): bytes
        // 2 (jj mod 2) .. + 1 of word jj / 2 of each
        const uint32_t w = __builtin_amdgcn_perm(vreg[u][1][jj >> 1], vreg[u][0][jj >> 1],
                                                 (jj & 1) ? 0x07060302u : 0x05040100u);
        *reinterpret_cast<uint32_t*>(vbuf[buf] + vto[u][jj >> 1] + (jj & 1) * 128) = w;
      }
    }
  };

  const float c2 = a.c2;
  f32x4 acc[2][kDt];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt)
#pragma unroll
    for (int dt = 0; dt < kDt; ++dt) acc[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m[2] = {-INFINITY, -INFINITY}, l[2] = {0.f, 0.f};

  load_k(0);
  load_v(0);
  wait_vm_all();
  write_k(0);
  write_vt(0);
  if (n_kv > 1) {
    load_k(1);
    load_v(1);
  }
  attn_barrier();

  for (int j = 0; j < n_kv; ++j) {
    const int buf = j & 1;
    const int key0 = j * kAttnKeys;
    if (key0 <= qw0 + 31) {  // some key of the tile is visible to a row of this wave
      const unsigned char* kt_base = kbuf[buf];
      const unsigned char* vt_base = vbuf[buf];
      // S^T tiles: kt (16 keys) x qt (16 queries).
      f32x4 s[4][2];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const int row = 16 * kt + r;
        bf16x8 kf[kKb];
#pragma unroll
        for (int kb = 0; kb < kKb; ++kb)
          kf[kb] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4*>(kt_base + row * kRowBytes + (((4 * kb + g) ^ (row & kSwz)) * 16)));
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
          f32x4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kb = 0; kb < kKb; ++kb) t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kb], qf[qt][kb], t, 0, 0, 0);
          s[kt][qt] = t;
        }
      }
      // Value fragment (A operand of O^T): V^T row d = 16 dt + r, chunk 4 kb2 + g.
      auto vfrag = [&](int dt, int kb2) {
        const int d = 16 * dt + r;
        return __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(vt_base + d * 128 + (((4 * kb2 + g) ^ ((d >> 1) & 7)) * 16)));
      };
      // The first d tile's value fragments are read before the exponentials.
      bf16x8 vcur[2] = {vfrag(0, 0), vfrag(0, 1)};
      __builtin_amdgcn_sched_barrier(0);
      const bool masked = key0 + kAttnKeys - 1 > qw0;
      bf16x8 pf[2][2];  // [qt][kb2]
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        const int qi = qw0 + 16 * qt + r;
        if (masked) {
          // key key0 + 16 kt + 4 g + i is past row qi iff 16 kt + i > lim
          const int lim = qi - key0 - 4 * g;
#pragma unroll
          for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (16 * kt + i > lim) s[kt][qt][i] = -INFINITY;
        }
        // The scale is positive, so the largest logit is the scaled largest
        // raw product; each exponent is then one FMA.
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[kt][qt][i]);
        mx = group_max(mx);
        const float mn = fmaxf(m[qt], mx * c2);
        const float alpha = __builtin_amdgcn_exp2f(m[qt] - mn);
        m[qt] = mn;
        float x[4][4];
        float sum = 0.f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            x[kt][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kt][qt][i], c2, -mn));
            sum += x[kt][i];
          }
        l[qt] = l[qt] * alpha + sum;
        // Rescale only when some row of the wave raised its maximum.
        if (__ballot(alpha != 1.f)) {
#pragma unroll
          for (int dt = 0; dt < kDt; ++dt) acc[qt][dt] *= alpha;
        }
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
          pf[qt][kb2] = bf16x8{(__bf16)x[2 * kb2][0], (__bf16)x[2 * kb2][1], (__bf16)x[2 * kb2][2],
                               (__bf16)x[2 * kb2][3], (__bf16)x[2 * kb2 + 1][0], (__bf16)x[2 * kb2 + 1][1],
                               (__bf16)x[2 * kb2 + 1][2], (__bf16)x[2 * kb2 + 1][3]};
      }
      // O^T += V^T P^T; the reads of d tile dt + 1 are issued before the
      // products of d tile dt.
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt) {
        bf16x8 vnxt[2];
        if (dt + 1 < kDt) {
          vnxt[0] = vfrag(dt + 1, 0);
          vnxt[1] = vfrag(dt + 1, 1);
        }
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
          for (int qt = 0; qt < 2; ++qt)
            acc[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vcur[kb2], pf[qt][kb2], acc[qt][dt], 0, 0, 0);
        if (dt + 1 < kDt) {
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // the two reads
          __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);  // then the four products
          vcur[0] = vnxt[0];
          vcur[1] = vnxt[1];
        }
      }
    }
    if (j + 1 < n_kv) {
      wait_vm_all();  // this thread's K and V rows of tile j + 1
      write_k(buf ^ 1);
      write_vt(buf ^ 1);
    }
    attn_barrier();  // tile j read by every wave; tile j + 1 written
    if (j + 2 < n_kv) {
      load_k(j + 2);
      load_v(j + 2);
    }
  }

  // Normalise and store: lane (g, r) holds O[row][16 dt + 4 g .. + 3].
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int qi = qw0 + 16 * qt + r;
    const float lt = group_sum(l[qt]);
    if (qi < L) {
      const float inv = 1.f / lt;
      __bf16* orow = a.out + ((int64_t)bhq * L + qi) * D;
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt) {
        const bf16x4 o = {(__bf16)(acc[qt][dt][0] * inv), (__bf16)(acc[qt][dt][1] * inv),
                          (__bf16)(acc[qt][dt][2] * inv), (__bf16)(acc[qt][dt][3] * inv)};
        *reinterpret_cast<bf16x4*>(orow + 16 * dt + 4 * g) = o;
      }
      if (g == 0) a.lse[(int64_t)bhq * L + qi] = (m[qt] + __log2f(lt)) * 0.69314718055994531f;
    }
  }
}

// lse_proxy[b, hq, p] = lse[b, hq, pos[p]] (NaN for a position outside
// [0, L), which a device copy that disagrees with the validated host
// positions could hold; nothing outside the head is read).
__global__ __launch_bounds__(256) void lse_gather_kernel(const float* lse, const int32_t* pos, int L, int P,
                                                         int64_t n, float* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int64_t bh = i / P;
  const int j = pos[i - bh * P];
  out[i] = j >= 0 && j < L ? lse[bh * L + j] : __builtin_nanf("");
}

}  // namespace

hipError_t launch_attention(const AttnLaunch& a, int D, const int32_t* pos, int P, float* lse_proxy,
                            hipStream_t stream) {
  const int64_t blocks = (int64_t)a.B * a.H * a.G * a.n_tiles;
  if (D == 128)
    hipLaunchKernelGGL(attn_fwd_kernel<128>, dim3((unsigned)blocks), dim3(kAttnThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<64>, dim3((unsigned)blocks), dim3(kAttnThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !lse_proxy) return e;
  const int64_t n = (int64_t)a.B * a.H * a.G * P;
  hipLaunchKernelGGL(lse_gather_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, a.lse, pos,
                     a.L, P, n, lse_proxy);
  return hipGetLastError();
}

}  // namespace nacl
