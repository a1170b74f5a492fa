// Internal interface between the C ABI (api.cpp) and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace nacl {

// Keys per score work-group = kScoreTilesPerWave * 4 waves * 16 keys.
constexpr int kScoreTilesPerWave = 8;
constexpr int kScoreChunkKeys = kScoreTilesPerWave * 4 * 16;

struct ScoreArgs {
  int B, H, L, P;
  int64_t qs[3], ks[3];
  const int* pos;   // device, P entries
  float c2;         // sm_scale * log2(e)
};

struct ScoreLaunch {
  ScoreArgs args;
  int dtype, D;
  const void* q;
  const void* k;
  bool run_pass1;        // false: caller supplied the log-sum-exp
  int n_chunks1, n_chunks2;
  float2* partials;      // workspace [B*H, n_chunks1, P]
  float* lse2_ws;        // workspace [B*H, P], base-2 log-sum-exp
  const float* lse_in;   // what pass 2 reads (lse2_ws or the caller's)
  float lse_mul;         // 1 for base 2, log2(e) for natural log-sum-exp
  float* scores;         // [B*H, L]
};

hipError_t launch_score(const ScoreLaunch& L, hipStream_t stream);

struct SelectLaunch {
  int B, H, L, P, n_protect, C, Cp, Cr, sampling;
  uint64_t seed;
  uint32_t layer;
  const int* pos;        // device, P entries
  const float* scores;   // [B*H, L]
  uint32_t* keys2;       // workspace [B*H, L]
  int32_t* keep;         // [B*H, C]
};

hipError_t launch_select(const SelectLaunch& L, hipStream_t stream);
size_t select_lds_bytes(int L);

struct CompactLaunch {
  int B, H, C, row_vecs;        // row_vecs = D * elt / 16
  int64_t ks[3], vs[3];         // strides in 16-byte units
  const void* k;
  const void* v;
  const int32_t* keep;
  void* k_out;
  void* v_out;
};

hipError_t launch_compact(const CompactLaunch& L, hipStream_t stream);

}  // namespace nacl
