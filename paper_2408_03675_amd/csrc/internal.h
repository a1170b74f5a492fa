// Internal interface between the C ABI (api.cpp) and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace nacl {

// Sets the thread-local error text of the C ABI and returns status.
int fail_status(int status, const char* fmt, ...);

// Score kernel shape.  A work item spans kScoreWaves waves x tpw tiles of 16
// keys; kScoreWavesPerSimd is the occupancy the register allocation targets.
#ifndef NACL_SCORE_TPW_MAX
#define NACL_SCORE_TPW_MAX 32
#endif
#ifndef NACL_SCORE_WAVES
#define NACL_SCORE_WAVES 2
#endif
// Scheduling: pass-1 items of about GROUP_ITEMS_PER_CU * CUs items form a
// head group; pass-2 items of group g follow pass-1 items of group g + LAG.
#ifndef NACL_SCORE_GROUP_ITEMS_PER_CU
#define NACL_SCORE_GROUP_ITEMS_PER_CU 2
#endif
#ifndef NACL_SCORE_SPLIT_GROUP_ITEMS_PER_CU
#define NACL_SCORE_SPLIT_GROUP_ITEMS_PER_CU 4
#endif
#ifndef NACL_SCORE_LAG
#define NACL_SCORE_LAG 1
#endif
// Tiles per wave and item: chosen per call among kScoreTpwMin * 2^i up to
// kScoreTpwMax.  The workspace is sized for the smallest.
constexpr int kScoreTpwMin = 8;
constexpr int kScoreTpwMax = NACL_SCORE_TPW_MAX;
constexpr int kScoreWavesPerSimd = NACL_SCORE_WAVES;
constexpr int kScoreWaves = 4;  // waves per work-group, each owning a quarter of the item's keys
// Proxy-split variant (bf16, D = 128, at least 128 proxies): the waves of a
// block share one ring of K tiles and split each group of 128 proxies, so an
// item is kSplitChunkKeys keys.
#ifndef NACL_SCORE_SPLIT
#define NACL_SCORE_SPLIT 1
#endif
#ifndef NACL_SPLIT_CHUNK
#define NACL_SPLIT_CHUNK 2048
#endif
constexpr int kSplitChunkKeys = NACL_SPLIT_CHUNK;
inline bool score_uses_split(int dtype, int D, int P) { return NACL_SCORE_SPLIT && dtype == 1 && D == 128 && P >= 128; }
// Proxy rows per group of the wide split kernel (from this many rows on it
// is the one launched), and its items per chunk along the rows.
constexpr int kSplitWideRows = 512;
inline int score_psplit(int dtype, int D, int P) {
  return score_uses_split(dtype, D, P) && P > kSplitWideRows ? (P + kSplitWideRows - 1) / kSplitWideRows : 1;
}
// Few proxy rows (one query row per head in generation-phase eviction, the
// single-token proxy set): the logits of every key are kept in the workspace
// (4 bytes per row and key) instead of reading K again, as long as that is
// cheaper than the second read of a K row.  A work-group of the logit kernel
// takes a chunk of 64 * t keys (t tiles of 16 keys per wave), at most
// kRowsChunkMax, and at least kRowsChunkMin unless the head is shorter.
constexpr int kRowsChunkMax = 1024;
constexpr int kRowsChunkMin = 256;
inline int score_rows_max(int dtype, int D) { return D * (dtype == 0 ? 4 : 2) >= 256 ? 16 : 8; }
inline bool score_uses_rows(int dtype, int D, int P) { return P <= score_rows_max(dtype, D); }
// Chunk length of the logit kernel for B*H heads of L keys: the fewest
// rounds of resident work-groups, the chunks sized to fill them.
int score_rows_chunk(int dtype, int D, int L, int BH, int cus);
// The workspace is sized for the shortest item of either queue kernel (and
// for kRowsChunkMin-key chunks on the few-row path).
constexpr int kScoreMinChunkKeys = std::min(kScoreTpwMin * kScoreWaves * 16, kSplitChunkKeys);

struct ScoreArgs {
  int B, H, L, P;   // P: proxy rows per K/V head = P0 * qg, row r = proxy r / qg of query head r % qg
  int P0, qg;       // proxies, query heads per K/V head
  int64_t qs[3], ks[3];
  const int* pos;   // device, P entries
  int p_last;       // pos[P - 1]
  float c2;         // sm_scale * log2(e)
};

// Work queue of the persistent score kernel (see score.hip).
struct ScoreSched {
  int tpw;               // tiles of 16 keys per wave and item (multiple of 4)
  int chunk_keys;        // keys per item: kScoreWaves * tpw * 16
  int n_chunks;          // key chunks per head
  int heads_per_group;   // heads per scheduling group
  int n_groups;          // B*H / heads_per_group
  int lag;               // pass-2 items of group g follow pass-1 items of group g + lag
  int total_items;
  int n_psplit;          // items per chunk along the proxy rows: 1, or one per group of
                         // kSplitWideRows rows (long proxy lists; the column sums of a chunk
                         // are then added in group order by the chunk's last item)
  int lse_given;         // 1: the caller supplied the log-sum-exp, only pass 2 runs
  uint32_t* queue;       // workspace counter words: queue, status, then per-head counters
  uint32_t* status;      // health words: [0] this call's, [1] sticky; bit 0 set if a pass-2
                         // wait hit its spin limit (never expected)
  uint32_t* head_cnt;    // [B*H]
  float2* partials;      // [B*H, n_chunks, P] base-2 (max, sum)
  float* lse2;           // [B*H, P] base-2 log-sum-exp
  uint32_t* chunk_cnt;   // [B*H, n_chunks] arrivals of a chunk's items (n_psplit > 1)
  float* colpart;        // [B*H, n_chunks, n_psplit, chunk_keys] per-group column sums (n_psplit > 1)
  float* logits;         // few-row path (nullptr otherwise): [B*H, P, logits_stride] raw logits
  int logits_stride;     // L rounded up to a multiple of 4
  int row_pos[16];       // few-row path: position of row r (proxy r / qg), from the host
  int n_clear;           // few-row path: counter words (from queue) its first work-group zeroes
  const float* lse_in;   // caller's log-sum-exp when lse_given
  float lse_mul;         // log2(e) for a natural log-sum-exp
  float* scores;         // [B*H, L]
  // Gumbel keys drawn by the column reduction for the selection that
  // follows (nullptr: none): mode and Philox key and layer as in the
  // selection.
  uint32_t* gkeys;       // [B*H, L]
  int g_mode;
  uint32_t g_k0, g_k1, g_layer;
};

struct ScoreLaunch {
  ScoreArgs args;
  ScoreSched sched;
  int dtype, D;
  const void* q;
  const void* k;
  int n_counter_words;   // words zeroed before the launch, from sched.queue
};

hipError_t launch_score(const ScoreLaunch& L, hipStream_t stream);

// Selection: heads of up to kSelRegMaxL tokens take one work-group each;
// longer heads are cut into slices of kSelSlice tokens, one work-group per
// slice (kSelPer consecutive tokens per thread), and the slices of a head
// exchange histograms and candidate lists through the workspace.
constexpr int kSelThreads = 1024;
constexpr int kSelPer = 16;
constexpr int kSelSlice = kSelThreads * kSelPer;
constexpr int kSelMaxSlices = (1 << 19) / kSelSlice;   // NACL_MAX_L / kSelSlice
constexpr int kSelHistWords = 4096 + 64;               // a slice's published bins and group totals
constexpr int kSelCandMax = 256;                       // bin keys ranked by every work-group
__host__ __device__ inline int select_slices(int L) { return (L + kSelSlice - 1) / kSelSlice; }
// Heads up to this length take the one-work-group kernel (keys in registers).
constexpr int kSelRegMaxL = 32 * kSelThreads;
inline bool select_uses_slices(int L) { return L > kSelRegMaxL; }

struct SelectLaunch {
  int B, H, L, P, n_protect, C, Cp, Cr, sampling;
  uint64_t seed;
  uint32_t layer;
  const int* pos;        // device, P entries
  const float* scores;   // [B*H, L]
  uint32_t* keys2;       // workspace [B*H, L]
  int32_t* keep;         // [B*H, C]
  int keys_ready;        // 1: keys2 already holds the Gumbel keys (drawn by the score kernel)
  int nb;                // slices per head
  uint32_t* sync;        // workspace: word 0 ticket, then (from word 64) one round counter per head; zero at launch
  uint32_t* xhist;       // workspace [B*H, 2, nb, kSelHistWords]: each slice's bins per round (by parity)
  uint32_t* xcand;       // workspace [B*H, 2, kSelCandMax, 2]: the k-th bin's (key, index) per round
  uint32_t* health;      // health words (call's, sticky) or nullptr
  int zero_sync;         // 1: clear the sync words first (0: the score call just did)
};

hipError_t launch_select(const SelectLaunch& L, hipStream_t stream);

struct CompactLaunch {
  int B, H, L, C, row_vecs;     // row_vecs = D * elt / 16
  int64_t ks[3], vs[3];         // strides in 16-byte units
  const void* k;
  const void* v;
  const int32_t* keep;
  void* k_out;                  // == k when in_place
  void* v_out;                  // == v when in_place
  int in_place;                 // 1: rows 0..C-1 of each head of k, v take the kept rows
  uint32_t* health;             // health words (call's, sticky) or nullptr
  int32_t* slots;               // slot form (k_out == k): [B*H, C] old row held by each slot, written
};

hipError_t launch_compact(const CompactLaunch& L, hipStream_t stream);
// Slot form of the in-place update: kept rows below C stay, the kept rows at
// or past C fill the other slots below C (see compact.hip).
hipError_t launch_compact_slots(const CompactLaunch& L, hipStream_t stream);

struct AppendLaunch {
  int B, H, row0, m, row_vecs;
  int64_t ks[3], vs[3];         // cache strides in 16-byte units
  void* k;
  void* v;
  const void* k_new;            // [B, H, m, D] contiguous
  const void* v_new;
};

hipError_t launch_append(const AppendLaunch& L, hipStream_t stream);

// Causal attention of the prefill with each row's log-sum-exp (attention.hip).
struct AttnLaunch {
  int B, H, G, L;      // batch, K/V heads, query heads per K/V head, rows
  int n_tiles;         // 128-row query tiles per head
  float c2;            // logit scale times log2(e)
  int64_t qs[3], ks[3], vs[3];  // element strides (q: per query head)
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  __bf16* out;         // [B, H*G, L, D]
  float* lse;          // [B, H*G, L]
};
// Also writes lse_proxy[b, hq, p] = lse[b, hq, pos[p]] when lse_proxy is set.
hipError_t launch_attention(const AttnLaunch& a, int D, const int32_t* pos, int P, float* lse_proxy,
                            hipStream_t stream);

}  // namespace nacl
