// C ABI of the eviction library: argument validation, workspace layout and
// stream-ordered launch sequencing.  No device memory is allocated here and
// the stream is never synchronised.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "../../include/nacl.h"
#include "internal.h"

#include <algorithm>

namespace {

thread_local char g_detail[512] = "";

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_detail, sizeof(g_detail), fmt, ap);
  va_end(ap);
  return status;
}

}  // namespace

int nacl::fail_status(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_detail, sizeof(g_detail), fmt, ap);
  va_end(ap);
  return status;
}

namespace {

int hip_fail(hipError_t e, const char* what) {
  return fail(NACL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int elt_bytes(int dtype) { return dtype == NACL_F32 ? 4 : 2; }

// Query heads per K/V head (0 means 1), and proxy rows per K/V head.
int q_group_of(const nacl_problem* p) { return p->q_group > 1 ? p->q_group : 1; }
int rows_of(const nacl_problem* p) { return p->P * q_group_of(p); }

int logits_stride(const nacl_problem* p) { return (p->L + 3) / 4 * 4; }

struct Layout {
  size_t cnt, pos, lse, part, keys, colpart, logits, xhist, xcand, total;
  int n_chunks;
  size_t sel_sync_word;   // first word of the selection's sync region inside the counter section
  size_t chunk_cnt_word;  // first word of the proxy-split score's per-chunk arrival counters
  int n_counter_words;    // counter words cleared before the score kernel (all but the sticky word)
};

constexpr int kCounterHeader = 64;  // queue + status words, padded to 256 bytes

Layout layout_of(const nacl_problem* p) {
  Layout l;
  const size_t BH = (size_t)p->B * p->H;
  const int min_chunk = nacl::score_uses_rows(p->dtype, p->D, rows_of(p)) ? nacl::kRowsChunkMin : nacl::kScoreMinChunkKeys;
  l.n_chunks = (p->L + min_chunk - 1) / min_chunk;  // most chunks any call uses
  size_t off = 0;
  l.cnt = off;
  // header, the score's per-head counters, then the selection's ticket
  // (padded to 64 words) and per-head round counters, then (long proxy
  // lists) the score's per-chunk counters
  const int psplit = nacl::score_psplit(p->dtype, p->D, rows_of(p));
  const size_t split_chunks = (p->L + nacl::kSplitChunkKeys - 1) / nacl::kSplitChunkKeys;
  l.sel_sync_word = kCounterHeader + BH;
  l.chunk_cnt_word = kCounterHeader + BH + 64 + BH;
  l.n_counter_words = (int)(l.chunk_cnt_word + (psplit > 1 ? BH * split_chunks : 0));
  off += align_up((size_t)l.n_counter_words * sizeof(uint32_t));
  l.pos = off;
  off += align_up((size_t)p->P * sizeof(int32_t));
  const size_t rows = (size_t)rows_of(p);
  l.lse = off;
  off += align_up(BH * rows * sizeof(float));
  l.part = off;
  off += align_up(BH * l.n_chunks * rows * sizeof(float2));
  l.keys = off;
  off += align_up(BH * p->L * sizeof(uint32_t));
  l.colpart = off;
  if (psplit > 1) off += align_up(BH * split_chunks * psplit * nacl::kSplitChunkKeys * sizeof(float));
  // Few proxy rows: every key's logits, rows padded to a multiple of 4 keys.
  l.logits = off;
  if (nacl::score_uses_rows(p->dtype, p->D, (int)rows))
    off += align_up(BH * rows * (size_t)logits_stride(p) * sizeof(float));
  // The sliced selection of long heads exchanges histograms and candidate
  // lists through these.
  const bool sliced = nacl::select_uses_slices(p->L);
  const size_t nb = nacl::select_slices(p->L);
  l.xhist = off;
  if (sliced) off += align_up(BH * 2 * nb * nacl::kSelHistWords * sizeof(uint32_t));
  l.xcand = off;
  if (sliced) off += align_up(BH * 2 * nacl::kSelCandMax * 2 * sizeof(uint32_t));
  l.total = off;
  return l;
}

// Byte extent [lo, hi) of a strided [B, H, L, D] tensor.
void extent(const void* base, const int64_t st[3], const nacl_problem* p, uintptr_t& lo,
            uintptr_t& hi) {
  const int64_t last = (int64_t)(p->B - 1) * st[0] + (int64_t)(p->H - 1) * st[1] +
                       (int64_t)(p->L - 1) * st[2] + p->D;
  lo = (uintptr_t)base;
  hi = lo + (uintptr_t)last * elt_bytes(p->dtype);
}

bool overlaps(uintptr_t a0, uintptr_t a1, uintptr_t b0, uintptr_t b1) { return a0 < b1 && b0 < a1; }

int check_problem(const nacl_problem* p) {
  if (!p) return fail(NACL_ERR_INVALID_ARG, "problem is NULL");
  if (p->B < 1 || p->H < 1 || p->L < 1)
    return fail(NACL_ERR_INVALID_ARG, "B, H, L must be >= 1 (got %d, %d, %d)", p->B, p->H, p->L);
  if (p->L > NACL_MAX_L) return fail(NACL_ERR_UNSUPPORTED, "L = %d exceeds %d", p->L, NACL_MAX_L);
  if ((int64_t)p->B * p->H > 65535)
    return fail(NACL_ERR_UNSUPPORTED, "B * H = %lld exceeds 65535", (long long)p->B * p->H);
  if (p->D != 64 && p->D != 128) return fail(NACL_ERR_UNSUPPORTED, "D must be 64 or 128 (got %d)", p->D);
  if (p->dtype != NACL_F32 && p->dtype != NACL_BF16)
    return fail(NACL_ERR_INVALID_ARG, "unknown dtype %d", p->dtype);
  if (p->P < 1 || p->P > p->L) return fail(NACL_ERR_INVALID_ARG, "P must lie in [1, L] (got %d)", p->P);
  if (p->P > NACL_MAX_P) return fail(NACL_ERR_UNSUPPORTED, "P = %d exceeds %d", p->P, NACL_MAX_P);
  if (p->q_group < 0 || p->q_group > 64)
    return fail(NACL_ERR_INVALID_ARG, "q_group must lie in [0, 64] (got %d)", p->q_group);
  if ((int64_t)p->B * p->H * q_group_of(p) > 65535)
    return fail(NACL_ERR_UNSUPPORTED, "B * H * q_group exceeds 65535");
  if (p->n_protect < 0 || p->n_protect > p->P)
    return fail(NACL_ERR_INVALID_ARG, "n_protect must lie in [0, P] (got %d)", p->n_protect);
  if (!(std::isfinite(p->sm_scale) && p->sm_scale > 0.f))
    return fail(NACL_ERR_INVALID_ARG, "sm_scale must be finite and > 0");
  if (!p->proxy_pos) return fail(NACL_ERR_INVALID_ARG, "proxy_pos is NULL");
  for (int i = 0; i < p->P; ++i) {
    const int32_t x = p->proxy_pos[i];
    if (x < 0 || x >= p->L)
      return fail(NACL_ERR_INVALID_ARG, "proxy_pos[%d] = %d outside [0, L)", i, x);
    if (i && x <= p->proxy_pos[i - 1])
      return fail(NACL_ERR_INVALID_ARG, "proxy_pos must be strictly increasing (index %d)", i);
  }
  const int eb = elt_bytes(p->dtype);
  const int64_t* strides[3] = {p->q_stride, p->k_stride, p->v_stride};
  const char* names[3] = {"q_stride", "k_stride", "v_stride"};
  for (int t = 0; t < 3; ++t)
    for (int i = 0; i < 3; ++i) {
      if (strides[t][i] < 0) return fail(NACL_ERR_INVALID_ARG, "%s[%d] < 0", names[t], i);
      if ((strides[t][i] * eb) % 16)
        return fail(NACL_ERR_INVALID_ARG, "%s[%d] * element size must be a multiple of 16 bytes",
                    names[t], i);
    }
  // The score kernel addresses one head's K rows through a buffer
  // descriptor with 32-bit byte offsets.
  if ((int64_t)(p->L - 1) * p->k_stride[2] * eb + (int64_t)p->D * eb >= ((int64_t)1 << 31))
    return fail(NACL_ERR_UNSUPPORTED, "one head's K rows span 2 GiB or more (L * k_stride[2])");
  return NACL_OK;
}

bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

int check_ws(const nacl_problem* p, const void* ws, size_t ws_bytes) {
  const size_t need = layout_of(p).total;
  if (ws_bytes < need)
    return fail(NACL_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, need);
  if (!ws) return fail(NACL_ERR_WORKSPACE, "workspace is NULL");
  if ((uintptr_t)ws % kAlign) return fail(NACL_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return NACL_OK;
}

int check_select_counts(const nacl_problem* p, int32_t C, int32_t Cr, int32_t sampling) {
  if (C < 0 || C > p->L) return fail(NACL_ERR_INVALID_ARG, "C must lie in [0, L] (got %d)", C);
  if (Cr < 0) return fail(NACL_ERR_INVALID_ARG, "Cr must be >= 0 (got %d)", Cr);
  if ((int64_t)p->n_protect + Cr > C)
    return fail(NACL_ERR_INVALID_ARG, "n_protect + Cr = %lld exceeds C = %d",
                (long long)p->n_protect + Cr, C);
  if (sampling < NACL_SAMPLE_SOFTMAX || sampling > NACL_SAMPLE_UNIFORM)
    return fail(NACL_ERR_INVALID_ARG, "unknown sampling mode %d", sampling);
  return NACL_OK;
}

// Device pointer of the proxy positions; stages the host array into the
// workspace when the caller gave no device copy.
int stage_positions(const nacl_problem* p, char* ws, const Layout& l, hipStream_t stream,
                    const int** out) {
  if (p->proxy_pos_dev) {
    *out = p->proxy_pos_dev;
    return NACL_OK;
  }
  int32_t* dst = reinterpret_cast<int32_t*>(ws + l.pos);
  hipError_t e = hipMemcpyAsync(dst, p->proxy_pos, (size_t)p->P * sizeof(int32_t),
                                hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return hip_fail(e, "staging proxy positions");
  *out = dst;
  return NACL_OK;
}

// Heads per scheduling group: the largest divisor of B*H whose items fill
// about one round of resident work-groups.
int heads_per_group(int BH, int n_chunks, int target_items) {
  int best = 1;
  for (int g = 1; g <= BH; ++g)
    if (BH % g == 0 && (int64_t)g * n_chunks <= target_items) best = g;
  return best;
}

// Gumbel keys for the selection that follows, drawn by the score kernel
// (inside nacl_evict only).
struct KeyDraw {
  bool on = false;
  int32_t sampling = 0;
  uint64_t seed = 0;
  uint32_t layer = 0;
};

int run_score(const nacl_problem* p, const void* q, const void* k, const float* lse, float* scores,
              char* ws, const Layout& l, const int* pos_dev, hipStream_t stream, const KeyDraw& kd = KeyDraw{}) {
  nacl::ScoreLaunch s{};
  s.args.B = p->B;
  s.args.H = p->H;
  s.args.L = p->L;
  s.args.P = rows_of(p);  // proxy rows per K/V head
  s.args.P0 = p->P;
  s.args.qg = q_group_of(p);
  for (int i = 0; i < 3; ++i) {
    s.args.qs[i] = p->q_stride[i];
    s.args.ks[i] = p->k_stride[i];
  }
  s.args.pos = pos_dev;
  s.args.p_last = p->proxy_pos[p->P - 1];
  s.args.c2 = (float)((double)p->sm_scale * 1.4426950408889634);
  s.dtype = p->dtype;
  s.D = p->D;
  s.q = q;
  s.k = k;
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return fail(NACL_ERR_HIP, "querying the device");
  const int BH = p->B * p->H;
  nacl::ScoreSched& sc = s.sched;
  sc.lse_given = lse != nullptr;
  uint32_t* words = reinterpret_cast<uint32_t*>(ws + l.cnt);
  sc.queue = words;
  sc.status = words + 1;
  sc.head_cnt = words + kCounterHeader;
  sc.scores = scores;
  sc.gkeys = kd.on ? reinterpret_cast<uint32_t*>(ws + l.keys) : nullptr;
  sc.g_mode = kd.sampling;
  sc.g_k0 = (uint32_t)(kd.seed & 0xFFFFFFFFu);
  sc.g_k1 = (uint32_t)(kd.seed >> 32);
  sc.g_layer = kd.layer;
  s.n_counter_words = l.n_counter_words;
  // Item size: the largest tpw whose items still number at least four per
  // resident work-group (two per CU); long items amortise the per-item Q
  // loads, partial stores and pipeline fill, too few leave a long tail.
  const int passes = sc.lse_given ? 1 : 2;
  sc.tpw = nacl::kScoreTpwMin;
  for (int t = nacl::kScoreTpwMin * 2; t <= nacl::kScoreTpwMax; t *= 2) {
    const int ck = t * nacl::kScoreWaves * 16;
    const int64_t items = (int64_t)passes * BH * ((p->L + ck - 1) / ck);
    if (items >= 4 * 2 * (int64_t)cus) sc.tpw = t;
  }
  sc.chunk_keys = sc.tpw * nacl::kScoreWaves * 16;
  // The proxy-split kernel takes fixed items of kSplitChunkKeys keys.
  if (nacl::score_uses_split(p->dtype, p->D, rows_of(p))) sc.chunk_keys = nacl::kSplitChunkKeys;
  sc.n_chunks = (p->L + sc.chunk_keys - 1) / sc.chunk_keys;  // <= l.n_chunks
  sc.n_psplit = nacl::score_psplit(p->dtype, p->D, rows_of(p));
  sc.chunk_cnt = words + l.chunk_cnt_word;
  sc.colpart = reinterpret_cast<float*>(ws + l.colpart);
  const int group_items = nacl::score_uses_split(p->dtype, p->D, rows_of(p)) ? NACL_SCORE_SPLIT_GROUP_ITEMS_PER_CU
                                                                       : NACL_SCORE_GROUP_ITEMS_PER_CU;
  sc.heads_per_group = heads_per_group(BH, sc.n_chunks * sc.n_psplit, group_items * cus);
  sc.n_groups = BH / sc.heads_per_group;
  sc.lag = std::min(NACL_SCORE_LAG, sc.n_groups);
  sc.total_items = passes * BH * sc.n_chunks * sc.n_psplit;
  sc.partials = reinterpret_cast<float2*>(ws + l.part);
  sc.lse2 = reinterpret_cast<float*>(ws + l.lse);
  sc.lse_in = lse;
  sc.lse_mul = 1.4426950408889634f;
  if (!sc.lse_given && nacl::score_uses_rows(p->dtype, p->D, rows_of(p))) {
    // Few proxy rows: K is read once and the logits are kept (see score.hip).
    sc.logits = reinterpret_cast<float*>(ws + l.logits);
    sc.logits_stride = logits_stride(p);
    sc.chunk_keys = nacl::score_rows_chunk(p->dtype, p->D, p->L, BH, cus);
    sc.n_chunks = (p->L + sc.chunk_keys - 1) / sc.chunk_keys;  // <= l.n_chunks
    for (int r = 0; r < rows_of(p); ++r) sc.row_pos[r] = p->proxy_pos[r / q_group_of(p)];
  }
  hipError_t e = nacl::launch_score(s, stream);
  if (e != hipSuccess) return hip_fail(e, "score kernel");
  return NACL_OK;
}

int run_select(const nacl_problem* p, const float* scores, int32_t C, int32_t Cr, int32_t sampling,
               uint64_t seed, uint32_t layer, int32_t* keep, char* ws, const Layout& l,
               const int* pos_dev, hipStream_t stream, bool keys_ready = false, bool sync_zeroed = false) {
  if (C == 0) return NACL_OK;
  nacl::SelectLaunch s{};
  s.B = p->B;
  s.H = p->H;
  s.L = p->L;
  s.P = p->P;
  s.n_protect = p->n_protect;
  s.C = C;
  s.Cr = Cr;
  s.Cp = C - p->n_protect - Cr;
  s.sampling = sampling;
  s.seed = seed;
  s.layer = layer;
  s.pos = pos_dev;
  s.scores = scores;
  s.keys2 = reinterpret_cast<uint32_t*>(ws + l.keys);
  s.keep = keep;
  s.keys_ready = keys_ready ? 1 : 0;
  s.nb = nacl::select_slices(p->L);
  uint32_t* words = reinterpret_cast<uint32_t*>(ws + l.cnt);
  s.sync = words + l.sel_sync_word;
  s.xhist = reinterpret_cast<uint32_t*>(ws + l.xhist);
  s.xcand = reinterpret_cast<uint32_t*>(ws + l.xcand);
  s.health = words + 1;
  s.zero_sync = !sync_zeroed;
  hipError_t e = nacl::launch_select(s, stream);
  if (e != hipSuccess) return hip_fail(e, "select kernels");
  return NACL_OK;
}

// Compaction outputs either alias the inputs exactly (k_out == k and
// v_out == v: in place, the kept rows move to the front of each head in the
// input's own layout) or overlap no input at all.
int check_compact_args(const nacl_problem* p, const void* k, const void* v, const int32_t* keep,
                       int32_t C, const void* k_out, const void* v_out, bool* in_place) {
  *in_place = false;
  if (C < 0 || C > p->L) return fail(NACL_ERR_INVALID_ARG, "C must lie in [0, L] (got %d)", C);
  if (C == 0) return NACL_OK;
  if (!k || !v || !keep || !k_out || !v_out)
    return fail(NACL_ERR_INVALID_ARG, "compaction pointers must be non-NULL");
  if (!aligned16(k) || !aligned16(v) || !aligned16(k_out) || !aligned16(v_out))
    return fail(NACL_ERR_INVALID_ARG, "K, V, k_out, v_out must be 16-byte aligned");
  uintptr_t k0, k1, v0, v1;
  extent(k, p->k_stride, p, k0, k1);
  extent(v, p->v_stride, p, v0, v1);
  const uintptr_t kk0 = (uintptr_t)keep, kk1 = kk0 + (uintptr_t)p->B * p->H * C * 4;
  if (overlaps(kk0, kk1, k0, k1) || overlaps(kk0, kk1, v0, v1))
    return fail(NACL_ERR_INVALID_ARG, "keep_idx overlaps K or V");
  if (k_out == k || v_out == v) {
    if (k_out != k || v_out != v)
      return fail(NACL_ERR_INVALID_ARG, "in-place compaction needs k_out == k and v_out == v");
    if (overlaps(k0, k1, v0, v1))
      return fail(NACL_ERR_INVALID_ARG, "in-place compaction needs K and V in disjoint memory");
    *in_place = true;
    return NACL_OK;
  }
  const uintptr_t ob = (uintptr_t)p->B * p->H * C * p->D * elt_bytes(p->dtype);
  const uintptr_t ko = (uintptr_t)k_out, vo = (uintptr_t)v_out;
  if (overlaps(ko, ko + ob, k0, k1) || overlaps(ko, ko + ob, v0, v1) || overlaps(vo, vo + ob, k0, k1) ||
      overlaps(vo, vo + ob, v0, v1) || overlaps(ko, ko + ob, vo, vo + ob) ||
      overlaps(ko, ko + ob, kk0, kk1) || overlaps(vo, vo + ob, kk0, kk1))
    return fail(NACL_ERR_INVALID_ARG, "k_out / v_out overlap an input or each other");
  return NACL_OK;
}

int run_compact(const nacl_problem* p, const void* k, const void* v, const int32_t* keep, int32_t C,
                void* k_out, void* v_out, bool in_place, uint32_t* health, hipStream_t stream) {
  if (C == 0) return NACL_OK;
  nacl::CompactLaunch c{};
  const int eb = elt_bytes(p->dtype);
  c.B = p->B;
  c.H = p->H;
  c.L = p->L;
  c.C = C;
  c.row_vecs = p->D * eb / 16;
  for (int i = 0; i < 3; ++i) {
    c.ks[i] = p->k_stride[i] * eb / 16;
    c.vs[i] = p->v_stride[i] * eb / 16;
  }
  c.k = k;
  c.v = v;
  c.keep = keep;
  c.k_out = k_out;
  c.v_out = v_out;
  c.in_place = in_place ? 1 : 0;
  c.health = health;
  hipError_t e = nacl::launch_compact(c, stream);
  if (e != hipSuccess) return hip_fail(e, "compact kernel");
  return NACL_OK;
}

// The slot form's arguments: an in-place update of k, v with keep_idx read
// and slot_idx written, neither overlapping the caches or each other.
int check_slots_args(const nacl_problem* p, const void* k, const void* v, const int32_t* keep,
                     int32_t C, const int32_t* slots) {
  if (C < 0 || C > p->L) return fail(NACL_ERR_INVALID_ARG, "C must lie in [0, L] (got %d)", C);
  if (C == 0) return NACL_OK;
  if (!k || !v || !keep || !slots) return fail(NACL_ERR_INVALID_ARG, "slot-form pointers must be non-NULL");
  if (!aligned16(k) || !aligned16(v)) return fail(NACL_ERR_INVALID_ARG, "K and V must be 16-byte aligned");
  uintptr_t k0, k1, v0, v1;
  extent(k, p->k_stride, p, k0, k1);
  extent(v, p->v_stride, p, v0, v1);
  const uintptr_t n = (uintptr_t)p->B * p->H * C * 4;
  const uintptr_t a0 = (uintptr_t)keep, s0 = (uintptr_t)slots;
  if (overlaps(k0, k1, v0, v1)) return fail(NACL_ERR_INVALID_ARG, "the slot form needs K and V in disjoint memory");
  if (overlaps(a0, a0 + n, k0, k1) || overlaps(a0, a0 + n, v0, v1) || overlaps(s0, s0 + n, k0, k1) ||
      overlaps(s0, s0 + n, v0, v1) || overlaps(a0, a0 + n, s0, s0 + n))
    return fail(NACL_ERR_INVALID_ARG, "keep_idx / slot_idx overlap K, V or each other");
  return NACL_OK;
}

int run_compact_slots(const nacl_problem* p, void* k, void* v, const int32_t* keep, int32_t C, int32_t* slots,
                      uint32_t* health, hipStream_t stream) {
  if (C == 0) return NACL_OK;
  nacl::CompactLaunch c{};
  const int eb = elt_bytes(p->dtype);
  c.B = p->B;
  c.H = p->H;
  c.L = p->L;
  c.C = C;
  c.row_vecs = p->D * eb / 16;
  for (int i = 0; i < 3; ++i) {
    c.ks[i] = p->k_stride[i] * eb / 16;
    c.vs[i] = p->v_stride[i] * eb / 16;
  }
  c.k = k;
  c.v = v;
  c.keep = keep;
  c.k_out = k;
  c.v_out = v;
  c.in_place = 1;
  c.health = health;
  c.slots = slots;
  hipError_t e = nacl::launch_compact_slots(c, stream);
  if (e != hipSuccess) return hip_fail(e, "slot-form compact kernel");
  return NACL_OK;
}

}  // namespace

extern "C" {

size_t nacl_workspace_bytes(const nacl_problem* p) {
  if (check_problem(p) != NACL_OK) return 0;
  return layout_of(p).total;
}

int nacl_score(const nacl_problem* p, const void* q, const void* k, const float* lse, float* scores,
               void* ws, size_t ws_bytes, void* stream) {
  g_detail[0] = 0;
  int st = check_problem(p);
  if (st) return st;
  if (!q || !k || !scores) return fail(NACL_ERR_INVALID_ARG, "q, k and scores must be non-NULL");
  if (!aligned16(q) || !aligned16(k)) return fail(NACL_ERR_INVALID_ARG, "q and k must be 16-byte aligned");
  if ((st = check_ws(p, ws, ws_bytes))) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Layout l = layout_of(p);
  const int* pos_dev = nullptr;
  if ((st = stage_positions(p, static_cast<char*>(ws), l, s, &pos_dev))) return st;
  return run_score(p, q, k, lse, scores, static_cast<char*>(ws), l, pos_dev, s);
}

int nacl_select(const nacl_problem* p, const float* scores, int32_t C, int32_t Cr, int32_t sampling,
                uint64_t seed, uint32_t layer, int32_t* keep_idx, void* ws, size_t ws_bytes,
                void* stream) {
  g_detail[0] = 0;
  int st = check_problem(p);
  if (st) return st;
  if ((st = check_select_counts(p, C, Cr, sampling))) return st;
  if (C > 0 && (!scores || !keep_idx))
    return fail(NACL_ERR_INVALID_ARG, "scores and keep_idx must be non-NULL");
  if ((st = check_ws(p, ws, ws_bytes))) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Layout l = layout_of(p);
  const int* pos_dev = nullptr;
  if ((st = stage_positions(p, static_cast<char*>(ws), l, s, &pos_dev))) return st;
  return run_select(p, scores, C, Cr, sampling, seed, layer, keep_idx, static_cast<char*>(ws), l,
                    pos_dev, s);
}

int nacl_compact(const nacl_problem* p, const void* k, const void* v, const int32_t* keep_idx,
                 int32_t C, void* k_out, void* v_out, void* stream) {
  g_detail[0] = 0;
  int st = check_problem(p);
  if (st) return st;
  bool in_place = false;
  if ((st = check_compact_args(p, k, v, keep_idx, C, k_out, v_out, &in_place))) return st;
  return run_compact(p, k, v, keep_idx, C, k_out, v_out, in_place, nullptr, static_cast<hipStream_t>(stream));
}

int nacl_compact_slots(const nacl_problem* p, void* k, void* v, const int32_t* keep_idx, int32_t C,
                       int32_t* slot_idx, void* stream) {
  g_detail[0] = 0;
  int st = check_problem(p);
  if (st) return st;
  if ((st = check_slots_args(p, k, v, keep_idx, C, slot_idx))) return st;
  return run_compact_slots(p, k, v, keep_idx, C, slot_idx, nullptr, static_cast<hipStream_t>(stream));
}

int nacl_append(const nacl_problem* p, void* k, void* v, int32_t row0, const void* k_new,
                const void* v_new, int32_t m, void* stream) {
  g_detail[0] = 0;
  int st = check_problem(p);
  if (st) return st;
  if (m < 0 || row0 < 0 || (int64_t)row0 + m > p->L)
    return fail(NACL_ERR_INVALID_ARG, "rows [%d, %lld) must lie in [0, L = %d)", row0, (long long)row0 + m, p->L);
  if (m == 0) return NACL_OK;
  if (!k || !v || !k_new || !v_new) return fail(NACL_ERR_INVALID_ARG, "append pointers must be non-NULL");
  if (!aligned16(k) || !aligned16(v) || !aligned16(k_new) || !aligned16(v_new))
    return fail(NACL_ERR_INVALID_ARG, "K, V, k_new, v_new must be 16-byte aligned");
  uintptr_t k0, k1, v0, v1;
  extent(k, p->k_stride, p, k0, k1);
  extent(v, p->v_stride, p, v0, v1);
  const uintptr_t nb = (uintptr_t)p->B * p->H * m * p->D * elt_bytes(p->dtype);
  const uintptr_t kn = (uintptr_t)k_new, vn = (uintptr_t)v_new;
  if (overlaps(kn, kn + nb, k0, k1) || overlaps(kn, kn + nb, v0, v1) || overlaps(vn, vn + nb, k0, k1) ||
      overlaps(vn, vn + nb, v0, v1) || overlaps(k0, k1, v0, v1))
    return fail(NACL_ERR_INVALID_ARG, "k_new / v_new overlap the cache, or K overlaps V");
  nacl::AppendLaunch a{};
  const int eb = elt_bytes(p->dtype);
  a.B = p->B;
  a.H = p->H;
  a.row0 = row0;
  a.m = m;
  a.row_vecs = p->D * eb / 16;
  for (int i = 0; i < 3; ++i) {
    a.ks[i] = p->k_stride[i] * eb / 16;
    a.vs[i] = p->v_stride[i] * eb / 16;
  }
  a.k = k;
  a.v = v;
  a.k_new = k_new;
  a.v_new = v_new;
  hipError_t e = nacl::launch_append(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "append kernel");
  return NACL_OK;
}

int nacl_attention(const nacl_problem* p, const void* q, const void* k, const void* v, void* out, float* lse,
                   float* lse_proxy, void* stream) {
  g_detail[0] = 0;
  int st = check_problem(p);
  if (st) return st;
  if (p->dtype != NACL_BF16) return fail(NACL_ERR_UNSUPPORTED, "attention takes bf16 Q, K, V only");
  if (!q || !k || !v || !out || !lse) return fail(NACL_ERR_INVALID_ARG, "q, k, v, out and lse must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
    return fail(NACL_ERR_INVALID_ARG, "q, k, v and out must be 16-byte aligned");
  if (lse_proxy && !p->proxy_pos_dev)
    return fail(NACL_ERR_INVALID_ARG, "lse_proxy needs proxy_pos_dev (the proxy rows on the device)");
  // Each head's rows are addressed through buffer descriptors with 32-bit
  // byte offsets, up to 127 rows past L.
  const int64_t rows[3] = {p->q_stride[2], p->k_stride[2], p->v_stride[2]};
  for (int t = 0; t < 3; ++t) {
    if (rows[t] < p->D) return fail(NACL_ERR_INVALID_ARG, "attention needs row strides of at least D");
    if ((int64_t)p->L * rows[t] * 2 >= ((int64_t)1 << 31) || rows[t] * 2 >= ((int64_t)1 << 24))
      return fail(NACL_ERR_UNSUPPORTED, "one head's rows span 2 GiB or more");
  }
  const int g = q_group_of(p);
  const int64_t Hq = (int64_t)p->H * g;
  const uintptr_t o0 = (uintptr_t)out, o1 = o0 + (uintptr_t)(p->B * Hq * p->L * p->D * 2);
  const uintptr_t l0 = (uintptr_t)lse, l1 = l0 + (uintptr_t)(p->B * Hq * p->L * 4);
  const uintptr_t x0 = (uintptr_t)lse_proxy, x1 = x0 + (lse_proxy ? (uintptr_t)(p->B * Hq * p->P * 4) : 0);
  nacl_problem pq = *p;  // Q's extent: H * q_group heads
  pq.H = (int32_t)Hq;
  uintptr_t q0, q1, k0, k1, v0, v1;
  extent(q, p->q_stride, &pq, q0, q1);
  extent(k, p->k_stride, p, k0, k1);
  extent(v, p->v_stride, p, v0, v1);
  const uintptr_t ins[3][2] = {{q0, q1}, {k0, k1}, {v0, v1}};
  for (int t = 0; t < 3; ++t)
    if (overlaps(o0, o1, ins[t][0], ins[t][1]) || overlaps(l0, l1, ins[t][0], ins[t][1]) ||
        (lse_proxy && overlaps(x0, x1, ins[t][0], ins[t][1])))
      return fail(NACL_ERR_INVALID_ARG, "out, lse or lse_proxy overlaps Q, K or V");
  if (overlaps(o0, o1, l0, l1) || (lse_proxy && (overlaps(x0, x1, o0, o1) || overlaps(x0, x1, l0, l1))))
    return fail(NACL_ERR_INVALID_ARG, "out, lse and lse_proxy must not overlap");
  nacl::AttnLaunch a{};
  a.B = p->B;
  a.H = p->H;
  a.G = g;
  a.L = p->L;
  a.n_tiles = (p->L + 127) / 128;
  a.c2 = p->sm_scale * 1.4426950408889634f;
  for (int i = 0; i < 3; ++i) {
    a.qs[i] = p->q_stride[i];
    a.ks[i] = p->k_stride[i];
    a.vs[i] = p->v_stride[i];
  }
  a.q = static_cast<const __bf16*>(q);
  a.k = static_cast<const __bf16*>(k);
  a.v = static_cast<const __bf16*>(v);
  a.out = static_cast<__bf16*>(out);
  a.lse = lse;
  if ((int64_t)a.B * Hq * a.n_tiles >= ((int64_t)1 << 31))
    return fail(NACL_ERR_UNSUPPORTED, "too many query tiles");
  hipError_t e = nacl::launch_attention(a, p->D, p->proxy_pos_dev, p->P, lse_proxy, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "attention kernel");
  return NACL_OK;
}

int nacl_evict(const nacl_problem* p, const void* q, const void* k, const void* v, int32_t C,
               int32_t Cr, int32_t sampling, uint64_t seed, uint32_t layer, float* scores,
               int32_t* keep_idx, void* k_out, void* v_out, void* ws, size_t ws_bytes,
               void* stream) {
  g_detail[0] = 0;
  int st = check_problem(p);
  if (st) return st;
  if ((st = check_select_counts(p, C, Cr, sampling))) return st;
  if (!q || !scores) return fail(NACL_ERR_INVALID_ARG, "q and scores must be non-NULL");
  if (!aligned16(q)) return fail(NACL_ERR_INVALID_ARG, "q must be 16-byte aligned");
  if (C > 0 && !keep_idx) return fail(NACL_ERR_INVALID_ARG, "keep_idx must be non-NULL");
  bool in_place = false;
  if ((st = check_compact_args(p, k, v, keep_idx, C, k_out, v_out, &in_place))) return st;
  if (!k) return fail(NACL_ERR_INVALID_ARG, "k must be non-NULL");
  if ((st = check_ws(p, ws, ws_bytes))) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Layout l = layout_of(p);
  char* w = static_cast<char*>(ws);
  const int* pos_dev = nullptr;
  if ((st = stage_positions(p, w, l, s, &pos_dev))) return st;
  // The column reduction also draws the Gumbel keys (the selection's key
  // kernel is then skipped); the keys are the same bits either way.
  KeyDraw kd;
  kd.on = C > 0 && Cr > 0;
  kd.sampling = sampling;
  kd.seed = seed;
  kd.layer = layer;
  if ((st = run_score(p, q, k, nullptr, scores, w, l, pos_dev, s, kd))) return st;
  // The score kernel's counter clearing also cleared the selection's.
  if ((st = run_select(p, scores, C, Cr, sampling, seed, layer, keep_idx, w, l, pos_dev, s, kd.on, true))) return st;
  uint32_t* health = reinterpret_cast<uint32_t*>(w + l.cnt) + 1;
  return run_compact(p, k, v, keep_idx, C, k_out, v_out, in_place, health, s);
}

int nacl_evict_slots(const nacl_problem* p, const void* q, void* k, void* v, int32_t C, int32_t Cr,
                     int32_t sampling, uint64_t seed, uint32_t layer, float* scores, int32_t* keep_idx,
                     int32_t* slot_idx, void* ws, size_t ws_bytes, void* stream) {
  g_detail[0] = 0;
  int st = check_problem(p);
  if (st) return st;
  if ((st = check_select_counts(p, C, Cr, sampling))) return st;
  if (!q || !scores) return fail(NACL_ERR_INVALID_ARG, "q and scores must be non-NULL");
  if (!aligned16(q)) return fail(NACL_ERR_INVALID_ARG, "q must be 16-byte aligned");
  if ((st = check_slots_args(p, k, v, keep_idx, C, slot_idx))) return st;
  if (!k) return fail(NACL_ERR_INVALID_ARG, "k must be non-NULL");
  if ((st = check_ws(p, ws, ws_bytes))) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Layout l = layout_of(p);
  char* w = static_cast<char*>(ws);
  const int* pos_dev = nullptr;
  if ((st = stage_positions(p, w, l, s, &pos_dev))) return st;
  KeyDraw kd;
  kd.on = C > 0 && Cr > 0;
  kd.sampling = sampling;
  kd.seed = seed;
  kd.layer = layer;
  if ((st = run_score(p, q, k, nullptr, scores, w, l, pos_dev, s, kd))) return st;
  if ((st = run_select(p, scores, C, Cr, sampling, seed, layer, keep_idx, w, l, pos_dev, s, kd.on, true))) return st;
  uint32_t* health = reinterpret_cast<uint32_t*>(w + l.cnt) + 1;
  return run_compact_slots(p, k, v, keep_idx, C, slot_idx, health, s);
}

const char* nacl_status_string(int status) {
  switch (status) {
    case NACL_OK: return "ok";
    case NACL_ERR_INVALID_ARG: return "invalid argument";
    case NACL_ERR_UNSUPPORTED: return "unsupported";
    case NACL_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case NACL_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* nacl_last_error_detail(void) { return g_detail; }

int nacl_version(void) { return NACL_VERSION; }

}  // extern "C"
