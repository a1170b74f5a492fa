/*
 * nacl.h -- C ABI of the MI355X (gfx950) implementation of NaCl's one-shot
 * encoding-phase KV-cache eviction.
 *
 * Paper: Chen et al., "NaCl: A General and Effective KV Cache Eviction
 * Framework for LLMs at Inference Time", arXiv 2408.03675.
 *
 * For every layer l, batch row b and head h (heads are independent; head-wise
 * eviction, Section 6.3):
 *   score   F[j] = sum over proxy tokens p_i of softmax_j(s * <Q[p_i], K[j]>),
 *           keys j <= p_i only (causal)            -- Section 5.1, F_score
 *   select  S = Pi  u  top-Cp of F over R  u  Cr tokens sampled without
 *           replacement from Softmax(F) over the rest, |S| = C
 *                                                  -- Section 5.1 argmax,
 *                                                     Section 5.2, Algorithm 1
 *   compact K' = K[S], V' = V[S]                   -- Section 3, encoding phase
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Device pointers are HIP device memory of the current device.  Host
 *   pointers are marked HOST.  The library allocates nothing, keeps no state
 *   between calls (apart from the thread-local error text), never
 *   synchronises, and enqueues all work on `stream` (a hipStream_t; NULL is
 *   the default stream).  Outputs are complete once the stream reaches them.
 * - Every function returns a nacl_status.  Arguments are validated on the
 *   host before anything is enqueued; on any error nothing is enqueued and
 *   outputs are untouched.  nacl_last_error_detail() explains the failure.
 * - Q, K, V are [B, H, L, D] tensors addressed by element strides for
 *   (b, h, l); d is contiguous.  Base pointers and every row start must be
 *   16-byte aligned.
 * - Scores are fp32 [B, H, L] contiguous; keep_idx is int32 [B, H, C]
 *   contiguous, strictly ascending per head; k_out / v_out are [B, H, C, D]
 *   contiguous in the input dtype and overlap no input, or are K and V
 *   themselves (in-place compaction, see nacl_compact).
 * - Overlapping calls that share a workspace race; give concurrent calls
 *   their own workspaces.
 */
#ifndef NACL_H
#define NACL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define NACL_VERSION 2
#define NACL_MAX_P 4096          /* proxy tokens per head */
#define NACL_MAX_L (1 << 19)     /* prompt length */

typedef enum {
  NACL_OK = 0,
  NACL_ERR_INVALID_ARG = 1,  /* an argument is out of range or inconsistent */
  NACL_ERR_UNSUPPORTED = 2,  /* valid in principle, not supported by the library */
  NACL_ERR_WORKSPACE = 3,    /* workspace missing, misaligned or too small */
  NACL_ERR_HIP = 4           /* a HIP runtime call or kernel launch failed */
} nacl_status;

typedef enum { NACL_F32 = 0, NACL_BF16 = 1 } nacl_dtype;

/* Distribution of the random eviction (Section 5.2).  SOFTMAX is the paper's
 * Softmax(F) (weights exp(F[j])); PROPORTIONAL uses weights F[j]; UNIFORM
 * uses equal weights (the ablation's uniform sampling). */
typedef enum {
  NACL_SAMPLE_SOFTMAX = 0,
  NACL_SAMPLE_PROPORTIONAL = 1,
  NACL_SAMPLE_UNIFORM = 2
} nacl_sampling;

/* The eviction problem of one layer (Section 3, encoding-phase eviction). */
typedef struct nacl_problem {
  int32_t B, H, L, D;        /* batch, heads, prompt length, head dim (64 or 128) */
  int32_t dtype;             /* nacl_dtype of Q, K, V (and of k_out, v_out) */
  int32_t P;                 /* number of proxy tokens, 1 <= P <= min(L, NACL_MAX_P) */
  int32_t n_protect;         /* the last n_protect proxies are always kept (0..P);
                                the paper keeps all proxies: n_protect = P */
  float sm_scale;            /* logit scale s > 0, normally 1/sqrt(D) */
  int64_t q_stride[3];       /* element strides of Q for b, h, l */
  int64_t k_stride[3];       /* element strides of K for b, h, l */
  int64_t v_stride[3];       /* element strides of V for b, h, l */
  const int32_t* proxy_pos;  /* HOST, P positions, strictly increasing, in [0, L);
                                shared by every b and h (Section 5.1) */
  const int32_t* proxy_pos_dev; /* optional DEVICE copy of proxy_pos (same values);
                                NULL: the library stages proxy_pos through the
                                workspace with a stream-ordered copy */
  int32_t q_group;           /* query heads per K/V head (grouped-query attention;
                                0 or 1: multi-head, 1..64).  H counts K/V heads:
                                K, V, scores, keep_idx and the outputs have H
                                heads, Q has H * q_group heads (q_stride[1] steps
                                one query head), and K/V head h is scored by the
                                proxy rows of query heads h*q_group ..
                                h*q_group + q_group - 1, so its score mass is
                                P * q_group.  lse (nacl_score) is then
                                [B, H * q_group, P]. */
} nacl_problem;

/* Workspace bytes the score, select and evict calls need for problem *p
 * (0 on invalid input).  The workspace is device memory, 256-byte aligned,
 * owned by the caller; its contents need no initialisation. */
size_t nacl_workspace_bytes(const nacl_problem* p);

/* Proxy-token scores F (Section 5.1, F_score; Appendix A.7 for the blockwise
 * recomputation).  q, k: device [B,H,L,D].  lse: optional device fp32
 * [B,H,P], the natural log-sum-exp of each proxy row's scaled causal logits
 * as a FlashAttention-2 forward returns it (Appendix A.7, Algorithm 2); with
 * it only the column reduction runs.  NULL: the library computes it (two
 * passes over K).  scores: device fp32 [B,H,L], fully overwritten; keys after
 * the last proxy get 0.
 * Health words (score and evict calls): uint32 word 1 of the workspace
 * (byte offset 4) is this call's, cleared by the call itself; word 2 (byte
 * offset 8) is sticky: every call ORs its bits into it and no call clears it,
 * so it covers every call since the caller last zeroed it (zero it when the
 * workspace is allocated; the Python binding does).  Bit 0: a wave gave up
 * waiting for a head's log-sum-exp after its bounded spin.  Bit 2 (evict
 * only): the compaction met a keep index outside [0, L).  Bit 3 (evict only,
 * heads of more than 32768 tokens): a work-group of the selection gave up
 * waiting for the other slices of its head, or its search for a threshold
 * ran out of rounds.  Never expected; whenever a call's word is non-zero once
 * the stream has completed it, that call's scores, keep_idx, k_out and v_out
 * are not valid. */
int nacl_score(const nacl_problem* p, const void* q, const void* k, const float* lse,
               float* scores, void* ws, size_t ws_bytes, void* stream);

/* Keep set S per head (Section 5.1 argmax, Section 5.2, Algorithm 1).
 * scores: device fp32 [B,H,L] (finite, >= 0).  C: total budget, with
 * n_protect + Cr <= C <= L; Cr: tokens drawn by the random eviction;
 * Cp = C - n_protect - Cr come from the top-Cp scores over the unprotected
 * tokens.  Ties go to the lower token index.  The random draw uses
 * Philox4x32-10 with key = seed and counter (j/4, h, b, layer), token j
 * taking word j mod 4, u = (word + 1/2) / 2^32, Gumbel g = -ln(-ln u) in
 * binary64, key = binary32(log-weight + g); the Cr largest keys among the
 * remaining tokens are kept (Gumbel-top-k).  keep_idx: device int32 [B,H,C],
 * ascending. */
int nacl_select(const nacl_problem* p, const float* scores, int32_t C, int32_t Cr,
                int32_t sampling, uint64_t seed, uint32_t layer, int32_t* keep_idx,
                void* ws, size_t ws_bytes, void* stream);

/* Cache update K0, V0 <- K_S, V_S (Section 3).  k, v: device [B,H,L,D] with
 * the problem's strides; keep_idx: device int32 [B,H,C], strictly ascending
 * per head (as nacl_select writes it); an entry outside [0, L) gives a row
 * of zeros (no memory outside the head is read).  Two output forms:
 *  - k_out, v_out: device [B,H,C,D] contiguous, overlapping no input;
 *  - in place (k_out == k and v_out == v, K and V disjoint): row c of each
 *    head takes row keep_idx[c] of the same head, in the input's own layout,
 *    for c < C; rows C..L-1 keep their old contents.  This is the cache
 *    update of the generation phase (Section 3, "Generation Phase Eviction"),
 *    where the cache is a fixed buffer of L rows per head.
 * Bit-exact row copies. */
int nacl_compact(const nacl_problem* p, const void* k, const void* v,
                 const int32_t* keep_idx, int32_t C, void* k_out, void* v_out,
                 void* stream);

/* Slot form of the in-place cache update, for a generation-phase cache whose
 * rows need not stay in token order (Section 3, "Generation Phase Eviction":
 * the paper fixes which entries stay, not where they sit).  keep_idx: device
 * int32 [B,H,C], the ascending keep set as nacl_select writes it (read only).
 * In each head of k, v (device [B,H,L,D] with the problem's strides, K and V
 * disjoint) the kept rows below C stay where they are and the kept rows at or
 * past C move, in ascending order, into the slots below C whose rows were
 * not kept (taken in ascending order); nothing else is written, so only the
 * kept rows past C are copied.  slot_idx: device int32 [B,H,C] (overlapping
 * nothing above) receives, for each slot c < C, the old row it holds
 * afterwards.  A keep list that is not an ascending set of rows in [0, L)
 * gives zero rows in the slots whose mover lies outside [C, L).  Bit copies. */
int nacl_compact_slots(const nacl_problem* p, void* k, void* v, const int32_t* keep_idx, int32_t C,
                       int32_t* slot_idx, void* stream);

/* Append of decode steps to the cache (Algorithm 1, generation phase: the
 * new token's key and value join the cache): rows [row0, row0 + m) of every
 * head of k, v (device [B,H,L,D] with the problem's k/v strides) take the m
 * rows of k_new, v_new (device [B,H,m,D] contiguous, overlapping neither
 * cache; K and V caches disjoint).  0 <= row0, row0 + m <= L.  Bit copies. */
int nacl_append(const nacl_problem* p, void* k, void* v, int32_t row0,
                const void* k_new, const void* v_new, int32_t m, void* stream);

/* The whole step for one layer: score, select, compact on one stream
 * (Algorithm 1, encoding phase).  Arguments as above; k_out, v_out may be
 * k, v themselves (in-place compaction).  The health words of nacl_score
 * apply: keep_idx, k_out and v_out are not valid when the call's word is
 * non-zero.
 * Generation-phase eviction (Section 3, "Generation Phase Eviction"; the
 * Generation function of Algorithm 1) is the same call at decode shapes:
 * the cache is a [B,H,L,D] buffer with L = C + m rows per head; after the
 * m decoding steps appended their rows (nacl_append at row0 = C + t), call
 * with the current token as the only proxy (proxy_pos = {L - 1},
 * n_protect = 1), its query as a [B,H,1,D] tensor with q_stride[2] = 0, and
 * k_out = k, v_out = v: the C kept entries move to rows 0..C-1 and the next
 * m steps append after them.  Use a different seed per eviction round so
 * the random draws differ between rounds. */
int nacl_evict(const nacl_problem* p, const void* q, const void* k, const void* v,
               int32_t C, int32_t Cr, int32_t sampling, uint64_t seed, uint32_t layer,
               float* scores, int32_t* keep_idx, void* k_out, void* v_out,
               void* ws, size_t ws_bytes, void* stream);

/* Generation-phase eviction with the slot form of the cache update
 * (Section 3, "Generation Phase Eviction"; the Generation function of
 * Algorithm 1): nacl_score, nacl_select and nacl_compact_slots on one stream,
 * in place in k, v.  Arguments as nacl_evict; keep_idx receives the
 * ascending keep set and slot_idx (device int32 [B,H,C]) the old row each
 * slot below C holds afterwards.  At decode shapes (L = C + m, the current
 * token as the only, protected, proxy) only the kept rows among the m newest
 * move, instead of nearly every kept row as in nacl_evict's in-place form.
 * The health words of nacl_score apply. */
int nacl_evict_slots(const nacl_problem* p, const void* q, void* k, void* v, int32_t C, int32_t Cr,
                     int32_t sampling, uint64_t seed, uint32_t layer, float* scores, int32_t* keep_idx,
                     int32_t* slot_idx, void* ws, size_t ws_bytes, void* stream);

/* The whole step without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc).  Arguments and results as nacl_evict,
 * which it runs; p->proxy_pos_dev is required (no host-to-device copy).  The
 * workspace is a built-in device array of NACL_NOALLOC_WORKSPACE_MAX bytes,
 * one per GPU, held until the process ends; problems needing more
 * (nacl_workspace_bytes) return NACL_ERR_UNSUPPORTED.  Nothing is allocated:
 * no hipMalloc, hipFree or allocating library routine.  Every call on a GPU
 * shares that GPU's array, so calls on one GPU that overlap in time (other
 * streams, other threads) race and must be serialised by the caller.
 * health: optional device uint32[2] that receives the call's health words
 * (this call's, then the sticky one accumulated over every such call on the
 * GPU; see nacl_score), copied on the stream after the eviction. */
#define NACL_NOALLOC_WORKSPACE_MAX (64u << 20)
int nacl_evict_noalloc(const nacl_problem* p, const void* q, const void* k, const void* v,
                       int32_t C, int32_t Cr, int32_t sampling, uint64_t seed, uint32_t layer,
                       float* scores, int32_t* keep_idx, void* k_out, void* v_out,
                       uint32_t* health, void* stream);

/* Causal attention of the prefill with the log-sum-exp of every query row:
 * the FlashAttention-2 forward pass whose log-sum-exp Appendix A.7 reuses,
 * so that the score of a layer runs as the single column reduction of
 * Algorithm 2 (nacl_score with lse = lse_proxy reads K once).  bf16 only
 * (NACL_ERR_UNSUPPORTED otherwise); D = 64 or 128; grouped query heads as in
 * the problem struct: query head hq reads K/V head hq / q_group.
 * q: device [B, H*q_group, L, D] with q_stride; k, v: device [B,H,L,D] with
 * k_stride, v_stride; every row stride at least D.
 * out: device bf16 [B, H*q_group, L, D] contiguous, row i of a query head =
 * sum over j <= i of softmax_j(sm_scale <q_i, k_j>) v_j (fp32 accumulation,
 * the probabilities rounded to bf16 for the value product, the row rounded
 * to bf16 once).
 * lse: device fp32 [B, H*q_group, L], the natural log of
 * sum over j <= i of exp(sm_scale <q_i, k_j>).
 * lse_proxy: optional device fp32 [B, H*q_group, P] receiving lse at the
 * proxy rows, the layout of nacl_score's lse argument; it needs
 * p->proxy_pos_dev.  out, lse and lse_proxy overlap nothing else.  The
 * problem is validated as for every call (its proxy fields included), but
 * the proxies change nothing except which rows lse_proxy receives. */
int nacl_attention(const nacl_problem* p, const void* q, const void* k, const void* v, void* out,
                   float* lse, float* lse_proxy, void* stream);

/* Static text for a status code. */
const char* nacl_status_string(int status);

/* Thread-local text describing the last failed call on this thread ("" if
 * none).  Valid until the next call on the same thread. */
const char* nacl_last_error_detail(void);

/* NACL_VERSION of the built library. */
int nacl_version(void);

#ifdef __cplusplus
}
#endif

#endif /* NACL_H */
