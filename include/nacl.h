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
 *   contiguous in the input dtype and must not overlap any input.
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

#define NACL_VERSION 1
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
 * Health word: once the stream has completed the call, the 32-bit word at
 * byte offset 4 of the workspace is 0.  Bit 0 set means a wave of the
 * two-pass kernel gave up waiting for a head's log-sum-exp after its bounded
 * spin, bit 1 the same for the single-read kernel's wait for a head's row
 * sums (never expected; the scores of that call are then not valid).  The
 * next nacl_score or nacl_evict call on the workspace clears it.
 * Kernel choice (also inside nacl_evict): two passes over K by default.  For
 * bf16, D = 128, exactly 128 proxies and lse == NULL, the environment
 * variable NACL_SCORE_PATH=fused selects a kernel that reads K once (same
 * results within the tolerance, slower on MI355X); NACL_SCORE_PATH=split
 * forces the two-pass kernels.  Both are meant for tests and measurements. */
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
 * the problem's strides; keep_idx: device int32 [B,H,C], each entry in
 * [0, L) (not checked on the device); k_out, v_out: device [B,H,C,D]
 * contiguous.  Bit-exact row copies. */
int nacl_compact(const nacl_problem* p, const void* k, const void* v,
                 const int32_t* keep_idx, int32_t C, void* k_out, void* v_out,
                 void* stream);

/* The whole step for one layer: score, select, compact on one stream
 * (Algorithm 1, encoding phase).  Arguments as above.
 * Generation-phase eviction (Section 3, "Generation Phase Eviction"; the
 * Generation function of Algorithm 1) is the same call at decode shapes:
 * every m steps, with the cache holding C + m entries, pass L = C + m, the
 * current token as the only proxy (proxy_pos = {L - 1}, n_protect = 1), and
 * its query as a [B,H,1,D] tensor with q_stride[2] = 0; k_out, v_out receive
 * the C kept entries (a second buffer: they may not alias k, v).  Use a
 * different seed per eviction round so the random draws differ between
 * rounds. */
int nacl_evict(const nacl_problem* p, const void* q, const void* k, const void* v,
               int32_t C, int32_t Cr, int32_t sampling, uint64_t seed, uint32_t layer,
               float* scores, int32_t* keep_idx, void* k_out, void* v_out,
               void* ws, size_t ws_bytes, void* stream);

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
