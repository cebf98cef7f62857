/*
 * speccascade.h -- C interface of libspeccascade, the verify/defer step of
 * speculative cascades on AMD Instinct MI355X (gfx950).
 *
 * One call performs, for a block of gamma drafted positions in each of B
 * sequences, the verification half of GenSpecSample (Alg. 4) with the
 * cascade target T_delta (eq. (6), Alg. 5) of "Faster Cascades via
 * Speculative Decoding" (Narasimhan et al., arXiv 2405.19261):
 *
 *   q_{t+j} = softmax(z^q_{t+j} / T),  p_{t+j} = softmax(z^p_{t+j} / T)   (j = 0..gamma)
 *   delta_j  by the deferral rule of Table 1 (Chow eq. (2), Diff eq. (5),
 *            OPT eq. (11) with D_TV of Lemma 3)
 *   pi_j     = (1 - delta_j) q_j + delta_j p_j                            (eq. (6))
 *   a_j      = 1(u_j < min(1, pi_j(x_j) / q_j(x_j))), j < gamma; a_gamma = 0
 *   j*       = min{ j : a_j = 0 }
 *   token    ~ norm(max(0, pi_{j*} - q_{j*}))  if j* < gamma,  else ~ pi_gamma
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers are DEVICE pointers on the current HIP device, allocated and
 *   owned by the caller.  The library reads inputs, writes outputs, and keeps
 *   no reference to either after the call returns.
 * - Work is enqueued on `stream` (NULL = the default stream) and is
 *   asynchronous: outputs are valid once the caller synchronises the stream.
 *   No call synchronises the host with the device.
 * - Logit tensors are row-major [B][gamma+1][V] (row stride V elements), in
 *   float32 or bfloat16.  Row gamma of the drafter tensor is the drafter's
 *   distribution at the bonus position t+gamma, which the extra-token target
 *   pi_{t+gamma} of Alg. 4 needs.
 * - Every argument is checked before any HIP call; a failed check returns
 *   its status and enqueues nothing.  spc_last_error() then describes it.
 * - Preconditions that are NOT checked: logits are finite or -inf, with at
 *   least one finite entry per row; uniforms lie in [0, 1).
 * - Defined behaviour: a draft token outside [0, V) rejects its position
 *   (no out-of-bounds read).  out_defer_mask is filled for all gamma+1
 *   positions, including those past j*.  Sequence b emits
 *   draft_tokens[b][0 .. accept_len[b]-1] followed by next_token[b].
 * - The internal workspace (used when no caller workspace is passed) is one
 *   buffer per device: calls that use it must not overlap in time on one
 *   device (issue them on one stream).  Calls with distinct caller
 *   workspaces may run concurrently.
 */
#ifndef SPECCASCADE_H
#define SPECCASCADE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of the logit tensors.  Entry points take it as an int32_t
 * `dtype` holding one of these values (any other value is rejected), so that
 * an out-of-range value never reaches the library as an enum. */
typedef enum { SPC_F32 = 0, SPC_BF16 = 1 } spc_dtype;

/* Deferral rules of Table 1, two constant rules, and the token-specific rules
 * of Section 4.4.  A token rule r(v) marks token v as not acceptable and uses
 * the target of Alg. 6 (TokenSpecCascade) in place of T_delta:
 *   pi(v) = q(v) (1 - r(v)) + p(v) eta,   eta = sum_v r(v) q(v).
 * For a token rule, out_defer_mask[b][j] reports r(x_j), the rule's verdict
 * on the draft token (0 at the bonus position j = gamma), and row statistic
 * column 6 holds eta.  At temperature 0 r is read at the drafter's argmax
 * with temperature-1 probabilities; the one-hot target then sits at argmax p
 * when r = 1 and at argmax q otherwise.
 *
 * The other targets of Tables 1 and 3: LOSSY is lossy speculative decoding
 * with beta = 1, whose target (Lemma 2) needs no deferral decision (the mask
 * reports 0): a draft is kept with probability min(1, p(x) / ((1 - alpha)
 * q(x))), a rejection draws from max(0, p - q), and the extra token comes
 * from p (the target is not a normalised distribution).  BILD and the
 * log-loss rules defer with the mixture target T_delta of eq. (6); their
 * statistic (D, H(q), or H(q) - H(p), in nats) is row statistic column 7.
 * At temperature 0 the log-loss rules read the entropies of the
 * temperature-1 softmax, BILD reads D = lse_p - z_p(argmax q) (temperature
 * 1), and LOSSY's one-hot target sits at argmax p. */
typedef enum {
  SPC_RULE_CHOW = 0,     /* delta = 1(max_v q(v) < 1 - alpha)                 eq. (2)  */
  SPC_RULE_DIFF = 1,     /* delta = 1(max_v q(v) < max_v p(v) - alpha)        eq. (5)  */
  SPC_RULE_OPT = 2,      /* delta = 1(max_v q(v) < max_v p(v) - alpha D_TV)   eq. (11) */
  SPC_RULE_ALWAYS = 3,   /* delta = 1: standard speculative decoding (Alg. 1)          */
  SPC_RULE_NEVER = 4,    /* delta = 0: the drafter's own distribution                  */
  SPC_RULE_TOKEN_V1 = 5, /* r(v) = 1(q(v) < max_v p(v) - alpha)          TokenV1, 4.4  */
  SPC_RULE_TOKEN_V2 = 6, /* r(v) = 1(p(v) < max_v p(v) - alpha)          TokenV2, 4.4  */
  SPC_RULE_TOKEN_V3 = 7, /* r(v) = 1(p(v) < max_v p(v) (1 - alpha))      TokenV3, 4.4  */
  SPC_RULE_LOSSY = 8,    /* lossy speculative decoding with beta = 1 (Lemma 2):
                            pi = max{min{q, p / (1 - alpha)}, p}; alpha < 1            */
  SPC_RULE_BILD = 9,     /* BiLD*: delta = 1(D(q, p) > alpha), D = -sum_v q(v) log p(v)
                            (temperature 0: -log p(argmax q))          Table 1, Sec. 6 */
  SPC_RULE_CHOWLOG = 10, /* delta = 1(H(q) > alpha)                     Table 3, App. B */
  SPC_RULE_DIFFLOG = 11, /* delta = 1(H(p) < H(q) - alpha)              Table 3, App. D */
  SPC_RULE_OPTLOG = 12   /* delta = 1(H(p) < H(q) - alpha D_TV(p, q))   Table 3, App. D */
} spc_rule;

typedef enum {
  SPC_OK = 0,
  SPC_E_NULL = -1,      /* a required pointer is NULL                                 */
  SPC_E_SHAPE = -2,     /* B < 1, gamma < 1, gamma > SPC_MAX_GAMMA or V < 2 (any B:
                           large batches run as several launches)                     */
  SPC_E_RULE = -3,      /* a rule id outside spc_rule                                 */
  SPC_E_PARAM = -4,     /* alpha not finite, temperature not > 0 and finite,
                           or an unknown dtype                                        */
  SPC_E_ALIGN = -5,     /* a logit base pointer not 16-byte aligned                   */
  SPC_E_WORKSPACE = -6, /* caller workspace too small or misaligned                   */
  SPC_E_HIP = -7        /* a HIP call failed; spc_last_error() holds its message      */
} spc_status;

/* Largest block size: the first-rejection search runs in one 64-lane wavefront. */
#define SPC_MAX_GAMMA 63

/*
 * spc_verify -- one verify step at temperature `temperature` > 0 with the same
 * rule, alpha and temperature for all B sequences.  A temperature below
 * 2^-107 (any float32 down to the smallest subnormal) is computed as 2^-107:
 * z / T stays finite for logits up to ~10^6 and the softmax is then already
 * its T -> 0 limit over logits that differ by more than ~10^-30.
 *
 *   q_logits, p_logits  [B][gamma+1][V] drafter / verifier logits, `dtype`
 *   draft_tokens        [B][gamma] int32: x_t .. x_{t+gamma-1}
 *   uniforms            [B][gamma+1] float32 in [0,1): u[b][j], j < gamma, is
 *                       the draw of a_j (Alg. 4); u[b][gamma] drives the one
 *                       replacement or extra-token sample (inverse CDF in
 *                       vocabulary order: the smallest k whose cumulative mass
 *                       exceeds u times the total)
 *   rule, alpha         deferral rule (spc_rule) and its parameter
 *   out_accept_len      [B] int32: j* in [0, gamma]
 *   out_next_token      [B] int32: the token emitted at position t + j*
 *   out_defer_mask      [B][gamma+1] uint8: delta_j at every position
 */
spc_status spc_verify(const void* q_logits, const void* p_logits, int32_t dtype,
                      const int32_t* draft_tokens, const float* uniforms, int32_t B,
                      int32_t gamma, int32_t V, int32_t rule, float alpha, float temperature,
                      int32_t* out_accept_len, int32_t* out_next_token,
                      uint8_t* out_defer_mask, hipStream_t stream);

/*
 * spc_greedy_verify -- the temperature-0 step (Lemma 6, greedy case).
 * q~ and p~ are one-hot at the argmax of the raw logits (lowest index on a
 * tie); the rule's max-probabilities come from the temperature-1 softmax and
 * D_TV(p~, q~) = 1(argmax q != argmax p).  A draft is kept exactly when it
 * equals the argmax of pi~_j = (1 - delta_j) q~_j + delta_j p~_j, and the
 * emitted token is that argmax at position j*.  No uniforms are used; the
 * result is a deterministic function of the inputs.
 */
spc_status spc_greedy_verify(const void* q_logits, const void* p_logits, int32_t dtype,
                             const int32_t* draft_tokens, int32_t B, int32_t gamma, int32_t V,
                             int32_t rule, float alpha, int32_t* out_accept_len,
                             int32_t* out_next_token, uint8_t* out_defer_mask,
                             hipStream_t stream);

/*
 * Extended arguments.  Every field may be NULL / 0.
 *   rule_per_seq, alpha_per_seq, temp_per_seq  [B] device arrays overriding
 *       the scalar rule / alpha / temperature per sequence.  A per-sequence
 *       temperature of 0 selects the greedy step for that sequence.  Values
 *       are checked by the kernels: an invalid one makes that sequence emit
 *       accept_len = -1 and next_token = -1.
 *   out_row_stats  [B][gamma+1][8] float32: {m_q, lse_q, maxprob_q, m_p,
 *       lse_p, maxprob_p, tv, s} with m = max_v z_v / T and lse = log sum_v
 *       exp(z_v / T); greedy rows hold the temperature-1 values and the
 *       one-hot TV (for a token rule, r at argmax q).  tv is computed for OPT
 *       and OPTLOG rows only (0 elsewhere); token-rule rows hold eta there.
 *       s is the statistic of BILD and the log-loss rules (0 elsewhere).
 *   out_argmax     [B][gamma+1][2] int32: argmax of raw q and p logits
 *       (filled for greedy rows; -1 elsewhere).
 *   out_sample_norm [B] float32: the total mass W of the distribution
 *       sampled at j* (for a replacement, sum_v max(0, p - q) = D_TV).
 *   workspace, workspace_bytes  caller-owned device buffer of at least
 *       spc_workspace_bytes(B, gamma, V, dtype) bytes, 256-byte aligned,
 *       whose first spc_workspace_zero_bytes(B, gamma, V, dtype) bytes are
 *       zero before its first use (the kernels leave them zero again).
 *       NULL selects the internal per-device workspace, allocated on first
 *       use and grown as needed.
 *   rules_present  with rule_per_seq: a bitmask (bit i = rule i) of the
 *       rules the array may hold, 0 = any.  It lets the library skip the
 *       passes no sequence needs (the second pass of OPT, OPTLOG and the
 *       token rules; the first moments of BiLD* and the log-loss rules).  A
 *       sequence whose rule lies outside a nonzero mask is invalid (it
 *       reports accept_len = -1 and next_token = -1).
 *   ev_tiles_begin, ev_tiles_end  for profiling: events (owned by the
 *       caller) recorded on `stream` right before and right after the
 *       statistics kernel of the call's first launch, so that their elapsed
 *       time is that kernel's duration; NULL records nothing.  A record
 *       that fails makes the call return SPC_E_HIP before any kernel of
 *       that launch.
 */
typedef struct {
  const int32_t* rule_per_seq;
  const float* alpha_per_seq;
  const float* temp_per_seq;
  float* out_row_stats;
  int32_t* out_argmax;
  float* out_sample_norm;
  void* workspace;
  size_t workspace_bytes;
  uint32_t rules_present;
  hipEvent_t ev_tiles_begin;
  hipEvent_t ev_tiles_end;
} spc_verify_ex_args;

/* spc_verify with extended arguments; `ex` may be NULL.  `temperature`
 * applies where temp_per_seq is NULL.  There it must be > 0, or exactly 0 for
 * the batch-wide greedy step of spc_greedy_verify (uniforms may then be
 * NULL), which this entry point then runs with its optional outputs. */
spc_status spc_verify_ex(const void* q_logits, const void* p_logits, int32_t dtype,
                         const int32_t* draft_tokens, const float* uniforms, int32_t B,
                         int32_t gamma, int32_t V, int32_t rule, float alpha, float temperature,
                         int32_t* out_accept_len, int32_t* out_next_token,
                         uint8_t* out_defer_mask, const spc_verify_ex_args* ex,
                         hipStream_t stream);

/*
 * spc_verify_noalloc -- spc_verify_ex for callers that cannot allocate
 * device memory: code being recorded into a HIP graph, serving loops that
 * must not call hipMalloc, harnesses that forbid allocation.  It computes
 * exactly what spc_verify_ex computes (same kernels), but its workspace is a
 * static device array of spc_noalloc_scratch_bytes() bytes (32 MiB) that
 * every device running it holds until the process ends; it calls no
 * hipMalloc, hipFree or allocating library routine.
 *   ex            as for spc_verify_ex, except that ex->workspace must be
 *                 NULL (SPC_E_WORKSPACE otherwise)
 * A batch whose layout exceeds the scratch is run in launches of as many
 * whole sequences as fit; a shape of which not even one sequence fits
 * (gamma and V large: the layout grows with (gamma + 1) * V) returns
 * SPC_E_WORKSPACE.  The first call on a device clears the array's counter
 * region with a fill kernel on `stream`; every call leaves it cleared.
 * All calls on one device share the array: calls that overlap on one device
 * (other streams, other host threads) race and must be serialised by the
 * caller.  Other errors as spc_verify_ex.
 */
spc_status spc_verify_noalloc(const void* q_logits, const void* p_logits, int32_t dtype,
                              const int32_t* draft_tokens, const float* uniforms, int32_t B,
                              int32_t gamma, int32_t V, int32_t rule, float alpha,
                              float temperature, int32_t* out_accept_len,
                              int32_t* out_next_token, uint8_t* out_defer_mask,
                              const spc_verify_ex_args* ex, hipStream_t stream);

/* Size in bytes of spc_verify_noalloc's static scratch. */
size_t spc_noalloc_scratch_bytes(void);

/*
 * spc_draft_sample -- the drafter's sampling step of GenSpecSample (Alg. 4):
 * x_{t+j} ~ q_{t+j} = softmax(z / T) for one position of each of B sequences.
 *
 *   logits        [B][V] drafter logits, `dtype`, rows contiguous
 *   temperature   T for every sequence (T = 0: the argmax of the raw logits,
 *                 lowest index on a tie), unless temp_per_seq is given
 *   temp_per_seq  [B] float32 per-sequence temperatures, or NULL; a row
 *                 whose temperature is negative or not finite gets
 *                 out_token = -1
 *   uniforms      [B] float32 in [0,1): the token is the smallest k whose
 *                 cumulative mass (vocabulary order) exceeds u times the
 *                 total; may be NULL only for the batch-wide argmax
                 (temperature 0 and temp_per_seq NULL): with temp_per_seq
                 it is required even if every entry is 0
 *   out_token     [B] int32
 * Uses the statistics tiles and the tile-mass draw of spc_verify (one pass
 * over the logits) and the internal workspace.  Errors as spc_verify; a
 * negative or non-finite temperature is SPC_E_PARAM, an invalid per-sequence
 * one gives out_token = -1.
 */
spc_status spc_draft_sample(const void* logits, int32_t dtype, int32_t B, int32_t V,
                            float temperature, const float* temp_per_seq,
                            const float* uniforms, int32_t* out_token, hipStream_t stream);

/*
 * spc_draft_sample_ws -- spc_draft_sample with a caller workspace of
 * workspace_bytes >= spc_draft_workspace_bytes(B, V, dtype) bytes, 256-byte
 * aligned, whose first spc_workspace_zero_bytes(1, 1, 2, dtype) bytes are zero
 * before its first use (the kernels leave them zero).  NULL selects the
 * internal workspace.  A too-small or misaligned workspace is SPC_E_WORKSPACE.
 * Calls with distinct workspaces may run concurrently.
 */
spc_status spc_draft_sample_ws(const void* logits, int32_t dtype, int32_t B, int32_t V,
                               float temperature, const float* temp_per_seq,
                               const float* uniforms, int32_t* out_token, void* workspace,
                               size_t workspace_bytes, hipStream_t stream);

/* Bytes of device workspace one spc_draft_sample_ws call of this shape needs. */
size_t spc_draft_workspace_bytes(int32_t B, int32_t V, int32_t dtype);

/* Bytes of device workspace one call of this shape needs. */
size_t spc_workspace_bytes(int32_t B, int32_t gamma, int32_t V, int32_t dtype);

/* Leading bytes of a workspace that must be zero before its first use
 * (completion counters at fixed offsets: the same for every shape, so one
 * zeroed workspace serves calls of any shape it is large enough for). */
size_t spc_workspace_zero_bytes(int32_t B, int32_t gamma, int32_t V, int32_t dtype);

/* Thread-local description of the last non-OK status ("" if none). */
const char* spc_last_error(void);

/* Frees the internal workspace of every device.  Not safe while a call that
 * uses it may still be running: synchronise first. */
void spc_release(void);

/* Library version string. */
const char* spc_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPECCASCADE_H */
