/*
 * spc_oracle.h -- plain fp64 CPU oracle of one speculative-cascade verify step.
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists so that tests, the smoke
 * check and the benchmark's CPU-baseline leg can check the GPU library
 * against an independent, slow, obviously correct implementation of the
 * paper "Faster Cascades via Speculative Decoding" (Narasimhan et al.,
 * arXiv 2405.19261).  No product code may link or call it, and it shares no
 * code, header or constant with the GPU library.
 *
 * Everything is computed in IEEE double precision with sequential loops in
 * vocabulary-index order.  Inputs of type float32 or bfloat16 widen to double
 * exactly, so the oracle sees exactly the values the GPU reads.
 *
 * Layouts (row-major, host memory, caller-owned):
 *   logits   [B][gamma+1][V]  dtype ORC_F32, ORC_BF16 (raw uint16 bits) or ORC_F64
 *   draft    [B][gamma]       int32
 *   uniforms [B][gamma+1]     float32 in [0,1): u[b][j<gamma] drive the
 *                             accept draws, u[b][gamma] the one replacement or
 *                             bonus sample
 *   rule/alpha/temperature    one value per sequence, [B]
 */
#ifndef SPC_ORACLE_H
#define SPC_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_F64 = 2 };

/* Largest block size gamma the oracle accepts. */
#define ORC_MAX_GAMMA 64

/* Deferral rules of Table 1 (Section 4.2 and eq. (2), (5), (11)), plus the two
 * constant rules: ALWAYS (delta = 1: standard speculative decoding, Alg. 1)
 * and NEVER (delta = 0: the drafter alone); the token-specific rules of
 * Section 4.4; and the other targets of Tables 1 and 3:
 *   LOSSY    lossy speculative decoding, pi = max{min{q, p/(1-alpha)}, p/beta}
 *            with beta = 1 (Lemma 2), alpha < 1
 *   BILD     BiLD*: delta = 1(D(q,p) > alpha), D the cross-entropy -sum q log p
 *            (temperature 0: -log p(argmax q))
 *   CHOWLOG  delta = 1(H(q) > alpha)
 *   DIFFLOG  delta = 1(H(p) < H(q) - alpha)
 *   OPTLOG   delta = 1(H(p) < H(q) - alpha D_TV(p,q))
 * with the mixture target T_delta of eq. (6) for BILD and the log rules. */
enum { ORC_CHOW = 0, ORC_DIFF = 1, ORC_OPT = 2, ORC_ALWAYS = 3, ORC_NEVER = 4,
       ORC_TOKEN_V1 = 5, ORC_TOKEN_V2 = 6, ORC_TOKEN_V3 = 7, ORC_LOSSY = 8, ORC_BILD = 9,
       ORC_CHOWLOG = 10, ORC_DIFFLOG = 11, ORC_OPTLOG = 12 };

/* Per-sequence flags reported by orc_verify / orc_greedy_verify. */
enum {
  ORC_FLAG_DRAFT_OUT_OF_RANGE = 1, /* a draft token outside [0,V) was rejected */
  ORC_FLAG_EMPTY_RESIDUAL = 2      /* rejection with zero residual mass: sampled p instead */
};

/* Statistics of one tempered softmax row (Section 2 notation; temperature
 * read as q = softmax(z / T)). */
typedef struct {
  double m;       /* max_v z_v / T                                */
  double lse;     /* log sum_v exp(z_v / T)                       */
  double maxprob; /* max_v softmax(z/T)_v                         */
  int32_t argmax; /* smallest v with z_v == max z (raw logits)    */
} orc_row_stats;

/* softmax(z / T) of one row of V logits; prob may be NULL.  T > 0. */
void orc_softmax_row(const void* z, int dtype, int64_t V, double T, double* prob,
                     orc_row_stats* st);

/* D_TV(p, q) = sum_v max(0, p_v - q_v)  (Lemma 3). */
double orc_tv(const double* p, const double* q, int64_t V);

/* Entropy H(q) = -sum_v q(v) log q(v) (natural log, 0 log 0 = 0) of the row
 * softmax(z / T), with log q(v) = z_v / T - lse taken from the logits. */
double orc_entropy_row(const void* z, int dtype, int64_t V, double T, const orc_row_stats* st);

/* Cross-entropy D(q, p) = -sum_v q(v) log p(v) of BiLD*'s temperature-sampling
 * discrepancy; +infinity when some v has q(v) > 0 (a finite drafter logit)
 * and p(v) = 0 (a verifier logit of -infinity). */
double orc_cross_entropy_row(const void* zq, const void* zp, int dtype, int64_t V, double T,
                             const orc_row_stats* sq, const orc_row_stats* sp);

/* delta of a log-loss rule (BILD, CHOWLOG, DIFFLOG, OPTLOG) from its statistic
 * s (D for BILD, H(q) for CHOWLOG, H(q) - H(p) for DIFFLOG and OPTLOG) and
 * the threshold alpha (alpha D_TV for OPTLOG): delta = 1(s > threshold),
 * strict.  *margin = |s - threshold| / max(1, mag, |threshold|), mag the size
 * of the entropies s is made of (s itself, max(H(q), H(p)) for a
 * difference): they are sums of terms up to log V in size, rounded relative
 * to that size. */
int orc_log_defer(double s, double threshold, double mag, double* margin);

/* Lossy target of Lemma 2 with beta = 1: pi(v) = max{min{q(v), p(v)/(1-alpha)},
 * p(v)} (not normalised).  alpha < 1. */
void orc_lossy_target(double alpha, const double* q, const double* p, int64_t V, double* pi);

/* delta(q, p) of Table 1 for one position; *margin = |lhs - rhs| of the
 * defining inequality (infinity for ALWAYS / NEVER). Returns 0 or 1, or -1 for
 * an unknown rule. */
int orc_defer(int rule, double alpha, double maxq, double maxp, double tv, double* margin);

/* pi = (1 - delta) q + delta p   (eq. (6)). */
void orc_target(int delta, const double* q, const double* p, int64_t V, double* pi);

/* Accept draw of Alg. 4: a = 1(u < min(1, pi_x / q_x)); a token with
 * q_x <= pi_x is always kept (Section 4.1).  *margin = |u - min(1, ratio)|. */
int orc_accept(double pi_x, double q_x, double u, double* margin);

/* Unnormalised residual w = max(0, pi - q) (Alg. 4); returns sum_v w_v. */
double orc_residual(const double* pi, const double* q, int64_t V, double* w);

/* Token-specific deferral (Section 4.4, the TokenV1/V2/V3 plug-in rules):
 * r(v) = 1 marks token v as not acceptable.
 *   V1: q(v) < max p - alpha;  V2: p(v) < max p - alpha;
 *   V3: p(v) < max p (1 - alpha).
 * margin = |lhs - rhs| / scale with scale = max(|lhs|, |rhs|), and for V1
 * and V2 also max p: there the threshold max p - alpha inherits the rounding
 * of max p itself, which is relative to max p, not to the (possibly much
 * smaller) difference.  Under V2 and V3 a token with p(v) = max p gets
 * 1(alpha < 0), exact, with an infinite margin. */
int orc_token_r(int rule, double alpha, double qv, double pv, double maxp, double* margin);

/* Target of Alg. 6 (TokenSpecCascade): pi(v) = q(v) (1 - r(v)) + p(v) eta with
 * eta = sum_v r(v) q(v) (vocabulary order).  Returns eta; *rmargin is the
 * smallest r-margin over the row (any r(v) that flips moves eta). */
double orc_token_target(int rule, double alpha, const double* q, const double* p, int64_t V,
                        double maxp, double* pi, double* rmargin);

/* Inverse-CDF draw from norm(w): the smallest k with C_k / W > u, where
 * C_k = sum_{v<=k} w_v in index order and W = C_{V-1}.  Returns -1 when W is
 * not positive.  *margin = min(C_k/W - u, u - C_{k-1}/W). */
int32_t orc_sample(const double* w, int64_t V, double u, double* margin);

/* One GenSpecSample (Alg. 4) with the target T_delta (Alg. 5) for each of B
 * sequences.  rule/alpha/temperature are per sequence.  Outputs:
 *   accept_len [B]            j* in [0, gamma]
 *   next_token [B]            the token emitted at position j*
 *   defer      [B][gamma+1]   delta at every position
 * Optional outputs (may be NULL):
 *   row_stats     [B][gamma+1][8] = {m_q, lse_q, maxprob_q, m_p, lse_p, maxprob_p, c6, c7}
 *                 c6 = D_TV (OPT, OPTLOG), eta (token rules), else 0;
 *                 c7 = the log-loss statistic s of orc_log_defer, else 0
 *   defer_margin  [B][gamma+1]
 *   accept_margin [B][gamma]      (infinity where the draw is exact)
 *   sample_margin [B]
 *   sample_norm   [B]             W = mass of the distribution sampled at j*
 *   flags         [B]             ORC_FLAG_*
 * Returns 0, or -1 on an argument error.  Sequences run in parallel (OpenMP). */
int orc_verify(const void* q_logits, const void* p_logits, int dtype, const int32_t* draft,
               const float* uniforms, int32_t B, int32_t gamma, int64_t V,
               const int32_t* rule, const float* alpha, const float* temperature,
               int32_t* accept_len, int32_t* next_token, uint8_t* defer, double* row_stats,
               double* defer_margin, double* accept_margin, double* sample_margin,
               double* sample_norm, int32_t* flags);

/* The greedy (temperature 0) step of Lemma 6: one-hot q~ and p~ at the
 * argmaxes of the raw logits, max-probabilities from the temperature-1
 * softmax, D_TV(p~, q~) = 1(argmax q != argmax p).  No uniforms.  row_stats
 * holds the temperature-1 statistics and the one-hot TV.  The log-loss rules
 * read entropies of the temperature-1 softmax; BILD reads D = -log p(argmax q)
 * (temperature 1).  LOSSY's one-hot target is at argmax p, as for ALWAYS. */
int orc_greedy_verify(const void* q_logits, const void* p_logits, int dtype,
                      const int32_t* draft, int32_t B, int32_t gamma, int64_t V,
                      const int32_t* rule, const float* alpha, int32_t* accept_len,
                      int32_t* next_token, uint8_t* defer, double* row_stats,
                      int32_t* argmax_qp, double* defer_margin, int32_t* flags);

/* The drafter's sampling step of Alg. 4, x_{t+j} ~ q_{t+j}: for each of B
 * rows of V logits, the inverse-CDF draw (orc_sample) from softmax(z / T_b)
 * with uniform u[b], or at T_b = 0 the argmax of the raw logits (smallest
 * index).  uniforms may be NULL when every T_b is 0.  tokens [B]; margin [B]
 * (may be NULL) is orc_sample's margin (infinity for an argmax).  Returns 0,
 * or -1 on an argument error. */
int orc_draft_sample(const void* logits, int dtype, int32_t B, int64_t V,
                     const float* temperature, const float* uniforms, int32_t* tokens,
                     double* margin);

/* Number of OpenMP threads orc_verify uses. */
int orc_num_threads(void);
/* Sets that number (n > 0); timing only, the results do not depend on it. */
void orc_set_num_threads(int n);

#ifdef __cplusplus
}
#endif

#endif
