/*
 * spc_oracle.c -- fp64 CPU oracle of the speculative-cascade verify step.
 *
 * TEST INFRASTRUCTURE ONLY (tests, smoke check, CPU-baseline timing).  It
 * shares no code with the GPU library.  Each function restates one step of
 * "Faster Cascades via Speculative Decoding" (Narasimhan et al.):
 *
 *   softmax rows      Section 2 notation; temperature read as softmax(z/T)
 *   D_TV              Lemma 3 (Section 4.3)
 *   deferral delta    Table 1; eq. (2) Chow, eq. (5) Diff, eq. (11) OPT
 *   target pi         eq. (6), T_delta of Alg. 5
 *   token rules       Section 4.4 (TokenV1/V2/V3), target of Alg. 6
 *   lossy target      Section 2 (lossy speculative decoding), Lemma 2, beta = 1
 *   BiLD*             Table 1 (D > alpha); D as the cross-entropy of the
 *                     experimental setup (temperature 0: -log p(argmax q))
 *   log-loss rules    Table 3, eq. of ChowLog (App. B), DiffLog and OPTLog
 *                     (App. D), with the entropy H(q) = -sum q log q
 *   accept / j* / residual / sample    Alg. 4 (GenSpecSample)
 *   greedy step       Lemma 6 (Appendix, greedy special case)
 *
 * Readings where the paper is silent (all documented alongside the build):
 *   - ties: the strict inequalities are taken as printed; delta ties do not
 *     defer; the inverse CDF takes the smallest k with C_k > u (zero-mass
 *     tokens are never drawn); argmax ties go to the lowest index.
 *   - the bonus target pi_{t+gamma} needs a drafter row at position gamma, so
 *     the drafter supplies gamma+1 rows.
 *   - one uniform per draft position and one more for the single sample.
 *   - token rules report delta_j = r(x_j), the rule's verdict on the draft
 *     token (0 at the bonus position); at temperature 0 r is read at the
 *     drafter's argmax with temperature-1 probabilities, so the one-hot
 *     target sits at argmax p when r = 1 and at argmax q otherwise.
 *   - the lossy target is not normalised; when every draft is kept the extra
 *     token comes from p_{t+gamma}, as in the lossy procedure that Lemma 2
 *     identifies Alg. 4 with.  alpha >= 1 is rejected.  The lossy rule has no
 *     deferral decision: delta is reported as 0.
 *   - BiLD's discrepancy at temperature 0 is -log p(argmax q) (a
 *     non-negative discrepancy), as printed in the experimental setup.
 *   - the log-loss rules at temperature 0 read the entropies of the
 *     temperature-1 softmax, as the Table 1 rules read its max-probabilities.
 */
#include "spc_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double logit_at(const void* base, int dtype, int64_t i) {
  if (dtype == ORC_F32) return (double)((const float*)base)[i];
  if (dtype == ORC_BF16) {
    /* a bfloat16 value is the top half of the float32 with the same bits */
    uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
  }
  return ((const double*)base)[i];
}

static size_t dtype_size(int dtype) {
  return dtype == ORC_F32 ? 4 : dtype == ORC_BF16 ? 2 : 8;
}

static const void* row_ptr(const void* base, int dtype, int64_t row, int64_t V) {
  return (const char*)base + (size_t)row * (size_t)V * dtype_size(dtype);
}

void orc_softmax_row(const void* z, int dtype, int64_t V, double T, double* prob,
                     orc_row_stats* st) {
  /* s_v = z_v / T; m = max_v s_v; Z = sum_v exp(s_v - m); lse = m + log Z. */
  double zmax = -INFINITY;
  int32_t amax = 0;
  for (int64_t v = 0; v < V; ++v) {
    double zv = logit_at(z, dtype, v);
    if (zv > zmax) { /* strict: the lowest index wins a tie */
      zmax = zv;
      amax = (int32_t)v;
    }
  }
  double m = zmax / T;
  double Z = 0.0;
  for (int64_t v = 0; v < V; ++v) Z += exp(logit_at(z, dtype, v) / T - m);
  double lse = m + log(Z);
  double maxprob = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    double pv = exp(logit_at(z, dtype, v) / T - lse);
    if (prob) prob[v] = pv;
    if (pv > maxprob) maxprob = pv;
  }
  st->m = m;
  st->lse = lse;
  st->maxprob = maxprob;
  st->argmax = amax;
}

double orc_tv(const double* p, const double* q, int64_t V) {
  double tv = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    double d = p[v] - q[v];
    if (d > 0.0) tv += d;
  }
  return tv;
}

static double logprob_at(const void* z, int dtype, int64_t v, double T, double lse) {
  return logit_at(z, dtype, v) / T - lse;
}

double orc_entropy_row(const void* z, int dtype, int64_t V, double T, const orc_row_stats* st) {
  double h = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    double lq = logprob_at(z, dtype, v, T, st->lse);
    double qv = exp(lq);
    if (qv > 0.0) h -= qv * lq; /* 0 log 0 = 0 */
  }
  return h;
}

double orc_cross_entropy_row(const void* zq, const void* zp, int dtype, int64_t V, double T,
                             const orc_row_stats* sq, const orc_row_stats* sp) {
  double d = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    if (logit_at(zq, dtype, v) == -INFINITY) continue; /* q(v) = 0 */
    double lp = logprob_at(zp, dtype, v, T, sp->lse);
    if (lp == -INFINITY) return INFINITY; /* q(v) > 0 = p(v) */
    d -= exp(logprob_at(zq, dtype, v, T, sq->lse)) * lp;
  }
  return d;
}

int orc_log_defer(double s, double threshold, double mag, double* margin) {
  double scale = 1.0;
  if (fabs(mag) > scale) scale = fabs(mag);
  if (fabs(threshold) > scale) scale = fabs(threshold);
  *margin = isinf(s) ? INFINITY : fabs(s - threshold) / scale;
  return s > threshold ? 1 : 0;
}

void orc_lossy_target(double alpha, const double* q, const double* p, int64_t V, double* pi) {
  const double beta = 1.0;
  for (int64_t v = 0; v < V; ++v) {
    double a = p[v] / (1.0 - alpha);
    double lo = q[v] < a ? q[v] : a;
    double b = p[v] / beta;
    pi[v] = lo > b ? lo : b;
  }
}

int orc_defer(int rule, double alpha, double maxq, double maxp, double tv, double* margin) {
  double lhs = maxq, rhs;
  switch (rule) {
    case ORC_CHOW: rhs = 1.0 - alpha; break;          /* eq. (2)  */
    case ORC_DIFF: rhs = maxp - alpha; break;         /* eq. (5)  */
    case ORC_OPT: rhs = maxp - alpha * tv; break;     /* eq. (11) */
    case ORC_ALWAYS: *margin = INFINITY; return 1;    /* T(q,p) = p, Alg. 1 */
    case ORC_NEVER: *margin = INFINITY; return 0;
    default: *margin = NAN; return -1;
  }
  *margin = fabs(lhs - rhs);
  return lhs < rhs ? 1 : 0;
}

void orc_target(int delta, const double* q, const double* p, int64_t V, double* pi) {
  double d = (double)delta;
  for (int64_t v = 0; v < V; ++v) pi[v] = (1.0 - d) * q[v] + d * p[v];
}

int orc_accept(double pi_x, double q_x, double u, double* margin) {
  if (q_x <= pi_x) { /* pi_x / q_x >= 1: min(1, .) = 1 and u < 1 always holds */
    *margin = 1.0 - u;
    return 1;
  }
  double r = pi_x / q_x; /* < 1 here, and q_x > 0 */
  *margin = fabs(u - r);
  return u < r ? 1 : 0;
}

int orc_token_r(int rule, double alpha, double qv, double pv, double maxp, double* margin) {
  double lhs, rhs;
  switch (rule) {
    case ORC_TOKEN_V1: lhs = qv; rhs = maxp - alpha; break;
    case ORC_TOKEN_V2: lhs = pv; rhs = maxp - alpha; break;
    case ORC_TOKEN_V3: lhs = pv; rhs = maxp * (1.0 - alpha); break;
    default: *margin = NAN; return -1;
  }
  if (rule != ORC_TOKEN_V1 && pv == maxp) {
    /* a token attaining max p meets max p (1 - alpha) or max p - alpha:
     * the verdict is 1(alpha < 0) exactly, with nothing rounded */
    *margin = INFINITY;
    return alpha < 0.0 ? 1 : 0;
  }
  double scale = fabs(lhs) > fabs(rhs) ? fabs(lhs) : fabs(rhs);
  if (rule != ORC_TOKEN_V3 && maxp > scale) scale = maxp; /* max p - alpha */
  *margin = scale > 0.0 ? fabs(lhs - rhs) / scale : 0.0;
  return lhs < rhs ? 1 : 0;
}

double orc_token_target(int rule, double alpha, const double* q, const double* p, int64_t V,
                        double maxp, double* pi, double* rmargin) {
  double eta = 0.0, mmin = INFINITY;
  for (int64_t v = 0; v < V; ++v) {
    double mg;
    if (orc_token_r(rule, alpha, q[v], p[v], maxp, &mg)) eta += q[v];
    if (mg < mmin) mmin = mg;
  }
  for (int64_t v = 0; v < V; ++v) {
    double mg;
    int r = orc_token_r(rule, alpha, q[v], p[v], maxp, &mg);
    pi[v] = q[v] * (1.0 - r) + p[v] * eta;
  }
  *rmargin = mmin;
  return eta;
}

double orc_residual(const double* pi, const double* q, int64_t V, double* w) {
  double W = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    double d = pi[v] - q[v];
    w[v] = d > 0.0 ? d : 0.0;
    W += w[v];
  }
  return W;
}

int32_t orc_sample(const double* w, int64_t V, double u, double* margin) {
  double W = 0.0;
  for (int64_t v = 0; v < V; ++v) W += w[v];
  if (!(W > 0.0)) {
    *margin = NAN;
    return -1;
  }
  double prev = 0.0, C = 0.0;
  int32_t last_pos = -1;
  for (int64_t v = 0; v < V; ++v) {
    if (w[v] > 0.0) last_pos = (int32_t)v;
    C += w[v];
    double c = C / W;
    if (c > u) {
      double a = c - u, b = u - prev;
      *margin = a < b ? a : b;
      return (int32_t)v;
    }
    prev = c;
  }
  /* rounding left the last cumulative value at or below u: take the last
   * token that has mass */
  *margin = 0.0;
  return last_pos;
}

/* ---------------------------------------------------------------------- */

int orc_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void orc_set_num_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

static int rule_ok(int r, float alpha) {
  if (r == ORC_LOSSY) return alpha < 1.0f;
  return r >= ORC_CHOW && r <= ORC_OPTLOG;
}
static int is_token(int r) { return r >= ORC_TOKEN_V1 && r <= ORC_TOKEN_V3; }
static int is_log(int r) { return r >= ORC_BILD && r <= ORC_OPTLOG; }

/* the statistic s and threshold of a log-loss rule for one row */
static void log_rule_stat(int rule, double alpha, double tv, const void* zq, const void* zp,
                          int dtype, int64_t V, double T, const orc_row_stats* sq,
                          const orc_row_stats* sp, double* s, double* threshold,
                          double* mag) {
  if (rule == ORC_BILD) {
    *s = *mag = orc_cross_entropy_row(zq, zp, dtype, V, T, sq, sp);
    *threshold = alpha;
  } else if (rule == ORC_CHOWLOG) {
    *s = *mag = orc_entropy_row(zq, dtype, V, T, sq);
    *threshold = alpha;
  } else { /* H(p) < H(q) - alpha [D_TV]  <=>  H(q) - H(p) > alpha [D_TV] */
    double hq = orc_entropy_row(zq, dtype, V, T, sq), hp = orc_entropy_row(zp, dtype, V, T, sp);
    *s = hq - hp;
    *mag = hq > hp ? hq : hp;
    *threshold = rule == ORC_OPTLOG ? alpha * tv : alpha;
  }
}

int orc_verify(const void* q_logits, const void* p_logits, int dtype, const int32_t* draft,
               const float* uniforms, int32_t B, int32_t gamma, int64_t V,
               const int32_t* rule, const float* alpha, const float* temperature,
               int32_t* accept_len, int32_t* next_token, uint8_t* defer, double* row_stats,
               double* defer_margin, double* accept_margin, double* sample_margin,
               double* sample_norm, int32_t* flags) {
  if (!q_logits || !p_logits || !draft || !uniforms || !rule || !alpha || !temperature ||
      !accept_len || !next_token || !defer)
    return -1;
  if (B < 1 || gamma < 1 || gamma > ORC_MAX_GAMMA || V < 1) return -1;
  if (dtype != ORC_F32 && dtype != ORC_BF16 && dtype != ORC_F64) return -1;
  for (int32_t b = 0; b < B; ++b)
    if (!rule_ok(rule[b], alpha[b]) || !(temperature[b] > 0.0f)) return -1;

  const int32_t G = gamma + 1; /* positions t .. t+gamma */
  int err = 0;

#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t b = 0; b < B; ++b) {
    double* q = malloc(sizeof(double) * (size_t)G * (size_t)V);
    double* p = malloc(sizeof(double) * (size_t)G * (size_t)V);
    double* pi = malloc(sizeof(double) * (size_t)G * (size_t)V);
    double* w = malloc(sizeof(double) * (size_t)V);
    if (!q || !p || !pi || !w) {
      free(q); free(p); free(pi); free(w);
#pragma omp atomic write
      err = 1;
      continue;
    }
    const double T = (double)temperature[b];
    const double al = (double)alpha[b];
    int32_t flag = 0;
    int dl[ORC_MAX_GAMMA + 1];

    /* Score every position: q_{t+j}, p_{t+j} and pi_{t+j} = T_delta(q, p) */
    for (int32_t j = 0; j < G; ++j) {
      int64_t row = (int64_t)b * G + j;
      double* qj = q + (size_t)j * V;
      double* pj = p + (size_t)j * V;
      orc_row_stats sq, sp;
      orc_softmax_row(row_ptr(q_logits, dtype, row, V), dtype, V, T, qj, &sq);
      orc_softmax_row(row_ptr(p_logits, dtype, row, V), dtype, V, T, pj, &sp);
      double tv, mg, s = 0.0;
      const void* zq = row_ptr(q_logits, dtype, row, V);
      const void* zp = row_ptr(p_logits, dtype, row, V);
      if (is_token(rule[b])) {
        /* Alg. 6: pi = q (1 - r) + p eta; reported delta_j = r(x_j) */
        tv = orc_token_target(rule[b], al, qj, pj, V, sp.maxprob, pi + (size_t)j * V, &mg);
        int32_t x = j < gamma ? draft[(int64_t)b * gamma + j] : -1;
        double xmg;
        dl[j] = (x >= 0 && x < V) ? orc_token_r(rule[b], al, qj[x], pj[x], sp.maxprob, &xmg) : 0;
      } else if (rule[b] == ORC_LOSSY) {
        /* Lemma 2: no deferral decision, the target itself is lossy */
        tv = 0.0;
        dl[j] = 0;
        mg = INFINITY;
        orc_lossy_target(al, qj, pj, V, pi + (size_t)j * V);
      } else {
        tv = orc_tv(pj, qj, V);
        if (is_log(rule[b])) {
          double th, mag;
          log_rule_stat(rule[b], al, tv, zq, zp, dtype, V, T, &sq, &sp, &s, &th, &mag);
          dl[j] = orc_log_defer(s, th, mag, &mg);
        } else {
          dl[j] = orc_defer(rule[b], al, sq.maxprob, sp.maxprob, tv, &mg);
        }
        orc_target(dl[j], qj, pj, V, pi + (size_t)j * V);
      }
      defer[row] = (uint8_t)dl[j];
      if (defer_margin) defer_margin[row] = mg;
      if (row_stats) {
        double* rs = row_stats + (size_t)row * 8;
        rs[0] = sq.m; rs[1] = sq.lse; rs[2] = sq.maxprob;
        rs[3] = sp.m; rs[4] = sp.lse; rs[5] = sp.maxprob;
        rs[6] = tv; rs[7] = s;
      }
    }

    /* Accept draws a_j for j < gamma (a_gamma = 0); j* = first zero */
    int32_t jstar = gamma;
    for (int32_t j = 0; j < gamma; ++j) {
      int64_t pos = (int64_t)b * gamma + j;
      int32_t x = draft[pos];
      double u = (double)uniforms[(int64_t)b * G + j];
      int a;
      double mg;
      if (x < 0 || x >= V) { /* outside the vocabulary: rejected */
        a = 0;
        mg = INFINITY;
        flag |= ORC_FLAG_DRAFT_OUT_OF_RANGE;
      } else if (dl[j] == 0 && rule[b] != ORC_LOSSY) { /* pi >= q at x: the ratio is 1 */
        a = 1;
        mg = INFINITY;
      } else {
        a = orc_accept(pi[(size_t)j * V + x], q[(size_t)j * V + x], u, &mg);
      }
      /* draws past j* decide nothing */
      if (accept_margin) accept_margin[pos] = (jstar == gamma) ? mg : INFINITY;
      if (!a && jstar == gamma) jstar = j;
    }

    /* p_res: norm(max(0, pi - q)) at a rejection, else pi_{t+gamma} */
    const double* target;
    double W;
    if (jstar < gamma) {
      W = orc_residual(pi + (size_t)jstar * V, q + (size_t)jstar * V, V, w);
      target = w;
      if (!(W > 0.0)) { /* cannot happen in exact arithmetic (Lemma 3) */
        flag |= ORC_FLAG_EMPTY_RESIDUAL;
        target = p + (size_t)jstar * V;
        W = 0.0;
        for (int64_t v = 0; v < V; ++v) W += target[v];
      }
    } else {
      /* pi_{t+gamma}; for the (unnormalised) lossy target, p_{t+gamma} */
      target = (rule[b] == ORC_LOSSY ? p : pi) + (size_t)gamma * V;
      W = 0.0;
      for (int64_t v = 0; v < V; ++v) W += target[v];
    }
    double smg;
    int32_t tok = orc_sample(target, V, (double)uniforms[(int64_t)b * G + gamma], &smg);

    accept_len[b] = jstar;
    next_token[b] = tok;
    if (sample_margin) sample_margin[b] = smg;
    if (sample_norm) sample_norm[b] = W;
    if (flags) flags[b] = flag;
    free(q); free(p); free(pi); free(w);
  }
  return err ? -1 : 0;
}

int orc_draft_sample(const void* logits, int dtype, int32_t B, int64_t V,
                     const float* temperature, const float* uniforms, int32_t* tokens,
                     double* margin) {
  if (!logits || !temperature || !tokens || B < 1 || V < 1) return -1;
  if (dtype != ORC_F32 && dtype != ORC_BF16 && dtype != ORC_F64) return -1;
  for (int32_t b = 0; b < B; ++b)
    if (!(temperature[b] >= 0.0f) || (temperature[b] > 0.0f && !uniforms)) return -1;
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t b = 0; b < B; ++b) {
    const void* z = row_ptr(logits, dtype, b, V);
    orc_row_stats st;
    if (temperature[b] == 0.0f) { /* greedy: argmax of the raw logits */
      orc_softmax_row(z, dtype, V, 1.0, NULL, &st);
      tokens[b] = st.argmax;
      if (margin) margin[b] = INFINITY;
      continue;
    }
    double* q = malloc(sizeof(double) * (size_t)V);
    if (!q) {
#pragma omp atomic write
      err = 1;
      continue;
    }
    orc_softmax_row(z, dtype, V, (double)temperature[b], q, &st);
    double mg;
    tokens[b] = orc_sample(q, V, (double)uniforms[b], &mg);
    if (margin) margin[b] = mg;
    free(q);
  }
  return err ? -1 : 0;
}

int orc_greedy_verify(const void* q_logits, const void* p_logits, int dtype,
                      const int32_t* draft, int32_t B, int32_t gamma, int64_t V,
                      const int32_t* rule, const float* alpha, int32_t* accept_len,
                      int32_t* next_token, uint8_t* defer, double* row_stats,
                      int32_t* argmax_qp, double* defer_margin, int32_t* flags) {
  if (!q_logits || !p_logits || !draft || !rule || !alpha || !accept_len || !next_token ||
      !defer)
    return -1;
  if (B < 1 || gamma < 1 || gamma > ORC_MAX_GAMMA || V < 1) return -1;
  if (dtype != ORC_F32 && dtype != ORC_BF16 && dtype != ORC_F64) return -1;
  for (int32_t b = 0; b < B; ++b)
    if (!rule_ok(rule[b], alpha[b])) return -1;
  const int32_t G = gamma + 1;

#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t b = 0; b < B; ++b) {
    int32_t aq[ORC_MAX_GAMMA + 1], ap[ORC_MAX_GAMMA + 1], tgt[ORC_MAX_GAMMA + 1];
    int dl[ORC_MAX_GAMMA + 1];
    int32_t flag = 0;
    for (int32_t j = 0; j < G; ++j) {
      int64_t row = (int64_t)b * G + j;
      orc_row_stats sq, sp;
      /* max-probabilities of the temperature-1 softmax; argmax on raw logits */
      orc_softmax_row(row_ptr(q_logits, dtype, row, V), dtype, V, 1.0, NULL, &sq);
      orc_softmax_row(row_ptr(p_logits, dtype, row, V), dtype, V, 1.0, NULL, &sp);
      aq[j] = sq.argmax;
      ap[j] = sp.argmax;
      /* one-hot q~, p~: D_TV(p~, q~) = 1(argmax q != argmax p) */
      double tv = (aq[j] != ap[j]) ? 1.0 : 0.0;
      double mg, s = 0.0;
      const void* zq = row_ptr(q_logits, dtype, row, V);
      const void* zp = row_ptr(p_logits, dtype, row, V);
      if (rule[b] == ORC_LOSSY) {
        /* max{min{q~, p~/(1-alpha)}, p~} is one-hot at argmax p */
        dl[j] = 0;
        mg = INFINITY;
        tgt[j] = ap[j];
      } else if (rule[b] == ORC_BILD) {
        /* D = -log p(argmax q), temperature 1 */
        s = sp.lse - logit_at(zp, dtype, aq[j]);
        dl[j] = orc_log_defer(s, (double)alpha[b], s, &mg);
      } else if (is_log(rule[b])) {
        double th, mag;
        log_rule_stat(rule[b], (double)alpha[b], tv, zq, zp, dtype, V, 1.0, &sq, &sp, &s, &th,
                      &mag);
        dl[j] = orc_log_defer(s, th, mag, &mg);
      } else if (is_token(rule[b])) {
        /* r at the drafter's argmax; eta~ = r(argmax q) for the one-hot q~ */
        const void* prow = row_ptr(p_logits, dtype, row, V);
        double pa = exp(logit_at(prow, dtype, aq[j]) - sp.lse);
        dl[j] = orc_token_r(rule[b], (double)alpha[b], sq.maxprob, pa, sp.maxprob, &mg);
        tv = (double)dl[j];
      } else {
        dl[j] = orc_defer(rule[b], (double)alpha[b], sq.maxprob, sp.maxprob, tv, &mg);
      }
      if (rule[b] != ORC_LOSSY) tgt[j] = dl[j] ? ap[j] : aq[j];
      defer[row] = (uint8_t)dl[j];
      if (defer_margin) defer_margin[row] = mg;
      if (row_stats) {
        double* rs = row_stats + (size_t)row * 8;
        rs[0] = sq.m; rs[1] = sq.lse; rs[2] = sq.maxprob;
        rs[3] = sp.m; rs[4] = sp.lse; rs[5] = sp.maxprob;
        rs[6] = tv; rs[7] = s;
      }
      if (argmax_qp) {
        argmax_qp[row * 2 + 0] = aq[j];
        argmax_qp[row * 2 + 1] = ap[j];
      }
    }
    /* pi~ = (1-delta) q~ + delta p~ is one-hot at (delta ? argmax p : argmax q):
     * a draft is kept exactly when it is that token. */
    int32_t jstar = gamma;
    for (int32_t j = 0; j < gamma; ++j) {
      int32_t x = draft[(int64_t)b * gamma + j];
      if (x < 0 || x >= V) flag |= ORC_FLAG_DRAFT_OUT_OF_RANGE;
      if (x != tgt[j]) {
        jstar = j;
        break;
      }
    }
    /* residual max(0, pi~ - q~) (or the bonus pi~_gamma) is one-hot at the
     * same token */
    accept_len[b] = jstar;
    next_token[b] = tgt[jstar];
    if (flags) flags[b] = flag;
  }
  return 0;
}
