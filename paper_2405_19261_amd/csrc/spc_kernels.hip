// spc_kernels.hip -- gfx950 kernels of the speculative-cascade verify step.
//
// The step (GenSpecSample, Alg. 4, with the cascade target T_delta of eq. (6)
// and the deferral rules of Table 1) runs as up to three vocabulary-streaming
// kernels.  A row is one position (b, j) of one tensor pair (q, p); a tile is
// one chunk of TILE consecutive vocabulary entries of a row.
//
//   k_stats   grid (tiles per row, rows).  Reads every logit of q and p once
//             and reduces each tile to {max z, sum 2^(z c - r)} (c = log2 e / T).
//             The last tile of a row to finish merges the row; the last row of
//             a sequence to finish runs the per-sequence decision (deferral
//             delta_j, accept draws a_j, first rejection j*), and, when the
//             sample is the extra token from q or p, the sample itself.
//   k_tv      only for OPT sequences: D_TV(p, q) = sum_v max(0, p_v - q_v)
//             (Lemma 3) needs both normalisers, so it is a second pass over
//             those rows; its last finisher per sequence runs the decision.
//   k_resid   for sequences rejected at j* < gamma: the mass of the residual
//             max(0, p - q) on each tile of row j*; the last finisher picks the
//             tile and scans it (inverse CDF in vocabulary order).
//
// Completion counters implement "last workgroup to arrive does the next step"
// with device-scope fences; each counter is reset to zero by its last
// arriver, so the zeroed workspace is zero again after every call.  Merges
// run in a fixed order, so results do not depend on scheduling.
#include <math.h>

#include "spc_internal.h"

namespace spc {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr double kLog2e = 1.4426950408889634074;  // log2(e)
constexpr double kLn2 = 0.69314718055994530942;   // ln(2)

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ geometry
template <int DT, bool VEC>
struct Geo {
  static constexpr int EB = (DT == 1) ? 2 : 4;  // element bytes (1 = bf16, 0 = f32)
  static constexpr int VW = VEC ? 16 / EB : 1;  // elements per lane load
  static constexpr int NW = VEC ? 4 : 1;        // 32-bit words per lane load
  static constexpr int U = VEC ? 8 : 16;        // lane loads per tensor per tile
  static constexpr int SLOTS = kThreads * U;    // lane loads per tensor per tile
  static constexpr int TILE = SLOTS * VW;       // vocabulary entries per tile
};

// bfloat16 -> float32 is exact: the bf16 bits are the top half of the float.
template <int DT, bool VEC>
__device__ __forceinline__ float elem(const uint32_t* w, int e) {
  if constexpr (DT == 1) {
    if constexpr (VEC) {
      const uint32_t x = w[e >> 1];
      return (e & 1) ? __uint_as_float(x & 0xffff0000u) : __uint_as_float(x << 16);
    } else {
      return __uint_as_float(w[0] << 16);
    }
  } else {
    return __uint_as_float(w[VEC ? e : 0]);
  }
}

// One lane load: VW entries starting at entry `slot * VW` of a row; entries
// at or past V read as -inf (they add nothing to any sum or max).
template <int DT, bool VEC, bool NT>
__device__ __forceinline__ void load_slot(const char* row, int64_t slot, int V, uint32_t* w) {
  using G = Geo<DT, VEC>;
  const int64_t e0 = slot * G::VW;
  if (e0 < V) {
    if constexpr (VEC) {
      const u32x4* src = reinterpret_cast<const u32x4*>(row + e0 * G::EB);
      u32x4 v;
      if constexpr (NT) v = __builtin_nontemporal_load(src);
      else v = *src;
      w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    } else if constexpr (DT == 1) {
      w[0] = *reinterpret_cast<const uint16_t*>(row + e0 * 2);
    } else {
      w[0] = *reinterpret_cast<const uint32_t*>(row + e0 * 4);
    }
  } else {
#pragma unroll
    for (int i = 0; i < G::NW; ++i) w[i] = (DT == 1) ? 0xff80ff80u : 0xff800000u;
  }
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// ------------------------------------------- cross-workgroup communication
// Agent-scope fences on gfx950 write back and invalidate the whole L2, which
// is ruinous when thousands of workgroups each publish a few bytes.  Instead,
// data shared between workgroups of one launch is written and read with
// agent-scope relaxed atomics (write-through / read-through the L2), and the
// order "data, then counter" is enforced by waiting for the stores to
// complete before the counter update (and the counter read before the data
// reads).
template <typename T>
__device__ __forceinline__ void st_dev(T* dst, const T& v) {
  static_assert(sizeof(T) % 8 == 0, "8-byte words");
  uint64_t w[sizeof(T) / 8];
  __builtin_memcpy(w, &v, sizeof(T));
  uint64_t* d = reinterpret_cast<uint64_t*>(dst);
#pragma unroll
  for (unsigned i = 0; i < sizeof(T) / 8; ++i)
    __hip_atomic_store(d + i, w[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename T>
__device__ __forceinline__ T ld_dev(const T* src) {
  static_assert(sizeof(T) % 8 == 0, "8-byte words");
  uint64_t w[sizeof(T) / 8];
  uint64_t* s = reinterpret_cast<uint64_t*>(const_cast<T*>(src));
#pragma unroll
  for (unsigned i = 0; i < sizeof(T) / 8; ++i)
    w[i] = __hip_atomic_load(s + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  T v;
  __builtin_memcpy(&v, w, sizeof(T));
  return v;
}

__device__ __forceinline__ void st_dev_f64(double* dst, double v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(dst), __double_as_longlong(v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double ld_dev_f64(const double* src) {
  return __longlong_as_double((long long)__hip_atomic_load(
      reinterpret_cast<uint64_t*>(const_cast<double*>(src)), __ATOMIC_RELAXED,
      __HIP_MEMORY_SCOPE_AGENT));
}

// Every vector-memory operation issued so far by this wave has completed.
__device__ __forceinline__ void vmem_drain() {
  __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xf << 8));  // vmcnt(0)
}

// ------------------------------------------------------- wavefront reductions
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ int wave_maxi(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
  return v;
}

struct PickState {
  int k;        // tile holding the sample
  int kind;     // SampleKind actually sampled
  double rem;   // target mass remaining at the start of that tile
};

struct Shared {
  float m[4][2];
  double d[4][2];
  int i[4][2];
  double scan[4];
  int flag;
  SeqState seq;
  PickState pk;
};

// All threads receive the block-wide max of (a, b).
__device__ __forceinline__ void block_max2(float& a, float& b, Shared& sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  a = wave_max(a);
  b = wave_max(b);
  if (lane == 0) { sh.m[wv][0] = a; sh.m[wv][1] = b; }
  __syncthreads();
  a = fmaxf(fmaxf(sh.m[0][0], sh.m[1][0]), fmaxf(sh.m[2][0], sh.m[3][0]));
  b = fmaxf(fmaxf(sh.m[0][1], sh.m[1][1]), fmaxf(sh.m[2][1], sh.m[3][1]));
}

// Block sums in a fixed order; valid in every thread.
__device__ __forceinline__ void block_sum2(double& a, double& b, Shared& sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  a = wave_sum(a);
  b = wave_sum(b);
  __syncthreads();  // sh.d may still be read by an earlier step
  if (lane == 0) { sh.d[wv][0] = a; sh.d[wv][1] = b; }
  __syncthreads();
  a = ((sh.d[0][0] + sh.d[1][0]) + sh.d[2][0]) + sh.d[3][0];
  b = ((sh.d[0][1] + sh.d[1][1]) + sh.d[2][1]) + sh.d[3][1];
}

__device__ __forceinline__ void block_min2(int& a, int& b, Shared& sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  a = wave_min(a);
  b = wave_min(b);
  __syncthreads();
  if (lane == 0) { sh.i[wv][0] = a; sh.i[wv][1] = b; }
  __syncthreads();
  a = min(min(sh.i[0][0], sh.i[1][0]), min(sh.i[2][0], sh.i[3][0]));
  b = min(min(sh.i[0][1], sh.i[1][1]), min(sh.i[2][1], sh.i[3][1]));
}

// Inclusive prefix sum over the block's threads in thread order (fp64); the
// last thread's value equals *total bit for bit.
__device__ __forceinline__ double block_incl_scan(double v, Shared& sh, double* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double n = __shfl_up(v, o, 64);
    if (lane >= o) v += n;
  }
  __syncthreads();
  if (lane == 63) sh.scan[wv] = v;
  __syncthreads();
  double off = 0.0;
  for (int w = 0; w < wv; ++w) off += sh.scan[w];
  *total = ((sh.scan[0] + sh.scan[1]) + sh.scan[2]) + sh.scan[3];
  return off + v;
}

// ------------------------------------------------------ per-sequence params
struct SeqParam {
  int rule;
  double alpha;
  double c;         // log2(e) / T  (T = 1 for greedy statistics)
  float c_hi, c_lo; // c = c_hi + c_lo with c_hi < c, c_lo > 0 (float32 pair)
  bool greedy;
  bool valid;
};

__device__ SeqParam seq_param(const Params& P, int b) {
  SeqParam s;
  s.rule = P.rule_ps ? P.rule_ps[b] : P.rule;
  const float alpha = P.alpha_ps ? P.alpha_ps[b] : P.alpha;
  const float T = P.temp_ps ? P.temp_ps[b] : P.temp;
  s.alpha = (double)alpha;
  s.valid = s.rule >= SPC_RULE_CHOW && s.rule <= SPC_RULE_NEVER && isfinite(alpha) &&
            isfinite(T) && T >= 0.0f && (T == 0.0f || T >= 1e-20f);
  s.greedy = P.force_greedy || T == 0.0f;
  s.c = kLog2e / ((s.greedy || !s.valid) ? 1.0 : (double)T);
  // split c so that z*c_hi + z*c_lo carries ~48 bits of c; c_lo > 0 keeps
  // -inf logits at -inf (never -inf + inf)
  float hi = __double2float_rd(s.c);
  if ((double)hi == s.c) hi = __uint_as_float(__float_as_uint(hi) - 1u);
  s.c_hi = hi;
  s.c_lo = (float)(s.c - (double)hi);
  return s;
}

__device__ __forceinline__ bool needs_tv(const SeqParam& s) {
  return s.valid && !s.greedy && s.rule == SPC_RULE_OPT;
}

// log2 of a normalised probability, evaluated as two float32 halves:
// z*c - lz = (z*c_hi - l_hi) + (z*c_lo - l_lo).
struct ProbScale {
  float c_hi, c_lo, q_hi, q_lo, p_hi, p_lo;
  double c;   // log2(e) / T
  double dl;  // lz_p - lz_q
};

__device__ __forceinline__ ProbScale prob_scale(const SeqParam& s, const RowStat& rs) {
  ProbScale ps;
  ps.c_hi = s.c_hi;
  ps.c_lo = s.c_lo;
  ps.q_hi = (float)rs.lz_q;
  ps.q_lo = (float)(rs.lz_q - (double)ps.q_hi);
  ps.p_hi = (float)rs.lz_p;
  ps.p_lo = (float)(rs.lz_p - (double)ps.p_hi);
  ps.c = s.c;
  ps.dl = rs.lz_p - rs.lz_q;
  return ps;
}

__device__ __forceinline__ float prob(float z, float c_hi, float c_lo, float l_hi, float l_lo) {
  return exp2_hw(fmaf(z, c_hi, -l_hi) + fmaf(z, c_lo, -l_lo));
}

// 2^d - 1 for d > 0 with a relative error of a few float32 ulps: a Taylor
// series of expm1(x), x = d ln 2, below d = 1/4 (where 2^d - 1 would cancel),
// the hardware 2^d above.
__device__ __forceinline__ float exp2m1_pos(float d) {
  const float x = d * 0.693147180559945309f;
  const float series =
      x * (1.0f + x * (0.5f + x * (1.0f / 6 + x * (1.0f / 24 + x * (1.0f / 120 + x * (1.0f / 720))))));
  return d < 0.25f ? series : exp2_hw(d) - 1.0f;
}

// Residual weight max(0, p_v - q_v) = q_v * max(0, 2^d - 1), d = log2(p_v / q_v)
// evaluated in fp64 so that p ~ q does not cancel.
__device__ __forceinline__ float residual_weight(float zq, float zp, const ProbScale& s) {
  // zp - zq is exact in fp64, so identical rows give d = 0 exactly
  const double d64 = fma((double)zp - (double)zq, s.c, -s.dl);
  const float d = (float)d64;
  if (!(d > 0.0f)) return 0.0f;  // p <= q, or both -inf
  if (zq == -__builtin_huge_valf()) return prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
  return prob(zq, s.c_hi, s.c_lo, s.q_hi, s.q_lo) * exp2m1_pos(d);
}

// Weight of one entry under the distribution sampled at j*.
__device__ __forceinline__ float sample_weight(int kind, float zq, float zp, const ProbScale& s) {
  if (kind == kQ) return prob(zq, s.c_hi, s.c_lo, s.q_hi, s.q_lo);
  if (kind == kP) return prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
  return residual_weight(zq, zp, s);
}

template <int DT>
__device__ __forceinline__ float load_logit(const void* base, int64_t row, int V, int x) {
  const int64_t i = row * (int64_t)V + x;
  if constexpr (DT == 1) {
    return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(base)[i] << 16);
  } else {
    return reinterpret_cast<const float*>(base)[i];
  }
}

// Table 1 deferral rules (strict inequalities as printed).
__device__ __forceinline__ int defer_rule(int rule, double alpha, double maxq, double maxp,
                                          double tv) {
  switch (rule) {
    case SPC_RULE_CHOW: return maxq < 1.0 - alpha;           // eq. (2)
    case SPC_RULE_DIFF: return maxq < maxp - alpha;          // eq. (5)
    case SPC_RULE_OPT: return maxq < maxp - alpha * tv;      // eq. (11)
    case SPC_RULE_ALWAYS: return 1;
    default: return 0;
  }
}

// --------------------------------------------------------------- row merge
// Wave 0 merges the K tile partials of row r into its RowStat (lane 0 writes).
__device__ void row_merge(const Params& P, int r, bool greedy) {
  const int lane = threadIdx.x;
  const int K = P.K;
  const TilePart* t = P.tiles + (int64_t)r * K;
  float rq = kNegInf, rp = kNegInf, zq = kNegInf, zp = kNegInf;
  for (int k = lane; k < K; k += 64) {
    const TilePart tk = ld_dev(t + k);
    rq = fmaxf(rq, tk.r_q);
    rp = fmaxf(rp, tk.r_p);
    zq = fmaxf(zq, tk.zmax_q);
    zp = fmaxf(zp, tk.zmax_p);
  }
  rq = wave_max(rq); rp = wave_max(rp); zq = wave_max(zq); zp = wave_max(zp);
  double sq = 0.0, sp = 0.0;
  int aq = 0x7fffffff, ap = 0x7fffffff;
  for (int k = lane; k < K; k += 64) {
    const TilePart tk = ld_dev(t + k);
    if (tk.r_q != kNegInf) sq += tk.s_q * exp2((double)tk.r_q - (double)rq);
    if (tk.r_p != kNegInf) sp += tk.s_p * exp2((double)tk.r_p - (double)rp);
    if (greedy) {
      if (tk.zmax_q == zq) aq = min(aq, tk.amax_q);
      if (tk.zmax_p == zp) ap = min(ap, tk.amax_p);
    }
  }
  sq = wave_sum(sq); sp = wave_sum(sp);
  aq = wave_min(aq); ap = wave_min(ap);
  if (lane == 0) {
    RowStat rs;
    rs.lz_q = (double)rq + log2(sq);
    rs.lz_p = (double)rp + log2(sp);
    rs.tv = 0.0;
    rs.zmax_q = zq;
    rs.zmax_p = zp;
    rs.amax_q = greedy ? aq : -1;
    rs.amax_p = greedy ? ap : -1;
    st_dev(P.rows + r, rs);
  }
}

// ------------------------------------------------------------- decision
// Wave 0: delta_j and the accept draws of one sequence, j*, and the outputs
// that follow from them (Alg. 4, first-rejection search by one ballot).
template <int DT>
__device__ void decide(const Params& P, int b, const SeqParam& sp, Shared& sh) {
  const int lane = threadIdx.x;
  const int gamma = P.gamma, g1 = gamma + 1;
  const bool on = lane < g1;
  const int64_t row = (int64_t)b * g1 + lane;
  if (!sp.valid) {
    if (on) P.out_defer[row] = 0;
    if (lane == 0) {
      P.out_accept[b] = -1;
      P.out_token[b] = -1;
      if (P.out_norm) P.out_norm[b] = 0.0f;
      sh.seq = SeqState{-1, kNone, 0.0f, 0};
    }
    return;
  }
  int delta = 0, keep = 1;
  RowStat rs{};
  if (on) {
    rs = ld_dev(P.rows + row);
    const double maxq = exp2((double)rs.zmax_q * sp.c - rs.lz_q);
    const double maxp = exp2((double)rs.zmax_p * sp.c - rs.lz_p);
    // greedy: one-hot q~, p~ give D_TV = 1(argmax q != argmax p)  (Lemma 6)
    const double tv = sp.greedy ? (rs.amax_q != rs.amax_p ? 1.0 : 0.0) : rs.tv;
    delta = defer_rule(sp.rule, sp.alpha, maxq, maxp, tv);
    if (lane < gamma) {
      const int x = P.draft[(int64_t)b * gamma + lane];
      if (x < 0 || x >= P.V) {
        keep = 0;
      } else if (sp.greedy) {
        keep = (x == (delta ? rs.amax_p : rs.amax_q));
      } else if (delta) {
        // pi = p here; keep if p(x) >= q(x), else with probability p(x)/q(x)
        const double lq = (double)load_logit<DT>(P.q, row, P.V, x) * sp.c - rs.lz_q;
        const double lp = (double)load_logit<DT>(P.p, row, P.V, x) * sp.c - rs.lz_p;
        if (lp < lq) keep = (double)P.uniforms[(int64_t)b * g1 + lane] < exp2(lp - lq);
      }
    } else {
      keep = 0;  // a_gamma = 0
    }
    P.out_defer[row] = (uint8_t)delta;
    if (P.out_stats) {
      const double T = sp.greedy ? 1.0 : kLog2e / sp.c;
      float* o = P.out_stats + row * 8;
      o[0] = (float)((double)rs.zmax_q / T);
      o[1] = (float)(rs.lz_q * kLn2);
      o[2] = (float)maxq;
      o[3] = (float)((double)rs.zmax_p / T);
      o[4] = (float)(rs.lz_p * kLn2);
      o[5] = (float)maxp;
      o[6] = (float)tv;
      o[7] = 0.0f;
    }
    if (P.out_argmax) {
      P.out_argmax[row * 2 + 0] = rs.amax_q;
      P.out_argmax[row * 2 + 1] = rs.amax_p;
    }
  }
  const unsigned long long rej = __ballot(on && !keep);
  const int jstar = __ffsll(rej) - 1;  // bit gamma is always set
  const int dstar = __shfl(delta, jstar, 64);
  const int aq = __shfl(rs.amax_q, jstar, 64);
  const int ap = __shfl(rs.amax_p, jstar, 64);
  if (lane == 0) {
    P.out_accept[b] = jstar;
    SeqState s{b * g1 + jstar, kNone, 0.0f, 0};
    if (sp.greedy) {
      P.out_token[b] = dstar ? ap : aq;
      if (P.out_norm) P.out_norm[b] = 1.0f;
    } else {
      // a rejection with delta = 0 only happens for an out-of-range draft;
      // its residual max(0, q - q) is empty, so p is sampled instead
      s.kind = (jstar < gamma) ? (dstar ? kResidual : kP) : (dstar ? kP : kQ);
      s.u = P.uniforms[(int64_t)b * g1 + gamma];
    }
    sh.seq = s;
  }
}

// Mass of tile k under `kind` (Q/P from the statistics pass, residual from
// the residual pass).
__device__ __forceinline__ double tile_mass(const Params& P, int b, int row, int k, int kind,
                                            const RowStat& rs) {
  if (kind == kResidual) return ld_dev_f64(P.masses + (int64_t)b * P.K + k);
  const TilePart t = ld_dev(P.tiles + (int64_t)row * P.K + k);
  const float r = (kind == kQ) ? t.r_q : t.r_p;
  if (r == kNegInf) return 0.0;
  const double s = (kind == kQ) ? t.s_q : t.s_p;
  return s * exp2((double)r - ((kind == kQ) ? rs.lz_q : rs.lz_p));
}

// Whole block: inverse-CDF draw at row s.row.  The smallest entry k with
// C_k > u * W (C the running mass in vocabulary order): tile masses -> tile,
// then block-wide inclusive scans over the tile's lane loads -> lane, then a
// sequential search inside the lane's entries.
template <int DT, bool VEC>
__device__ void pick(const Params& P, int b, const SeqState& s, const SeqParam& sp,
                     Shared& sh) {
  using G = Geo<DT, VEC>;
  const int tid = threadIdx.x;
  const int K = P.K;
  const RowStat rs = ld_dev(P.rows + s.row);
  if (tid == 0) {
    int kind = s.kind;
    double W = 0.0;
    for (int k = 0; k < K; ++k) W += tile_mass(P, b, s.row, k, kind, rs);
    if (kind == kResidual && !(W > 0.0)) {  // empty residual (rounding): sample p
      kind = kP;
      W = 0.0;
      for (int k = 0; k < K; ++k) W += tile_mass(P, b, s.row, k, kind, rs);
    }
    const double target = (double)s.u * W;
    double C = 0.0, rem = 0.0;
    int ks = -1, klast = -1;
    for (int k = 0; k < K; ++k) {
      const double m = tile_mass(P, b, s.row, k, kind, rs);
      if (m > 0.0) klast = k;
      if (ks < 0 && C + m > target) {
        ks = k;
        rem = target - C;
      }
      C += m;
    }
    if (ks < 0) {  // rounding left u*W at or past the end: last entry with mass
      ks = klast;
      rem = __builtin_huge_val();
    }
    sh.pk = PickState{ks, kind, rem};
    if (P.out_norm) P.out_norm[b] = (float)W;
  }
  __syncthreads();
  const PickState pk = sh.pk;
  if (pk.k < 0) {
    if (tid == 0) P.out_token[b] = -1;
    return;
  }
  const ProbScale ps = prob_scale(sp, rs);
  const int V = P.V;
  const char* qrow = (const char*)P.q + (int64_t)s.row * V * G::EB;
  const char* prow = (const char*)P.p + (int64_t)s.row * V * G::EB;
  const int64_t slot0 = (int64_t)pk.k * G::SLOTS;
  double rem = pk.rem;
  int token = 0x7fffffff, last_pos = -1;
  for (int i = 0; i < G::U; ++i) {
    const int64_t slot = slot0 + (int64_t)i * kThreads + tid;
    uint32_t wq[G::NW], wp[G::NW];
    load_slot<DT, VEC, false>(qrow, slot, V, wq);
    load_slot<DT, VEC, false>(prow, slot, V, wp);
    float w[G::VW];
    double tsum = 0.0;
#pragma unroll
    for (int e = 0; e < G::VW; ++e) {
      w[e] = sample_weight(pk.kind, elem<DT, VEC>(wq, e), elem<DT, VEC>(wp, e), ps);
      tsum += (double)w[e];
      if (w[e] > 0.0f) last_pos = (int)(slot * G::VW + e);
    }
    double total;
    const double incl = block_incl_scan(tsum, sh, &total);
    if (total > rem) {  // block-uniform: the draw falls in this block of entries
      int cand = (incl > rem) ? tid : 0x7fffffff, unused = 0;
      block_min2(cand, unused, sh);
      if (tid == cand) {
        double run = incl - tsum;
        int hit = -1, lastw = -1;
#pragma unroll
        for (int e = 0; e < G::VW; ++e) {
          run += (double)w[e];
          if (w[e] > 0.0f) lastw = e;
          if (hit < 0 && run > rem) hit = e;
        }
        if (hit < 0) hit = lastw;  // rounding inside the lane: its last entry with mass
        P.out_token[b] = (int)(slot * G::VW + hit);
      }
      return;
    }
    rem -= total;
  }
  // rounding: no block reached u*W; take the last entry of the tile with mass
  int lp = last_pos, unused = 0;
  lp = -lp;
  block_min2(lp, unused, sh);
  if (tid == 0) P.out_token[b] = -lp;
  (void)token;
}

// After the decision: sample now (extra token from q or p) or leave the
// sequence to the residual pass.
template <int DT, bool VEC>
__device__ void decide_and_sample(const Params& P, int b, const SeqParam& sp, Shared& sh) {
  if (threadIdx.x < 64) decide<DT>(P, b, sp, sh);
  __syncthreads();
  const SeqState s = sh.seq;
  if (threadIdx.x == 0) st_dev(P.seqs + b, s);
  if (s.kind == kQ || s.kind == kP) pick<DT, VEC>(P, b, s, sp, sh);
}

// "Am I the last of `n` arrivals?" for the whole block.  Data this block
// shares was written with st_dev by thread 0 before the call; on true, the
// counter is reset and the caller reads the other arrivals' data with ld_dev.
__device__ __forceinline__ bool arrive_last(uint32_t* cnt, uint32_t n, Shared& sh) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    vmem_drain();  // this thread's shared stores are complete
    const uint32_t prev =
        __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const bool last = (prev == n - 1);
    if (last) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    sh.flag = last;
  }
  __syncthreads();
  const bool last = sh.flag;
  if (last) {
    vmem_drain();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  }
  return last;
}

// ================================================================ kernels

template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void k_stats(Params P) {
  using G = Geo<DT, VEC>;
  __shared__ Shared sh;
  const int k = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  const int g1 = P.gamma + 1, b = r / g1;
  const SeqParam sp = seq_param(P, b);
  const int V = P.V;
  const char* qrow = (const char*)P.q + (int64_t)r * V * G::EB;
  const char* prow = (const char*)P.p + (int64_t)r * V * G::EB;
  const int64_t slot0 = (int64_t)k * G::SLOTS;

  uint32_t wq[G::U][G::NW], wp[G::U][G::NW];
#pragma unroll
  for (int i = 0; i < G::U; ++i) {
    load_slot<DT, VEC, true>(qrow, slot0 + i * kThreads + tid, V, wq[i]);
    load_slot<DT, VEC, true>(prow, slot0 + i * kThreads + tid, V, wp[i]);
  }
  float mq = kNegInf, mp = kNegInf;
#pragma unroll
  for (int i = 0; i < G::U; ++i)
#pragma unroll
    for (int e = 0; e < G::VW; ++e) {
      mq = fmaxf(mq, elem<DT, VEC>(wq[i], e));
      mp = fmaxf(mp, elem<DT, VEC>(wp[i], e));
    }
  float Mq = mq, Mp = mp;
  block_max2(Mq, Mp, sh);

  int aq = -1, ap = -1;
  if (sp.greedy) {  // lowest entry attaining the tile max (only lanes holding it search)
    int cq = 0x7fffffff, cp = 0x7fffffff;
    if (mq == Mq && Mq != kNegInf) {
      for (int i = 0; i < G::U && cq == 0x7fffffff; ++i)
        for (int e = 0; e < G::VW; ++e)
          if (elem<DT, VEC>(wq[i], e) == Mq) {
            cq = (int)((slot0 + i * kThreads + tid) * G::VW + e);
            break;
          }
    }
    if (mp == Mp && Mp != kNegInf) {
      for (int i = 0; i < G::U && cp == 0x7fffffff; ++i)
        for (int e = 0; e < G::VW; ++e)
          if (elem<DT, VEC>(wp[i], e) == Mp) {
            cp = (int)((slot0 + i * kThreads + tid) * G::VW + e);
            break;
          }
    }
    block_min2(cq, cp, sh);
    aq = cq;
    ap = cp;
  }

  // sum over the tile of 2^(z c - r), r = Mq * c_hi rounded (a reference, not
  // an exact product: the partial is exact with respect to its own r)
  const float rq = (Mq == kNegInf) ? 0.0f : Mq * sp.c_hi;
  const float rp = (Mp == kNegInf) ? 0.0f : Mp * sp.c_hi;
  float sq = 0.0f, spp = 0.0f;
#pragma unroll
  for (int i = 0; i < G::U; ++i) {
    float tq[G::VW], tp[G::VW];
#pragma unroll
    for (int e = 0; e < G::VW; ++e) {
      const float zq = elem<DT, VEC>(wq[i], e), zp = elem<DT, VEC>(wp[i], e);
      tq[e] = exp2_hw(fmaf(zq, sp.c_lo, fmaf(zq, sp.c_hi, -rq)));
      tp[e] = exp2_hw(fmaf(zp, sp.c_lo, fmaf(zp, sp.c_hi, -rp)));
    }
#pragma unroll
    for (int w = 1; w < G::VW; w <<= 1)
#pragma unroll
      for (int e = 0; e + w < G::VW; e += 2 * w) {
        tq[e] += tq[e + w];
        tp[e] += tp[e + w];
      }
    sq += tq[0];
    spp += tp[0];
  }
  double Sq = sq, Sp = spp;
  block_sum2(Sq, Sp, sh);
  if (tid == 0) {
    TilePart t;
    t.s_q = Sq;
    t.s_p = Sp;
    t.r_q = (Mq == kNegInf) ? kNegInf : rq;
    t.r_p = (Mp == kNegInf) ? kNegInf : rp;
    t.zmax_q = Mq;
    t.zmax_p = Mp;
    t.amax_q = aq;
    t.amax_p = ap;
    st_dev(P.tiles + (int64_t)r * P.K + k, t);
  }
  if (!arrive_last(P.row_cnt + r, (uint32_t)P.K, sh)) return;
  if (tid < 64) row_merge(P, r, sp.greedy);
  if (!arrive_last(P.seq_cnt + b, (uint32_t)g1, sh)) return;
  if (needs_tv(sp)) return;  // the TV pass decides OPT sequences
  decide_and_sample<DT, VEC>(P, b, sp, sh);
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void k_tv(Params P) {
  using G = Geo<DT, VEC>;
  __shared__ Shared sh;
  const int k = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  const int g1 = P.gamma + 1, b = r / g1;
  const SeqParam sp = seq_param(P, b);
  if (!needs_tv(sp)) return;  // block-uniform
  const RowStat rs = ld_dev(P.rows + r);
  const ProbScale ps = prob_scale(sp, rs);
  const int V = P.V;
  const char* qrow = (const char*)P.q + (int64_t)r * V * G::EB;
  const char* prow = (const char*)P.p + (int64_t)r * V * G::EB;
  const int64_t slot0 = (int64_t)k * G::SLOTS;
  uint32_t wq[G::U][G::NW], wp[G::U][G::NW];
#pragma unroll
  for (int i = 0; i < G::U; ++i) {
    load_slot<DT, VEC, true>(qrow, slot0 + i * kThreads + tid, V, wq[i]);
    load_slot<DT, VEC, true>(prow, slot0 + i * kThreads + tid, V, wp[i]);
  }
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < G::U; ++i) {
    float t[G::VW];
#pragma unroll
    for (int e = 0; e < G::VW; ++e)
      t[e] = sample_weight(kResidual, elem<DT, VEC>(wq[i], e), elem<DT, VEC>(wp[i], e), ps);
#pragma unroll
    for (int w = 1; w < G::VW; w <<= 1)
#pragma unroll
      for (int e = 0; e + w < G::VW; e += 2 * w) t[e] += t[e + w];
    acc += t[0];
  }
  double tv = acc, unused = 0.0;
  block_sum2(tv, unused, sh);
  if (tid == 0) st_dev_f64(P.tvpart + (int64_t)r * P.K + k, tv);
  if (!arrive_last(P.tv_row_cnt + r, (uint32_t)P.K, sh)) return;
  if (tid == 0) {
    double s = 0.0;
    for (int j = 0; j < P.K; ++j) s += ld_dev_f64(P.tvpart + (int64_t)r * P.K + j);
    st_dev_f64(&P.rows[r].tv, s);
  }
  if (!arrive_last(P.tv_seq_cnt + b, (uint32_t)g1, sh)) return;
  decide_and_sample<DT, VEC>(P, b, sp, sh);
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void k_resid(Params P) {
  using G = Geo<DT, VEC>;
  __shared__ Shared sh;
  const int k = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const SeqState s = ld_dev(P.seqs + b);
  if (s.kind != kResidual) return;  // block-uniform
  const SeqParam sp = seq_param(P, b);
  const RowStat rs = ld_dev(P.rows + s.row);
  const ProbScale ps = prob_scale(sp, rs);
  const int V = P.V;
  const char* qrow = (const char*)P.q + (int64_t)s.row * V * G::EB;
  const char* prow = (const char*)P.p + (int64_t)s.row * V * G::EB;
  const int64_t slot0 = (int64_t)k * G::SLOTS;
  uint32_t wq[G::U][G::NW], wp[G::U][G::NW];
#pragma unroll
  for (int i = 0; i < G::U; ++i) {
    load_slot<DT, VEC, false>(qrow, slot0 + i * kThreads + tid, V, wq[i]);
    load_slot<DT, VEC, false>(prow, slot0 + i * kThreads + tid, V, wp[i]);
  }
  double acc = 0.0;
#pragma unroll
  for (int i = 0; i < G::U; ++i)
#pragma unroll
    for (int e = 0; e < G::VW; ++e)
      acc += (double)sample_weight(kResidual, elem<DT, VEC>(wq[i], e),
                                   elem<DT, VEC>(wp[i], e), ps);
  double unused = 0.0;
  block_sum2(acc, unused, sh);
  if (tid == 0) st_dev_f64(P.masses + (int64_t)b * P.K + k, acc);
  if (!arrive_last(P.samp_cnt + b, (uint32_t)P.K, sh)) return;
  pick<DT, VEC>(P, b, s, sp, sh);
}

template <int DT, bool VEC>
hipError_t launch_t(const Params& P, bool need_tv, bool need_sample, hipEvent_t e0,
                    hipEvent_t e1, hipStream_t st) {
  const unsigned R = (unsigned)(P.B * (P.gamma + 1));
  hipError_t err;
  if (e0 && (err = hipEventRecord(e0, st)) != hipSuccess) return err;
  hipLaunchKernelGGL((k_stats<DT, VEC>), dim3(P.K, R), dim3(kThreads), 0, st, P);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  if (e1 && (err = hipEventRecord(e1, st)) != hipSuccess) return err;
  if (need_tv) {
    hipLaunchKernelGGL((k_tv<DT, VEC>), dim3(P.K, R), dim3(kThreads), 0, st, P);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  if (need_sample) {
    hipLaunchKernelGGL((k_resid<DT, VEC>), dim3(P.K, P.B), dim3(kThreads), 0, st, P);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace

int tile_elems(int dtype, bool vec) {
  if (dtype == 1) return vec ? Geo<1, true>::TILE : Geo<1, false>::TILE;
  return vec ? Geo<0, true>::TILE : Geo<0, false>::TILE;
}

hipError_t launch_verify(const Params& P, int dtype, bool vec, bool need_tv, bool need_sample,
                         hipEvent_t e0, hipEvent_t e1, hipStream_t st) {
  if (dtype == 1) {
    return vec ? launch_t<1, true>(P, need_tv, need_sample, e0, e1, st)
               : launch_t<1, false>(P, need_tv, need_sample, e0, e1, st);
  }
  return vec ? launch_t<0, true>(P, need_tv, need_sample, e0, e1, st)
             : launch_t<0, false>(P, need_tv, need_sample, e0, e1, st);
}

}  // namespace spc
