// spc_kernels.hip -- gfx950 kernels of the speculative-cascade verify step.
//
// The step (GenSpecSample, Alg. 4, with the cascade target T_delta of eq. (6)
// and the deferral rules of Table 1) runs as two or three kernels.  A row is
// one position (b, j) of the logit pair (q, p); rows are cut into tiles of
// consecutive vocabulary entries.
//
//   k_stats   grid (stats tiles per row, rows), one small tile per workgroup.
//             Reads every logit of q and p once and reduces the tile to
//             {max z, sum 2^(z c - r)} for both tensors (c = log2(e) / T);
//             the tile partial goes to the workspace with plain stores.
//   k_tv      OPT sequences at temperature > 0 only: D_TV(p, q) of Lemma 3
//             needs both normalisers, so it is a second pass over those rows,
//             one partial per tile.
//   k_sample  grid (sample tiles per row, sequences).  Every workgroup of
//             sequence b merges that sequence's row partials and takes the
//             per-sequence decision (deferral delta_j, accept draws a_j, first
//             rejection j*) -- a small, fixed-order computation, so every
//             workgroup reaches the same result -- then computes the mass of
//             its tile of row j* under the sampled distribution (residual
//             max(0, p - q), or the extra-token target q or p).  The last tile
//             to finish picks the token: inverse CDF in vocabulary order.
//
// Kernel boundaries order the passes; within k_sample one completion counter
// per sequence ("last workgroup to arrive draws") is reset by its last
// arriver, so the zeroed workspace is zero again after every call.  All
// merges run in a fixed order: results do not depend on scheduling.
#include <math.h>

#include "spc_internal.h"

namespace spc {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr double kLog2e = 1.4426950408889634074;  // log2(e)
constexpr double kLn2 = 0.69314718055994530942;   // ln(2)

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ geometry
// A lane load is one 16-byte vector (8 bf16 or 4 f32 entries) on the vector
// path, one entry on the scalar path (rows not 16-byte aligned).  A tile is U
// lane loads per thread, U * kThreads * VW entries.
template <int DT, bool VEC, int U_>
struct Tile {
  static constexpr int EB = (DT == 1) ? 2 : 4;  // element bytes (1 = bf16, 0 = f32)
  static constexpr int VW = VEC ? 16 / EB : 1;  // entries per lane load
  static constexpr int NW = VEC ? 4 : 1;        // 32-bit words per lane load
  static constexpr int U = U_;                  // lane loads per thread
  static constexpr int N = kThreads * U * VW;   // entries per tile
};
// statistics / TV tiles: small, so that many workgroups are resident
template <int DT, bool VEC>
using StatTile = Tile<DT, VEC, VEC ? 2 : 8>;
// sampling tiles
template <int DT, bool VEC>
using SampTile = Tile<DT, VEC, VEC ? 8 : 16>;

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

// Lane loads of one tile of one row into w[U][NW].  Thread t's lane load i
// covers entries e = t0 + (OWN ? t*U + i : i*kThreads + t) * VW .. + VW - 1:
// interleaved (coalesced) when OWN is false, thread-contiguous when true.
// Entries at or past `end` read as -inf; a lane past the end re-reads a valid
// address and discards the value, so the loads are branch-free.
template <int DT, bool VEC, int U, bool OWN, bool NT>
__device__ __forceinline__ void load_tile(const char* row, int64_t t0, int64_t end,
                                          uint32_t (&w)[U][Tile<DT, VEC, U>::NW]) {
  using T = Tile<DT, VEC, U>;
  constexpr uint32_t kPad = (DT == 1) ? 0xff80ff80u : 0xff800000u;
  const bool full = t0 + T::N <= end;
#pragma unroll
  for (int i = 0; i < U; ++i) {
    const int64_t slot = OWN ? (int64_t)threadIdx.x * U + i : (int64_t)i * kThreads + threadIdx.x;
    const int64_t e = t0 + slot * T::VW;
    const bool ok = full || e < end;
    const int64_t ec = ok ? e : t0;  // a valid address; the value is discarded
    const char* a = row + ec * T::EB;
    if constexpr (VEC) {
      const u32x4* src = reinterpret_cast<const u32x4*>(a);
      const u32x4 v = NT ? __builtin_nontemporal_load(src) : *src;
      w[i][0] = ok ? v.x : kPad;
      w[i][1] = ok ? v.y : kPad;
      w[i][2] = ok ? v.z : kPad;
      w[i][3] = ok ? v.w : kPad;
    } else if constexpr (DT == 1) {
      const uint32_t v = *reinterpret_cast<const uint16_t*>(a);
      w[i][0] = ok ? v : kPad;
    } else {
      const uint32_t v = *reinterpret_cast<const uint32_t*>(a);
      w[i][0] = ok ? v : kPad;
    }
  }
}

// Entry index of lane load i, element e of this thread (layout as load_tile).
template <int DT, bool VEC, int U, bool OWN>
__device__ __forceinline__ int64_t entry_of(int64_t t0, int i, int e) {
  using T = Tile<DT, VEC, U>;
  const int64_t slot = OWN ? (int64_t)threadIdx.x * U + i : (int64_t)i * kThreads + threadIdx.x;
  return t0 + slot * T::VW + e;
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// ------------------------------------------- cross-workgroup communication
// Agent-scope fences on gfx950 write back and invalidate the whole L2, which
// is ruinous when thousands of workgroups each publish a few bytes.  Instead,
// data shared between workgroups of one launch is written and read with
// agent-scope relaxed atomics (write-through / read-through the L2), and the
// order "data, then counter" is enforced by waiting for the stores to
// complete before the counter update (and the counter read before the data
// reads).  Data from an earlier kernel needs nothing: the kernel boundary
// orders it.
__device__ __forceinline__ void st_dev_f64(double* dst, double v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(dst), (uint64_t)__double_as_longlong(v),
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
// Inclusive prefix sum over a wavefront's lanes (fp64, fixed order).
__device__ __forceinline__ double wave_incl_scan(double v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double n = __shfl_up(v, o, 64);
    if (lane >= o) v += n;
  }
  return v;
}

struct PickState {
  int k;        // tile holding the sample
  int kind;     // SampleKind actually sampled
  double rem;   // target mass remaining at the start of that tile
};

constexpr int kPickLds = 256;  // tile masses kept in LDS by the sampler

struct Shared {
  float m[4][2];
  double d[4][2];
  int i[4][2];
  double scan[4];
  int flag;
};

// Per-sequence state built by every sampling workgroup.
struct SeqShared {
  RowStat rows[SPC_MAX_GAMMA + 1];
  SeqState seq;
  PickState pk;
  double mass[kPickLds];
};

// All threads receive the block-wide max of (a, b).
__device__ __forceinline__ void block_max2(float& a, float& b, Shared& sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  a = wave_max(a);
  b = wave_max(b);
  __syncthreads();  // sh.m may still be read by an earlier step
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
  __syncthreads();
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
  v = wave_incl_scan(v);
  __syncthreads();
  if (lane == 63) sh.scan[wv] = v;
  __syncthreads();
  double off = 0.0;
  for (int w = 0; w < wv; ++w) off += sh.scan[w];
  *total = ((sh.scan[0] + sh.scan[1]) + sh.scan[2]) + sh.scan[3];
  return off + v;
}

// "Am I the last of `n` arrivals?" for the whole block.  Thread 0 wrote the
// data it shares with st_dev_* before the call; on true, the counter is reset
// and the block reads the other arrivals' data with ld_dev_*.
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

// ------------------------------------------------------ per-sequence params
struct SeqParam {
  int rule;
  double alpha;
  double c;         // log2(e) / T  (T = 1 for greedy statistics)
  float c_hi, c_lo; // c = c_hi + c_lo with c_hi < c, c_lo > 0 (float32 pair)
  bool greedy;
  bool valid;
};

__device__ __forceinline__ SeqParam seq_param(const Params& P, int b) {
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

template <int KIND>
__device__ __forceinline__ float weight_of(float zq, float zp, const ProbScale& s) {
  if constexpr (KIND == kQ) return prob(zq, s.c_hi, s.c_lo, s.q_hi, s.q_lo);
  else if constexpr (KIND == kP) return prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
  else return residual_weight(zq, zp, s);
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

// ------------------------------------------------------------- row merge
// One wavefront merges the nt tile partials of row r (fixed order: lanes take
// tiles lane, lane+64, ...; a butterfly combines the lanes), adding the TV
// partials when `tv`.  Every lane returns the same RowStat.
__device__ __forceinline__ RowStat merge_row(const Params& P, int r, bool greedy, bool tv) {
  const int lane = threadIdx.x & 63;
  const int nt = P.nt;
  const TilePart* t = P.tiles + (int64_t)r * nt;
  float zq = kNegInf, zp = kNegInf, rq = kNegInf, rp = kNegInf;
  for (int k = lane; k < nt; k += 64) {
    zq = fmaxf(zq, t[k].zmax_q);
    zp = fmaxf(zp, t[k].zmax_p);
    rq = fmaxf(rq, t[k].r_q);
    rp = fmaxf(rp, t[k].r_p);
  }
  zq = wave_max(zq);
  zp = wave_max(zp);
  rq = wave_max(rq);
  rp = wave_max(rp);
  double sq = 0.0, sp = 0.0, tvs = 0.0;
  int aq = 0x7fffffff, ap = 0x7fffffff;
  for (int k = lane; k < nt; k += 64) {
    const TilePart tk = t[k];
    if (tk.r_q != kNegInf) sq += tk.s_q * exp2((double)tk.r_q - (double)rq);
    if (tk.r_p != kNegInf) sp += tk.s_p * exp2((double)tk.r_p - (double)rp);
    if (greedy) {
      if (tk.zmax_q == zq) aq = min(aq, tk.amax_q);
      if (tk.zmax_p == zp) ap = min(ap, tk.amax_p);
    }
    if (tv) tvs += P.tvpart[(int64_t)r * nt + k];
  }
  sq = wave_sum(sq);
  sp = wave_sum(sp);
  tvs = wave_sum(tvs);
  aq = wave_min(aq);
  ap = wave_min(ap);
  RowStat rs;
  rs.lz_q = (double)rq + log2(sq);
  rs.lz_p = (double)rp + log2(sp);
  rs.tv = tvs;
  rs.zmax_q = zq;
  rs.zmax_p = zp;
  rs.amax_q = greedy ? aq : -1;
  rs.amax_p = greedy ? ap : -1;
  return rs;
}

// ------------------------------------------------------------- decision
// Wave 0: delta_j and the accept draws of one sequence from its merged rows,
// j* (first-rejection search by one ballot), and the sampling state.  With
// `write`, also the outputs that follow (every sampling workgroup of the
// sequence computes the same decision; one writes it).
template <int DT>
__device__ __forceinline__ void decide(const Params& P, int b, const SeqParam& sp,
                                       SeqShared& ss, bool write) {
  const int lane = threadIdx.x;
  const int gamma = P.gamma, g1 = gamma + 1;
  const bool on = lane < g1;
  const int64_t row = (int64_t)b * g1 + lane;
  if (!sp.valid) {
    if (write) {
      if (on) P.out_defer[row] = 0;
      if (lane == 0) {
        P.out_accept[b] = -1;
        P.out_token[b] = -1;
        if (P.out_norm) P.out_norm[b] = 0.0f;
      }
    }
    if (lane == 0) ss.seq = SeqState{-1, kNone, 0.0f, 0};
    return;
  }
  int delta = 0, keep = 1;
  RowStat rs{};
  if (on) {
    rs = ss.rows[lane];
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
    if (write) {
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
  }
  const unsigned long long rej = __ballot(on && !keep);
  const int jstar = __ffsll(rej) - 1;  // bit gamma is always set
  const int dstar = __shfl(delta, jstar, 64);
  const int aq = __shfl(rs.amax_q, jstar, 64);
  const int ap = __shfl(rs.amax_p, jstar, 64);
  if (lane == 0) {
    SeqState s{jstar, kNone, 0.0f, 0};
    if (sp.greedy) {
      if (write) {
        P.out_token[b] = dstar ? ap : aq;
        if (P.out_norm) P.out_norm[b] = 1.0f;
      }
    } else {
      // a rejection with delta = 0 only happens for an out-of-range draft;
      // its residual max(0, q - q) is empty, so p is sampled instead
      s.kind = (jstar < gamma) ? (dstar ? kResidual : kP) : (dstar ? kP : kQ);
      s.u = P.uniforms[(int64_t)b * g1 + gamma];
    }
    if (write) P.out_accept[b] = jstar;
    ss.seq = s;
  }
}

// Whole block: merge the rows of sequence b into ss.rows and decide it.
template <int DT>
__device__ __forceinline__ void merge_and_decide(const Params& P, int b, const SeqParam& sp,
                                                 SeqShared& ss, bool write) {
  const int wv = threadIdx.x >> 6, g1 = P.gamma + 1;
  const bool tv = needs_tv(sp);
  if (sp.valid) {
    for (int j = wv; j < g1; j += kThreads / 64) {
      const RowStat rs = merge_row(P, b * g1 + j, sp.greedy, tv);
      if ((threadIdx.x & 63) == 0) ss.rows[j] = rs;
    }
  }
  __syncthreads();
  if (threadIdx.x < 64) decide<DT>(P, b, sp, ss, write);
  __syncthreads();
}

// ------------------------------------------------------------- sampling
// Whole block: the mass of sampling tile k of a row under the sampled
// distribution (valid in every thread).
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ double block_tile_mass(const char* qrow, const char* prow, int V,
                                                  int k, const ProbScale& ps, Shared& sh) {
  using T = SampTile<DT, VEC>;
  const int64_t t0 = (int64_t)k * T::N;
  uint32_t wq[T::U][T::NW] = {}, wp[T::U][T::NW] = {};
  if (KIND != kP) load_tile<DT, VEC, T::U, false, false>(qrow, t0, V, wq);
  if (KIND != kQ) load_tile<DT, VEC, T::U, false, false>(prow, t0, V, wp);
  double acc = 0.0;
#pragma unroll
  for (int i = 0; i < T::U; ++i) {
    float t = 0.0f;
#pragma unroll
    for (int e = 0; e < T::VW; ++e)
      t += weight_of<KIND>(elem<DT, VEC>(wq[i], e), elem<DT, VEC>(wp[i], e), ps);
    acc += (double)t;
  }
  double unused = 0.0;
  block_sum2(acc, unused, sh);
  return acc;
}

// The in-tile part of the draw: each thread takes U consecutive lane loads of
// tile pk.k, one block-wide scan of the per-thread masses finds the thread,
// and that thread walks its entries.
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ void pick_in_tile(const Params& P, int b, int row, const PickState& pk,
                                             const ProbScale& ps, Shared& sh) {
  using T = SampTile<DT, VEC>;
  const int tid = threadIdx.x;
  const int V = P.V;
  const char* qrow = (const char*)P.q + (int64_t)row * V * T::EB;
  const char* prow = (const char*)P.p + (int64_t)row * V * T::EB;
  const int64_t t0 = (int64_t)pk.k * T::N;
  uint32_t wq[T::U][T::NW] = {}, wp[T::U][T::NW] = {};
  if (KIND != kP) load_tile<DT, VEC, T::U, true, false>(qrow, t0, V, wq);
  if (KIND != kQ) load_tile<DT, VEC, T::U, true, false>(prow, t0, V, wp);
  // per lane-load masses, in entry order
  double slot_mass[T::U];
  double tsum = 0.0;
  int last_pos = -1;
#pragma unroll
  for (int i = 0; i < T::U; ++i) {
    double m = 0.0;
#pragma unroll
    for (int e = 0; e < T::VW; ++e) {
      const float w = weight_of<KIND>(elem<DT, VEC>(wq[i], e), elem<DT, VEC>(wp[i], e), ps);
      m += (double)w;
      if (w > 0.0f) last_pos = (int)entry_of<DT, VEC, T::U, true>(t0, i, e);
    }
    slot_mass[i] = m;
    tsum += m;
  }
  double total;
  const double incl = block_incl_scan(tsum, sh, &total);
  if (total > pk.rem) {  // block-uniform
    int cand = (incl > pk.rem) ? tid : 0x7fffffff, unused = 0;
    block_min2(cand, unused, sh);
    if (tid == cand) {
      // the lane load where the running mass crosses, then its entries
      double run = incl - tsum, before = 0.0;
      int islot = -1;
#pragma unroll
      for (int i = 0; i < T::U; ++i) {
        if (islot < 0 && run + slot_mass[i] > pk.rem) {
          islot = i;
          before = run;
        }
        run += slot_mass[i];
      }
      int hit = -1;
      if (islot >= 0) {
        uint32_t sq[T::NW] = {}, sp_[T::NW] = {};
#pragma unroll
        for (int i = 0; i < T::U; ++i)
          if (i == islot)
#pragma unroll
            for (int j = 0; j < T::NW; ++j) {
              sq[j] = wq[i][j];
              sp_[j] = wp[i][j];
            }
        run = before;
        int lastw = -1;
        const int64_t base = entry_of<DT, VEC, T::U, true>(t0, islot, 0);
#pragma unroll
        for (int e = 0; e < T::VW; ++e) {
          const float w = weight_of<KIND>(elem<DT, VEC>(sq, e), elem<DT, VEC>(sp_, e), ps);
          run += (double)w;
          if (w > 0.0f) lastw = (int)(base + e);
          if (hit < 0 && run > pk.rem && w > 0.0f) hit = (int)(base + e);
        }
        if (hit < 0) hit = lastw;  // rounding inside the lane load
      }
      // rounding inside the thread: its last entry with mass
      P.out_token[b] = hit >= 0 ? hit : last_pos;
    }
    return;
  }
  // rounding: no thread reached u*W; take the last entry of the tile with mass
  int lp = -last_pos, unused = 0;
  block_min2(lp, unused, sh);
  if (tid == 0) P.out_token[b] = -lp;
}

// Wave 0 gathers the K tile masses of sequence b (into LDS when they fit);
// returns their total W to the whole block.
__device__ __forceinline__ double gather_masses(const Params& P, int b, SeqShared& ss,
                                                Shared& sh) {
  const int lane = threadIdx.x & 63, K = P.K;
  __syncthreads();
  if (threadIdx.x < 64) {
    double W = 0.0;
    for (int k0 = 0; k0 < K; k0 += 64) {
      const int k = k0 + lane;
      const double m = (k < K) ? ld_dev_f64(P.masses + (int64_t)b * K + k) : 0.0;
      if (k < K && k < kPickLds) ss.mass[k] = m;
      W += wave_sum(m);
    }
    if (lane == 0) sh.d[0][0] = W;
  }
  __syncthreads();
  return sh.d[0][0];
}

// Whole block: inverse-CDF draw at row j* of sequence b -- the smallest entry
// k with C_k > u * W, C the running mass in vocabulary order and W the total.
// Wave 0 scans the tile masses (64 at a time) to find the tile, then
// pick_in_tile finds the entry.
template <int DT, bool VEC>
__device__ __forceinline__ void pick(const Params& P, int b, const SeqParam& sp, SeqShared& ss,
                                     Shared& sh) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int K = P.K;
  const SeqState s = ss.seq;
  const int row = b * (P.gamma + 1) + s.row;
  const ProbScale ps = prob_scale(sp, ss.rows[s.row]);
  int kind = s.kind;
  double W = gather_masses(P, b, ss, sh);
  if (kind == kResidual && !(W > 0.0)) {
    // empty residual (possible only through rounding): sample p instead
    kind = kP;
    const int V = P.V;
    const char* qrow = (const char*)P.q + (int64_t)row * V * SampTile<DT, VEC>::EB;
    const char* prow = (const char*)P.p + (int64_t)row * V * SampTile<DT, VEC>::EB;
    for (int k = 0; k < K; ++k) {
      const double m = block_tile_mass<DT, VEC, kP>(qrow, prow, V, k, ps, sh);
      if (tid == 0) st_dev_f64(P.masses + (int64_t)b * K + k, m);
    }
    if (tid == 0) vmem_drain();
    W = gather_masses(P, b, ss, sh);
  }
  if (tid < 64) {
    const double target = (double)s.u * W;
    double carry = 0.0, rem = 0.0;
    int ks = -1, klast = -1;
    for (int k0 = 0; k0 < K; k0 += 64) {
      const int k = k0 + lane;
      const double m = (k >= K) ? 0.0
                       : (k < kPickLds) ? ss.mass[k] : ld_dev_f64(P.masses + (int64_t)b * K + k);
      const double incl = carry + wave_incl_scan(m);
      const unsigned long long pos = __ballot(m > 0.0);
      const unsigned long long hit = __ballot(m > 0.0 && incl > target);
      if (pos) klast = k0 + 63 - __clzll(pos);
      if (ks < 0 && hit) {
        const int l = __ffsll(hit) - 1;
        ks = k0 + l;
        rem = target - (__shfl(incl, l, 64) - __shfl(m, l, 64));
      }
      carry = __shfl(incl, 63, 64);
    }
    if (ks < 0) {  // rounding left u*W at or past the end: last entry with mass
      ks = klast;
      rem = __builtin_huge_val();
    }
    if (lane == 0) {
      ss.pk = PickState{ks, kind, rem};
      if (P.out_norm) P.out_norm[b] = (float)W;
    }
  }
  __syncthreads();
  const PickState pk = ss.pk;
  if (pk.k < 0) {
    if (tid == 0) P.out_token[b] = -1;
    return;
  }
  if (pk.kind == kQ) pick_in_tile<DT, VEC, kQ>(P, b, row, pk, ps, sh);
  else if (pk.kind == kP) pick_in_tile<DT, VEC, kP>(P, b, row, pk, ps, sh);
  else pick_in_tile<DT, VEC, kResidual>(P, b, row, pk, ps, sh);
}

// ================================================================ kernels

// Statistics pass.  grid (nt, R): stats tile k of row r.  Each thread takes
// the exact max of its entries and the sum of 2^(z c - r_t), r_t = max * c_hi
// (a reference near its largest z c); the block combines the threads against
// the tile max.  With ARGMAX (batches that may hold greedy rows) the lowest
// entry attaining the max is found as well.
template <int DT, bool VEC, bool ARGMAX>
__global__ __launch_bounds__(kThreads) void k_stats(Params P) {
  using T = StatTile<DT, VEC>;
  __shared__ Shared sh;
  const int k = blockIdx.x, r = blockIdx.y;
  const SeqParam sp = seq_param(P, r / (P.gamma + 1));
  const int V = P.V;
  const char* qrow = (const char*)P.q + (int64_t)r * V * T::EB;
  const char* prow = (const char*)P.p + (int64_t)r * V * T::EB;
  const int64_t t0 = (int64_t)k * T::N;
  uint32_t wq[T::U][T::NW], wp[T::U][T::NW];
  load_tile<DT, VEC, T::U, false, true>(qrow, t0, V, wq);
  load_tile<DT, VEC, T::U, false, true>(prow, t0, V, wp);

  float mq = kNegInf, mp = kNegInf;
#pragma unroll
  for (int i = 0; i < T::U; ++i)
#pragma unroll
    for (int e = 0; e < T::VW; ++e) {
      mq = fmaxf(mq, elem<DT, VEC>(wq[i], e));
      mp = fmaxf(mp, elem<DT, VEC>(wp[i], e));
    }
  int iq = 0x7fffffff, ip = 0x7fffffff;
  if constexpr (ARGMAX) {
    // entries are visited in increasing index order: the first match wins
#pragma unroll
    for (int i = 0; i < T::U; ++i)
#pragma unroll
      for (int e = 0; e < T::VW; ++e) {
        const int idx = (int)entry_of<DT, VEC, T::U, false>(t0, i, e);
        if (iq == 0x7fffffff && elem<DT, VEC>(wq[i], e) == mq) iq = idx;
        if (ip == 0x7fffffff && elem<DT, VEC>(wp[i], e) == mp) ip = idx;
      }
  }
  const float rq = (mq == kNegInf) ? 0.0f : mq * sp.c_hi;
  const float rp = (mp == kNegInf) ? 0.0f : mp * sp.c_hi;
  float sq = 0.0f, spp = 0.0f;
#pragma unroll
  for (int i = 0; i < T::U; ++i) {
    float tq[T::VW], tp[T::VW];
#pragma unroll
    for (int e = 0; e < T::VW; ++e) {
      const float zq = elem<DT, VEC>(wq[i], e), zp = elem<DT, VEC>(wp[i], e);
      tq[e] = exp2_hw(fmaf(zq, sp.c_lo, fmaf(zq, sp.c_hi, -rq)));
      tp[e] = exp2_hw(fmaf(zp, sp.c_lo, fmaf(zp, sp.c_hi, -rp)));
    }
#pragma unroll
    for (int h = 1; h < T::VW; h <<= 1)
#pragma unroll
      for (int e = 0; e + h < T::VW; e += 2 * h) {
        tq[e] += tq[e + h];
        tp[e] += tp[e + h];
      }
    sq += tq[0];
    spp += tp[0];
  }
  float Mq = mq, Mp = mp;
  block_max2(Mq, Mp, sh);
  const float Rq = Mq * sp.c_hi, Rp = Mp * sp.c_hi;
  double dq = (mq == kNegInf) ? 0.0 : (double)sq * (double)exp2_hw(rq - Rq);
  double dp = (mp == kNegInf) ? 0.0 : (double)spp * (double)exp2_hw(rp - Rp);
  block_sum2(dq, dp, sh);
  if constexpr (ARGMAX) {
    iq = (mq == Mq) ? iq : 0x7fffffff;
    ip = (mp == Mp) ? ip : 0x7fffffff;
    block_min2(iq, ip, sh);
  }
  if (threadIdx.x == 0) {
    TilePart t;
    t.s_q = dq;
    t.s_p = dp;
    t.r_q = (Mq == kNegInf) ? kNegInf : Rq;
    t.r_p = (Mp == kNegInf) ? kNegInf : Rp;
    t.zmax_q = Mq;
    t.zmax_p = Mp;
    t.amax_q = ARGMAX ? iq : -1;
    t.amax_p = ARGMAX ? ip : -1;
    P.tiles[(int64_t)r * P.nt + k] = t;
  }
}

// TV pass (OPT rows at temperature > 0): D_TV(p, q) of Lemma 3, which needs
// both normalisers.  grid (nt, R): stats tile k of row r; wave 0 merges the
// row's statistics first (a fixed-order computation every tile of the row
// repeats identically).
template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void k_tv(Params P) {
  using T = StatTile<DT, VEC>;
  __shared__ Shared sh;
  __shared__ RowStat srow;
  const int k = blockIdx.x, r = blockIdx.y;
  const SeqParam sp = seq_param(P, r / (P.gamma + 1));
  if (!needs_tv(sp)) return;  // block-uniform
  const int V = P.V;
  const char* qrow = (const char*)P.q + (int64_t)r * V * T::EB;
  const char* prow = (const char*)P.p + (int64_t)r * V * T::EB;
  const int64_t t0 = (int64_t)k * T::N;
  uint32_t wq[T::U][T::NW], wp[T::U][T::NW];
  load_tile<DT, VEC, T::U, false, true>(qrow, t0, V, wq);
  load_tile<DT, VEC, T::U, false, true>(prow, t0, V, wp);
  if (threadIdx.x < 64) {
    const RowStat rs = merge_row(P, r, false, false);
    if (threadIdx.x == 0) srow = rs;
  }
  __syncthreads();
  const ProbScale ps = prob_scale(sp, srow);
  double acc = 0.0;
#pragma unroll
  for (int i = 0; i < T::U; ++i) {
    float t = 0.0f;
#pragma unroll
    for (int e = 0; e < T::VW; ++e)
      t += residual_weight(elem<DT, VEC>(wq[i], e), elem<DT, VEC>(wp[i], e), ps);
    acc += (double)t;
  }
  double unused = 0.0;
  block_sum2(acc, unused, sh);
  if (threadIdx.x == 0) P.tvpart[(int64_t)r * P.nt + k] = acc;
}

// Sampling pass.  grid (K, B): every workgroup of sequence b merges the
// sequence's rows and decides it (workgroup 0 writes the outputs); sampling
// tile k of row j* then computes its mass and the last tile to finish draws.
template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void k_sample(Params P) {
  __shared__ Shared sh;
  __shared__ SeqShared ss;
  const int k = blockIdx.x, b = blockIdx.y;
  const SeqParam sp = seq_param(P, b);
  merge_and_decide<DT>(P, b, sp, ss, k == 0);
  const SeqState s = ss.seq;
  if (s.kind == kNone) return;  // block-uniform
  const int row = b * (P.gamma + 1) + s.row;
  const ProbScale ps = prob_scale(sp, ss.rows[s.row]);
  const int V = P.V;
  constexpr int EB = SampTile<DT, VEC>::EB;
  const char* qrow = (const char*)P.q + (int64_t)row * V * EB;
  const char* prow = (const char*)P.p + (int64_t)row * V * EB;
  double m;
  if (s.kind == kQ) m = block_tile_mass<DT, VEC, kQ>(qrow, prow, V, k, ps, sh);
  else if (s.kind == kP) m = block_tile_mass<DT, VEC, kP>(qrow, prow, V, k, ps, sh);
  else m = block_tile_mass<DT, VEC, kResidual>(qrow, prow, V, k, ps, sh);
  if (threadIdx.x == 0) st_dev_f64(P.masses + (int64_t)b * P.K + k, m);
  if (!arrive_last(P.samp_cnt + b, (uint32_t)P.K, sh)) return;
  pick<DT, VEC>(P, b, sp, ss, sh);
}

template <int DT, bool VEC>
hipError_t launch_t(const Params& P, bool need_tv, bool need_sample, bool need_argmax,
                    hipEvent_t e0, hipEvent_t e1, hipStream_t st) {
  const unsigned R = (unsigned)(P.B * (P.gamma + 1));
  hipError_t err;
  if (e0 && (err = hipEventRecord(e0, st)) != hipSuccess) return err;
  if (need_argmax)
    hipLaunchKernelGGL((k_stats<DT, VEC, true>), dim3(P.nt, R), dim3(kThreads), 0, st, P);
  else
    hipLaunchKernelGGL((k_stats<DT, VEC, false>), dim3(P.nt, R), dim3(kThreads), 0, st, P);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  if (e1 && (err = hipEventRecord(e1, st)) != hipSuccess) return err;
  if (need_tv) {
    hipLaunchKernelGGL((k_tv<DT, VEC>), dim3(P.nt, R), dim3(kThreads), 0, st, P);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  // a batch with no sequence at temperature > 0 only needs the decisions
  hipLaunchKernelGGL((k_sample<DT, VEC>), dim3(need_sample ? P.K : 1, P.B), dim3(kThreads), 0,
                     st, P);
  return hipGetLastError();
}

}  // namespace

int stat_tile_elems(int dtype, bool vec) {
  if (dtype == 1) return vec ? StatTile<1, true>::N : StatTile<1, false>::N;
  return vec ? StatTile<0, true>::N : StatTile<0, false>::N;
}

int samp_tile_elems(int dtype, bool vec) {
  if (dtype == 1) return vec ? SampTile<1, true>::N : SampTile<1, false>::N;
  return vec ? SampTile<0, true>::N : SampTile<0, false>::N;
}

hipError_t launch_verify(const Params& P, int dtype, bool vec, bool need_tv, bool need_sample,
                         bool need_argmax, hipEvent_t e0, hipEvent_t e1, hipStream_t st) {
  if (dtype == 1) {
    return vec ? launch_t<1, true>(P, need_tv, need_sample, need_argmax, e0, e1, st)
               : launch_t<1, false>(P, need_tv, need_sample, need_argmax, e0, e1, st);
  }
  return vec ? launch_t<0, true>(P, need_tv, need_sample, need_argmax, e0, e1, st)
             : launch_t<0, false>(P, need_tv, need_sample, need_argmax, e0, e1, st);
}

}  // namespace spc
