// spc_kernels.hip -- gfx950 kernels of the speculative-cascade verify step.
//
// The step (GenSpecSample, Alg. 4, with the cascade target T_delta of eq. (6)
// and the deferral rules of Table 1) runs as two or three kernels.  A row is
// one position (b, j) of the logit pair (q, p); rows are cut into tiles of
// consecutive vocabulary entries.
//
//   k_stats   grid (tiles per row, rows), one tile per 256-thread workgroup.
//             Reads every logit of q and p once and reduces the tile to
//             {max z, sum 2^(z c - r), argmax} for both tensors
//             (c = log2(e) / T); the tile partial goes to the workspace.
//   k_tv      OPT sequences at temperature > 0 only: D_TV(p, q) of Lemma 3
//             needs both normalisers, so it is a second pass over those rows,
//             one partial per tile.
//   k_sample  grid (K, sequences), 1024-thread workgroups.  Every workgroup
//             of sequence b merges that sequence's row partials and takes the
//             per-sequence decision (deferral delta_j, accept draws a_j, first
//             rejection j*) -- a small, fixed-order computation, so every
//             workgroup reaches the same result.  A replacement from the
//             residual max(0, p - q) of a non-OPT row needs a second look at
//             row j*: the K workgroups sum its residual per chunk and the last
//             to finish draws.  Every other draw takes its per-tile masses
//             from the statistics or TV partials and is made by workgroup 0.
//             Draws are inverse CDF in vocabulary order.
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

constexpr int kWaves = kThreads / 64;
// The sampling pass runs 1024-thread workgroups: a wavefront per row while
// deciding, a 256-thread group per tile while summing residual masses.
constexpr int kSampThreads = 1024;
constexpr int kSampWaves = kSampThreads / 64;

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
using StatTile = Tile<DT, VEC, VEC ? 4 : 8>;

// drafter tiles: one tensor, M times the lane loads of a statistics tile
// (M = 2: the same bytes per workgroup, for large batches; M = 1: twice the
// workgroups, for small ones)
template <int DT, bool VEC, int M>
using DraftTile = Tile<DT, VEC, M * StatTile<DT, VEC>::U>;

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

// Lane loads of one tile of one row into w[U][NW] by the GT threads of a
// group, tid the thread's index in it.  Thread t's lane load i covers entries
// e = t0 + (i*GT + t) * VW .. + VW - 1 (interleaved, so each load
// instruction of a wavefront reads one contiguous 1 KiB).
// Entries at or past `end` read as -inf; a lane past the end re-reads a valid
// address and discards the value, so the loads are branch-free.  With MASK
// false the caller guarantees a whole tile before `end`.
template <int DT, bool VEC, int U, bool NT, int GT = kThreads, bool MASK = true>
__device__ __forceinline__ void load_tile(const char* row, int64_t t0, int64_t end,
                                          uint32_t (&w)[U][Tile<DT, VEC, U>::NW], int tid) {
  using T = Tile<DT, VEC, U>;
  constexpr uint32_t kPad = (DT == 1) ? 0xff80ff80u : 0xff800000u;
  const bool full = !MASK || t0 + (int64_t)GT * U * T::VW <= end;
#pragma unroll
  for (int i = 0; i < U; ++i) {
    const int64_t slot = (int64_t)i * GT + tid;
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

// The lowest entry attaining m among a thread's U lane loads w (lane load i
// holds entries base + i * GT * VW + e, e < VW), given each lane load's
// maximum g[i]: the first lane load whose maximum is m, then the first entry
// of it equal to m.  INT_MAX when m = -inf (no finite entry).
template <int DT, bool VEC, int U, int GT>
__device__ __forceinline__ int first_max_index(const uint32_t (&w)[U][Tile<DT, VEC, U>::NW],
                                               const float (&g)[U], float m, int base) {
  using T = Tile<DT, VEC, U>;
  int gi = 0;
#pragma unroll
  for (int i = U - 1; i >= 0; --i)
    if (g[i] == m) gi = i;
  uint32_t s[T::NW];
#pragma unroll
  for (int j = 0; j < T::NW; ++j) s[j] = w[0][j];
#pragma unroll
  for (int i = 1; i < U; ++i)
#pragma unroll
    for (int j = 0; j < T::NW; ++j) s[j] = (gi == i) ? w[i][j] : s[j];
  int ei = 0;
#pragma unroll
  for (int e = T::VW - 1; e >= 0; --e)
    if (elem<DT, VEC>(s, e) == m) ei = e;
  return m == kNegInf ? 0x7fffffff : base + gi * GT * T::VW + ei;
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float log2_hw(float x) { return __builtin_amdgcn_logf(x); }

// 2^d in fp64 by exact argument reduction, d = n + f with n = floor(d) and
// f in [0, 1), and the hardware 2^f: relative error about one float32 ulp.
// Arguments below -1022 give 0.
__device__ __forceinline__ double exp2_acc(double d) {
  if (d < -1022.0) return 0.0;
  const double n = floor(d);
  return ldexp((double)exp2_hw((float)(d - n)), (int)n);
}

// log2 of a positive finite fp64 value: S = m 2^e with m in [1/sqrt(2),
// sqrt(2)), m = head + tail with a float32 head, log2(m) = log2(head) +
// tail / (head ln 2): absolute error about one float32 ulp of |log2 m| <= 1/2.
__device__ __forceinline__ double log2_acc(double S) {
  int e;
  double m = frexp(S, &e);
  if (m < 0.70710678118654752) {
    m *= 2.0;
    --e;
  }
  const float mh = (float)m;
  const double tail = m - (double)mh;
  return (double)e + (double)log2_hw(mh) + tail * (double)__builtin_amdgcn_rcpf(mh) * kLog2e;
}

// First moments h = sum 2^a a (a = z c - r) moved from reference r to a
// reference r' >= r: with d = r - r' (exact in fp64) and f = 2^d, every weight
// scales by f and every argument grows by d, so h' = f (h + d s), s the sum
// of the weights.  For x = sum 2^(a_q) a_p, f is the q factor and d the p
// shift.  An empty side (s = 0) stays 0 and a -inf moment stays -inf.
// Floating-point contraction is off here and in mom_add, so that the q and
// p moments of identical rows take identical operations at every call site
// (H(q) - H(p) is then exactly 0 for p = q).
__device__ __forceinline__ double mom_move(double h, double s, double f, double d) {
#pragma clang fp contract(off)
  if (s == 0.0) return 0.0;
  if (h == -__builtin_huge_val()) return h;
  return f * (h + d * s);
}
__device__ __forceinline__ void mom_add(double& acc, double h, double s, double f, double d) {
#pragma clang fp contract(off)
  acc = acc + mom_move(h, s, f, d);
}

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

// A tile partial written and read within one launch: five 64-bit words with
// agent-scope atomics.
static_assert(sizeof(TilePart) == 40, "TilePart is five 64-bit words");
__device__ __forceinline__ void st_tile(TilePart* dst, const TilePart& t) {
  uint64_t w[5];
  __builtin_memcpy(w, &t, sizeof w);
#pragma unroll
  for (int i = 0; i < 5; ++i)
    __hip_atomic_store(reinterpret_cast<uint64_t*>(dst) + i, w[i], __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ TilePart ld_tile(const TilePart* src) {
  uint64_t w[5];
#pragma unroll
  for (int i = 0; i < 5; ++i)
    w[i] = __hip_atomic_load(reinterpret_cast<uint64_t*>(const_cast<TilePart*>(src)) + i,
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  TilePart t;
  __builtin_memcpy(&t, w, sizeof w);
  return t;
}

// Every vector-memory operation issued so far by this wave has completed.
__device__ __forceinline__ void vmem_drain() {
  __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xf << 8));  // vmcnt(0)
}

// ------------------------------------------------------- wavefront reductions
// DPP row operations combine the lanes of each 16-lane row without going
// through LDS; readlane then brings the four row results to every lane in a
// fixed order, so every lane (and every run) gets the same value.  All 64
// lanes must be active.
constexpr int kDppXor1 = 0xb1;         // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4e;         // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror
constexpr int kDppMirror = 0x140;      // row_mirror
constexpr int kDppShr = 0x110;         // row_shr:n is kDppShr + n

// Lanes with no source lane (row_shr at the start of a row) read 0.
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(dpp_i32<CTRL>(__float_as_int(v)));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const int lo = dpp_i32<CTRL>(__double2loint(v));
  const int hi = dpp_i32<CTRL>(__double2hiint(v));
  return __hiloint2double(hi, lo);
}

// Value of lane l (l uniform across the wave).
__device__ __forceinline__ int lane_i32(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ float lane_f32(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ double lane_f64(double v, int l) {
  return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(v), l),
                          __builtin_amdgcn_readlane(__double2loint(v), l));
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f32<kDppXor1>(v));
  v = fmaxf(v, dpp_f32<kDppXor2>(v));
  v = fmaxf(v, dpp_f32<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f32<kDppMirror>(v));
  return fmaxf(fmaxf(lane_f32(v, 0), lane_f32(v, 16)), fmaxf(lane_f32(v, 32), lane_f32(v, 48)));
}
__device__ __forceinline__ double wave_sum(double v) {
  v += dpp_f64<kDppXor1>(v);
  v += dpp_f64<kDppXor2>(v);
  v += dpp_f64<kDppHalfMirror>(v);
  v += dpp_f64<kDppMirror>(v);
  return (lane_f64(v, 0) + lane_f64(v, 16)) + (lane_f64(v, 32) + lane_f64(v, 48));
}
__device__ __forceinline__ int wave_min(int v) {
  v = min(v, dpp_i32<kDppXor1>(v));
  v = min(v, dpp_i32<kDppXor2>(v));
  v = min(v, dpp_i32<kDppHalfMirror>(v));
  v = min(v, dpp_i32<kDppMirror>(v));
  return min(min(lane_i32(v, 0), lane_i32(v, 16)), min(lane_i32(v, 32), lane_i32(v, 48)));
}
// Inclusive prefix sum over a wavefront's lanes (fp64, fixed order): a
// Hillis-Steele scan inside each row, then the earlier rows' totals.
__device__ __forceinline__ double wave_incl_scan(double v) {
  v += dpp_f64<kDppShr + 1>(v);
  v += dpp_f64<kDppShr + 2>(v);
  v += dpp_f64<kDppShr + 4>(v);
  v += dpp_f64<kDppShr + 8>(v);
  const double t0 = lane_f64(v, 15), t1 = lane_f64(v, 31), t2 = lane_f64(v, 47);
  const int row = (threadIdx.x & 63) >> 4;
  const double off = row == 0 ? 0.0 : row == 1 ? t0 : row == 2 ? t0 + t1 : (t0 + t1) + t2;
  return off + v;
}

// Block-wide scratch of a workgroup of NWV wavefronts.
template <int NWV>
struct SharedT {
  static constexpr int kNW = NWV;
  float m[NWV][2];
  double d[NWV][2];
  double dv[64];  // per sub-chunk sums of a tile draw
  double h[NWV][3];
  int i[NWV][2];
  int flag;
};
using Shared = SharedT<kWaves>;
using SampShared = SharedT<kSampWaves>;

// Merged statistics and decision of one row of a sequence.
struct RowDecision {
  RowStat rs;
  float maxq, maxp, tv;  // inputs of the deferral rule
  float u;               // the row's uniform
  int delta, keep;       // delta_j and a_j
};

// Per-sequence state built by every sampling workgroup.
// The part of a draw found by wave 0, for the whole workgroup.
struct PickState {
  int k;       // part holding the sample (-1: nothing to draw)
  int kind;    // SampleKind actually sampled
  int src;     // MassSrc of the part masses
  double rem;  // target mass remaining at the start of that part
};

struct SeqShared {
  RowDecision rows[SPC_MAX_GAMMA + 1];
  SeqState seq;
  PickState pk;
};

// Block sums: per-wave results combined in wave order (a fixed order, so
// every thread and every run gets the same value); valid in every thread.
template <int NWV>
__device__ __forceinline__ void block_sum2(double& a, double& b, SharedT<NWV>& sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  a = wave_sum(a);
  b = wave_sum(b);
  __syncthreads();
  if (lane == 0) { sh.d[wv][0] = a; sh.d[wv][1] = b; }
  __syncthreads();
  a = sh.d[0][0];
  b = sh.d[0][1];
#pragma unroll
  for (int w = 1; w < NWV; ++w) {
    a += sh.d[w][0];
    b += sh.d[w][1];
  }
}

// "Am I the last of `n` arrivals?" for the whole block.  Thread 0 wrote the
// data it shares with st_dev_* before the call; on true, the counter is reset
// and the block reads the other arrivals' data with ld_dev_*.
template <int NWV>
__device__ __forceinline__ bool arrive_last(uint32_t* cnt, uint32_t n, SharedT<NWV>& sh) {
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
  s.valid = s.rule >= SPC_RULE_CHOW && s.rule <= SPC_RULE_OPTLOG && isfinite(alpha) &&
            isfinite(T) && T >= 0.0f && (T == 0.0f || T >= 1e-20f) &&
            (s.rule != SPC_RULE_LOSSY || alpha < 1.0f) &&
            (!P.rule_ps || !P.rule_mask || ((P.rule_mask >> s.rule) & 1u));
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

__device__ __forceinline__ bool is_token(int rule) {
  return rule >= SPC_RULE_TOKEN_V1 && rule <= SPC_RULE_TOKEN_V3;
}

// BiLD* and the log-loss rules of Table 3: delta from a statistic in nats.
__device__ __forceinline__ bool is_log(int rule) {
  return rule >= SPC_RULE_BILD && rule <= SPC_RULE_OPTLOG;
}

// Rules whose deferral reads D_TV (Lemma 3), which the second pass sums.
__device__ __forceinline__ bool has_tv_parts(int rule) {
  return rule == SPC_RULE_OPT || rule == SPC_RULE_OPTLOG;
}

// Sequences whose rows need the second pass: OPT and OPTLOG (D_TV of
// Lemma 3) and the token rules (eta of Alg. 6) at temperature > 0.
__device__ __forceinline__ bool needs_pass2(const SeqParam& s) {
  return s.valid && !s.greedy && (has_tv_parts(s.rule) || is_token(s.rule));
}

// Sequences whose statistics tiles also take first moments: the entropies of
// the log-loss rules (at temperature 0, of the temperature-1 softmax) and
// BiLD*'s cross-entropy at temperature > 0.
__device__ __forceinline__ bool needs_mom(const SeqParam& s) {
  return s.valid && is_log(s.rule) && !(s.rule == SPC_RULE_BILD && s.greedy);
}

// Token-specific rules (Section 4.4) as a threshold on one logit of the row:
// r(v) = 1 iff z(v) < theta, z the drafter's logit for TokenV1 (q(v) <
// max p - alpha) and the verifier's for TokenV2 (p(v) < max p - alpha) and
// TokenV3 (p(v) < max p (1 - alpha)).  theta is solved in fp64 from the row
// statistics and rounded upward to float, so that z < theta in float equals
// the comparison against the fp64 threshold; a threshold at or below zero
// probability gives theta = -inf (r = 0 everywhere).
struct TokenRule {
  float theta;
  bool on_p;
};

// The threshold is written as max p * f, f = 1 - alpha (V3) or
// 1 - alpha / max p (V1, V2), and moved into logit space relative to the
// largest p logit: p(v) < max p f  <=>  z_p(v) < zmax_p + log2(f) / c, and
// for V1 q(v) < max p f  <=>  z_q(v) < zmax_p + (lz_q - lz_p + log2 f) / c.
// Rounding up to float keeps the comparison exact for float logits.  Tokens
// attaining max p (V2, V3) get the exact verdict 1(alpha < 0) whatever the
// rounding of log2 f.
__device__ __forceinline__ TokenRule token_rule(const SeqParam& s, const RowStat& rs,
                                                double maxp) {
  TokenRule t;
  t.on_p = s.rule != SPC_RULE_TOKEN_V1;
  const double f = s.rule == SPC_RULE_TOKEN_V3 ? 1.0 - s.alpha : 1.0 - s.alpha / maxp;
  double th = -__builtin_huge_val();
  if (f > 0.0) {
    const double g = log2(f) + (t.on_p ? 0.0 : rs.lz_q - rs.lz_p);
    th = (double)rs.zmax_p + g / s.c;
  }
  float theta = __double2float_ru(th);
  if (t.on_p) {
    if (s.alpha < 0.0f)
      theta = fmaxf(theta, nextafterf(rs.zmax_p, __builtin_huge_valf()));
    else
      theta = fminf(theta, rs.zmax_p);
  }
  t.theta = theta;
  return t;
}

__device__ __forceinline__ bool token_r(const TokenRule& t, float zq, float zp) {
  return (t.on_p ? zp : zq) < t.theta;
}

// log2 of a normalised probability, evaluated as two float32 halves:
// z*c - lz = (z*c_hi - l_hi) + (z*c_lo - l_lo).
struct ProbScale {
  float c_hi, c_lo, q_hi, q_lo, p_hi, p_lo;
  double c;   // log2(e) / T
  double dl;  // lz_p - lz_q
  TokenRule tok;  // token rules only
};

// With `token` (a token rule's distributions) the p scale carries eta:
// p(v) eta = 2^(z c - (lz_p - log2 eta)), so the weights of Alg. 6's target
// reuse the p-side formulas (eta = 0 leaves every p-side weight at 0).
__device__ __forceinline__ ProbScale prob_scale(const SeqParam& s, const RowStat& rs,
                                                bool token = false) {
  ProbScale ps;
  ps.c_hi = s.c_hi;
  ps.c_lo = s.c_lo;
  ps.q_hi = (float)rs.lz_q;
  ps.q_lo = (float)(rs.lz_q - (double)ps.q_hi);
  ps.c = s.c;
  double lzp = rs.lz_p;
  ps.tok = TokenRule{kNegInf, false};
  if (token) {
    ps.tok = token_rule(s, rs, exp2_acc((double)rs.zmax_p * s.c - rs.lz_p));
    lzp = rs.tv > 0.0 ? rs.lz_p - log2(rs.tv) : __builtin_huge_val();
  }
  ps.p_hi = (float)lzp;
  ps.p_lo = isfinite(lzp) ? (float)(lzp - (double)ps.p_hi) : 0.0f;
  ps.dl = lzp - rs.lz_q;
  return ps;
}

__device__ __forceinline__ float prob(float z, float c_hi, float c_lo, float l_hi, float l_lo) {
  return exp2_hw(fmaf(z, c_hi, -l_hi) + fmaf(z, c_lo, -l_lo));
}

// (2^d - 1) / d for d in [0, 1/4]: a degree-4 polynomial fitted here for
// relative error (4e-10 in exact arithmetic, about one float32 ulp as
// evaluated), so 2^d - 1 keeps full relative precision as d -> 0.
__device__ __forceinline__ float exp2m1_over_d(float d) {
  float r = 0.0014333005528897047f;
  r = fmaf(r, d, 0.009596072137355804f);
  r = fmaf(r, d, 0.05550608038902283f);
  r = fmaf(r, d, 0.24022644758224487f);
  return fmaf(r, d, 0.6931471824645996f);
}

// Residual weight max(0, p_v - q_v), without branches.  d = log2(p_v / q_v) is
// formed in fp64 from the exact difference zp - zq, so p ~ q does not cancel:
// below d = 1/4 the weight is q_v (2^d - 1); above, p_v - q_v itself, where
// p_v > 1.18 q_v bounds the cancellation.  Both -inf gives a NaN d and weight
// 0; zq = -inf alone gives d = +inf and weight p_v.
__device__ __forceinline__ float residual_weight(float zq, float zp, const ProbScale& s) {
  const float d = (float)fma((double)zp - (double)zq, s.c, -s.dl);
  const float pq = prob(zq, s.c_hi, s.c_lo, s.q_hi, s.q_lo);
  const float pp = prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
  float small = pq * (d * exp2m1_over_d(d)), big = pp - pq;
  // both arms stay computed: left alone, the compiler sinks each into a
  // divergent branch, which costs more than evaluating both
  asm volatile("" : "+v"(small), "+v"(big));
  const float w = d < 0.25f ? small : big;
  return d > 0.0f ? w : 0.0f;
}

// Weight of one entry under a sampled distribution.  With a token rule the p
// scale carries eta (prob_scale): the residual max(0, pi - q) of Alg. 6's
// target is p eta where r = 0 and max(0, p eta - q) where r = 1, and the
// target itself is p eta where r = 1 and q + p eta where r = 0.
template <int KIND>
__device__ __forceinline__ float weight_of(float zq, float zp, const ProbScale& s) {
  if constexpr (KIND == kQ) {
    return prob(zq, s.c_hi, s.c_lo, s.q_hi, s.q_lo);
  } else if constexpr (KIND == kP) {
    return prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
  } else if constexpr (KIND == kResidual) {
    return residual_weight(zq, zp, s);
  } else if constexpr (KIND == kTokRes) {
    float res = residual_weight(zq, zp, s), pe = prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
    asm volatile("" : "+v"(res), "+v"(pe));
    return token_r(s.tok, zq, zp) ? res : pe;
  } else {
    const float pe = prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
    const float qe = prob(zq, s.c_hi, s.c_lo, s.q_hi, s.q_lo);
    return token_r(s.tok, zq, zp) ? pe : qe + pe;
  }
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
// The first 64 tile partials of row r (lane l holds tile l) and their TV
// partials: the loads of a merge, issued ahead of it.
struct PartHead {
  TilePart t;
  double tv;
  TileMom m;
};

// Tile partial k of row r; with DEV written earlier in the same launch (read
// with agent-scope loads).
template <bool DEV>
__device__ __forceinline__ TilePart part_at(const Params& P, int r, int k) {
  if constexpr (DEV) return ld_tile(P.tiles + (int64_t)r * P.nt + k);
  else return P.tiles[(int64_t)r * P.nt + k];
}

template <bool DEV = false>
__device__ __forceinline__ PartHead load_head(const Params& P, int r, bool tv, bool mom) {
  const int lane = threadIdx.x & 63;
  PartHead h{{0.0, 0.0, kNegInf, kNegInf, kNegInf, kNegInf, 0x7fffffff, 0x7fffffff}, 0.0,
             {0.0, 0.0, 0.0}};
  if (lane < P.nt) {
    h.t = part_at<DEV>(P, r, lane);
    if (tv) h.tv = P.tvpart[(int64_t)r * P.nt + lane];
    if (mom) h.m = P.moms[(int64_t)r * P.nt + lane];
  }
  return h;
}

// A log-loss rule's statistic (nats) from row sums S and moments against the
// row references (contraction off, as in mom_move).
__device__ __forceinline__ double log_stat(int rule, double lq2, double lp2, double sq, double sp,
                                           double mhq, double mhp, double mx) {
#pragma clang fp contract(off)
  const double Hq = kLn2 * (lq2 - mhq / sq), Hp = kLn2 * (lp2 - mhp / sp);
  return rule == SPC_RULE_BILD      ? kLn2 * (lp2 - mx / sq)
         : rule == SPC_RULE_CHOWLOG ? Hq
                                    : Hq - Hp;
}

// One wavefront merges the nt tile partials of row r in a fixed order (lane l
// takes tiles l, l + 64, ...; butterflies combine the lanes), adding the TV
// partials when `tv`, and with mrule (a log-loss rule or BiLD*) its
// statistic from the tiles' first moments: against the row references,
//   H(q) = ln 2 (log2 S_q - H_q / S_q),  H(p) = ln 2 (log2 S_p - H_p / S_p),
//   D(q, p) = -sum q log p = ln 2 (log2 S_p - X / S_q),
// each a sum of two non-negative terms.  Every lane returns the same RowStat.
template <bool DEV = false>
__device__ __forceinline__ RowStat merge_row(const Params& P, int r, bool greedy, bool tv,
                                             int mrule, const PartHead& h) {
  const int lane = threadIdx.x & 63;
  const int nt = P.nt;
  const double* tvp = P.tvpart + (int64_t)r * nt;
  const TilePart& t0 = h.t;
  double tvs = h.tv;
  float zq = t0.zmax_q, zp = t0.zmax_p, rq = t0.r_q, rp = t0.r_p;
  for (int k = lane + 64; k < nt; k += 64) {
    const TilePart tk = part_at<DEV>(P, r, k);
    zq = fmaxf(zq, tk.zmax_q);
    zp = fmaxf(zp, tk.zmax_p);
    rq = fmaxf(rq, tk.r_q);
    rp = fmaxf(rp, tk.r_p);
  }
  zq = wave_max(zq);
  zp = wave_max(zp);
  rq = wave_max(rq);
  rp = wave_max(rp);
  double sq = 0.0, sp = 0.0, mhq = 0.0, mhp = 0.0, mx = 0.0;
  int aq = 0x7fffffff, ap = 0x7fffffff;
  auto add = [&](const TilePart& tk, const TileMom& mk) {
    // r_k - r is exact in fp64; an all -inf tile has s = 0
    const double gq = (double)tk.r_q - (double)rq, gp = (double)tk.r_p - (double)rp;
    const double fq = exp2_acc(gq), fp = exp2_acc(gp);
    sq += tk.s_q * fq;
    sp += tk.s_p * fp;
    if (greedy) {
      if (tk.zmax_q == zq) aq = min(aq, tk.amax_q);
      if (tk.zmax_p == zp) ap = min(ap, tk.amax_p);
    }
    if (mrule) {
      mom_add(mhq, mk.hq, tk.s_q, fq, gq);
      mom_add(mhp, mk.hp, tk.s_p, fp, gp);
      mom_add(mx, mk.x, tk.s_q, fq, gp);
    }
  };
  add(t0, h.m);
  for (int k = lane + 64; k < nt; k += 64) {
    add(part_at<DEV>(P, r, k), mrule ? P.moms[(int64_t)r * nt + k] : TileMom{0.0, 0.0, 0.0});
    if (tv) tvs += tvp[k];
  }
  sq = wave_sum(sq);
  sp = wave_sum(sp);
  tvs = wave_sum(tvs);
  aq = wave_min(aq);
  ap = wave_min(ap);
  RowStat rs;
  const double lq2 = log2_acc(sq), lp2 = log2_acc(sp);
  rs.lz_q = (double)rq + lq2;
  rs.lz_p = (double)rp + lp2;
  rs.tv = tvs;
  rs.slog = 0.0;
  if (mrule) {
    mhq = wave_sum(mhq);
    mhp = wave_sum(mhp);
    mx = wave_sum(mx);
    rs.slog = log_stat(mrule, lq2, lp2, sq, sp, mhq, mhp, mx);
  }
  rs.zmax_q = zq;
  rs.zmax_p = zp;
  rs.amax_q = greedy ? aq : -1;
  rs.amax_p = greedy ? ap : -1;
  return rs;
}

__device__ __forceinline__ RowStat merge_row(const Params& P, int r, bool greedy, bool tv) {
  return merge_row(P, r, greedy, tv, 0, load_head(P, r, tv, false));
}

// ------------------------------------------------------------- decision
// delta_j by the rule of Table 1 and the accept draw a_j of Alg. 4 for row j
// of a sequence, from its merged statistics.  x is the draft token x_{t+j},
// zqx / zpx its two logits and u its uniform (lane-uniform values).  For a
// greedy token-rule row, zpx is p's logit at the drafter's argmax instead.
__device__ __forceinline__ RowDecision decide_row(const SeqParam& sp, const RowStat& rs, int j,
                                                  int gamma, int V, int x, float zqx, float zpx,
                                                  float u) {
  RowDecision d;
  d.rs = rs;
  d.u = u;
  const double maxq = exp2_acc((double)rs.zmax_q * sp.c - rs.lz_q);
  const double maxp = exp2_acc((double)rs.zmax_p * sp.c - rs.lz_p);
  d.maxq = (float)maxq;
  d.maxp = (float)maxp;
  if (is_token(sp.rule)) {
    // Alg. 6's target pi = q (1 - r) + p eta; reported delta_j = r(x_j)
    const TokenRule tr = token_rule(sp, rs, maxp);
    if (sp.greedy) {
      // r at argmax q (temperature-1 statistics): one-hot pi~ at argmax p
      // when r = 1, else at argmax q; eta~ = r
      // (TokenV1 there is max q < max p - alpha: Diff's comparison, made alike)
      d.delta = tr.on_p ? zpx < tr.theta
                        : defer_rule(SPC_RULE_DIFF, sp.alpha, maxq, maxp, 0.0);
      d.tv = (float)d.delta;
      d.keep = j < gamma && x >= 0 && x < V && x == (d.delta ? rs.amax_p : rs.amax_q);
      return d;
    }
    d.tv = (float)rs.tv;
    if (j >= gamma || x < 0 || x >= V) {
      d.delta = 0;
      d.keep = 0;  // a_gamma = 0; a draft outside the vocabulary is rejected
    } else {
      d.delta = token_r(tr, zqx, zpx);
      if (!d.delta || zqx == kNegInf) {
        d.keep = 1;  // pi(x) >= q(x)
      } else {
        // pi(x) / q(x) = p(x) eta / q(x) = 2^dd
        const double le = rs.tv > 0.0 ? log2(rs.tv) : -__builtin_huge_val();
        const double dd = ((double)zpx - (double)zqx) * sp.c - (rs.lz_p - rs.lz_q) + le;
        d.keep = !(dd < 0.0) || (double)u < exp2_acc(dd);
      }
    }
    return d;
  }
  // greedy: one-hot q~, p~ give D_TV = 1(argmax q != argmax p)  (Lemma 6)
  const double tv = sp.greedy ? (rs.amax_q != rs.amax_p ? 1.0 : 0.0) : rs.tv;
  d.tv = (float)tv;
  if (sp.rule == SPC_RULE_LOSSY) {
    // Lemma 2 (beta = 1): no deferral; pi(x) / q(x) = min(1, p(x) / ((1 -
    // alpha) q(x))) where p(x) < q(x) (alpha < 0: p(x) / q(x)), and >= 1
    // elsewhere; the one-hot greedy target sits at argmax p
    d.delta = 0;
    if (j >= gamma || x < 0 || x >= V) {
      d.keep = 0;
    } else if (sp.greedy) {
      d.keep = x == rs.amax_p;
    } else {
      const double L = sp.alpha > 0.0 ? -log2(1.0 - sp.alpha) : 0.0;
      const double dd = (((double)zpx * sp.c - rs.lz_p) - ((double)zqx * sp.c - rs.lz_q)) + L;
      d.keep = !(dd < 0.0) || (double)u < exp2_acc(dd);
    }
    return d;
  }
  if (is_log(sp.rule)) {
    // statistic in nats against alpha (OPTLOG: alpha D_TV); greedy BiLD* reads
    // D = lse_p - z_p(argmax q) at temperature 1, zpx being that logit
    if (sp.rule == SPC_RULE_BILD && sp.greedy) d.rs.slog = rs.lz_p * kLn2 - (double)zpx;
    const double th = sp.rule == SPC_RULE_OPTLOG ? sp.alpha * tv : sp.alpha;
    d.delta = d.rs.slog > th;
  } else {
    d.delta = defer_rule(sp.rule, sp.alpha, maxq, maxp, tv);
  }
  if (j >= gamma || x < 0 || x >= V) {
    d.keep = 0;  // a_gamma = 0; a draft outside the vocabulary is rejected
  } else if (sp.greedy) {
    d.keep = (x == (d.delta ? rs.amax_p : rs.amax_q));
  } else if (d.delta) {
    // pi = p here: keep if p(x) >= q(x), else with probability p(x) / q(x)
    const double lq = (double)zqx * sp.c - rs.lz_q;
    const double lp = (double)zpx * sp.c - rs.lz_p;
    d.keep = !(lp < lq) || (double)u < exp2_acc(lp - lq);
  } else {
    d.keep = 1;  // pi = q: accepted with probability 1
  }
  return d;
}

// Wave 0: j* (the first rejection, by one ballot), the outputs when `write`,
// and the sampling state of sequence b.
__device__ __forceinline__ void finish_seq(const Params& P, int b, const SeqParam& sp,
                                           SeqShared& ss, bool write) {
  const int lane = threadIdx.x;
  const int gamma = P.gamma, g1 = gamma + 1;
  const bool on = lane < g1;
  const int64_t row = (int64_t)b * g1 + lane;
  RowDecision d{};
  if (on && sp.valid) d = ss.rows[lane];
  // a NaN second-pass statistic marks a row whose one-read pass gave up
  // waiting for its tiles: the sequence is reported invalid
  const bool lost = needs_pass2(sp) && __ballot(on && d.tv != d.tv) != 0;
  if (!sp.valid || lost) {
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
  if (write && on) {
    P.out_defer[row] = (uint8_t)d.delta;
    if (P.out_stats) {
      const double T = sp.greedy ? 1.0 : kLog2e / sp.c;
      float* o = P.out_stats + row * 8;
      o[0] = (float)((double)d.rs.zmax_q / T);
      o[1] = (float)(d.rs.lz_q * kLn2);
      o[2] = d.maxq;
      o[3] = (float)((double)d.rs.zmax_p / T);
      o[4] = (float)(d.rs.lz_p * kLn2);
      o[5] = d.maxp;
      o[6] = d.tv;
      o[7] = (float)d.rs.slog;
    }
    if (P.out_argmax) {
      P.out_argmax[row * 2 + 0] = d.rs.amax_q;
      P.out_argmax[row * 2 + 1] = d.rs.amax_p;
    }
  }
  const unsigned long long rej = __ballot(on && !d.keep);
  const int jstar = __ffsll(rej) - 1;  // bit gamma is always set
  const int dstar = lane_i32(d.delta, jstar);
  const int aq = lane_i32(d.rs.amax_q, jstar);
  const int ap = lane_i32(d.rs.amax_p, jstar);
  const float ug = lane_f32(d.u, gamma);
  if (lane == 0) {
    SeqState s{jstar, kNone, 0.0f, 0};
    if (sp.greedy) {
      if (write) {
        P.out_token[b] = (dstar || sp.rule == SPC_RULE_LOSSY) ? ap : aq;
        if (P.out_norm) P.out_norm[b] = 1.0f;
      }
    } else {
      if (is_token(sp.rule)) {
        s.kind = (jstar < gamma) ? kTokRes : kTokPi;
      } else if (sp.rule == SPC_RULE_LOSSY) {
        // residual max(0, pi - q) = max(0, p - q); extra token from p
        s.kind = (jstar < gamma) ? kResidual : kP;
      } else {
        // a rejection with delta = 0 only happens for an out-of-range draft;
        // its residual max(0, q - q) is empty, so p is sampled instead
        s.kind = (jstar < gamma) ? (dstar ? kResidual : kP) : (dstar ? kP : kQ);
      }
      s.u = ug;
    }
    if (write) P.out_accept[b] = jstar;
    ss.seq = s;
  }
}

// Whole block: merge and decide the rows of sequence b (wave w takes rows
// w, w + 4, ...), then wave 0 finds j*.  With `write` the outputs are written
// too: every sampling workgroup of a sequence reaches the same decision by
// the same fixed-order computation, and one of them writes it.
template <int DT>
__device__ __forceinline__ void decide_seq(const Params& P, int b, const SeqParam& sp,
                                           SeqShared& ss, bool write) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int gamma = P.gamma, g1 = gamma + 1, V = P.V;
  if (sp.valid) {
    // Loads in dependency order: the first row's partials and the draft
    // data (lane l of wave wv takes row wv + kSampWaves * l) go out together;
    // the logits at the draft tokens follow the tokens and stay in flight
    // while the rows merge.
    const bool tv = needs_pass2(sp);
    const bool mom = needs_mom(sp);
    // greedy TokenV2/V3 and BiLD* read p at the drafter's argmax
    const bool greedy_pa = sp.greedy && ((is_token(sp.rule) && sp.rule != SPC_RULE_TOKEN_V1) ||
                                         sp.rule == SPC_RULE_BILD);
    PartHead h{};
    if (wv < g1) h = load_head(P, b * g1 + wv, tv, mom);
    const int jl = wv + kSampWaves * lane;
    int x = -1;
    float zqx = 0.0f, zpx = 0.0f, u = 0.0f;
    if (jl < g1) {
      const int64_t row = (int64_t)b * g1 + jl;
      if (!sp.greedy) u = P.uniforms[row];
      if (jl < gamma) {
        x = P.draft[(int64_t)b * gamma + jl];
        if (!sp.greedy && x >= 0 && x < V) {
          zqx = load_logit<DT>(P.q, row, V, x);
          zpx = load_logit<DT>(P.p, row, V, x);
        }
      }
    }
    for (int i = 0; wv + kSampWaves * i < g1; ++i) {
      const int j = wv + kSampWaves * i;
      // the next row's partials load while this row merges
      PartHead hn{};
      if (j + kSampWaves < g1) hn = load_head(P, b * g1 + j + kSampWaves, tv, mom);
      const RowStat rs = merge_row(P, b * g1 + j, sp.greedy, tv, mom ? sp.rule : 0, h);
      h = hn;
      const float zpa = (greedy_pa && rs.amax_q >= 0 && rs.amax_q < V)
                            ? load_logit<DT>(P.p, (int64_t)b * g1 + j, V, rs.amax_q)
                            : lane_f32(zpx, i);
      const RowDecision d = decide_row(sp, rs, j, gamma, V, lane_i32(x, i), lane_f32(zqx, i),
                                       zpa, lane_f32(u, i));
      if (lane == 0) ss.rows[j] = d;
    }
  }
  __syncthreads();
  if (threadIdx.x < 64) finish_seq(P, b, sp, ss, write);
  __syncthreads();
}

// ------------------------------------------------------------- sampling
// A chunk is what one wavefront covers reading wave-contiguously: lane l's
// lane load i covers entries (i * 64 + l) * VW .. + VW - 1 of it.  The
// residual pass sums SampChunks; a statistics tile is kSampWaves consecutive
// SubChunks, one per wavefront of a sampling workgroup.
template <int DT, bool VEC, int U_>
struct Chunk {
  static constexpr int U = U_;
  static constexpr int NW = Tile<DT, VEC, U_>::NW, VW = Tile<DT, VEC, U_>::VW;
  static constexpr int N = 64 * U * VW;  // entries per chunk
};
// A sub-chunk of a TN-entry tile drawn from by NWV wavefronts: one per
// wavefront, or several of at most 4 lane loads each.
template <int DT, bool VEC, int NWV, int TN = StatTile<DT, VEC>::N>
using SubChunk = Chunk<DT, VEC, (TN / (64 * NWV * Tile<DT, VEC, 1>::VW) < 4)
                                    ? TN / (64 * NWV * Tile<DT, VEC, 1>::VW)
                                    : 4>;
template <int DT, bool VEC>
using SampChunk = Chunk<DT, VEC, VEC ? 2 : 8>;

template <class C>
using ChunkRegs = uint32_t[C::U][C::NW];

// Lane loads of the chunk starting at entry c0 of a row (V entries); a chunk
// past the row reads entry 0 and masks everything.
template <int DT, bool VEC, class C>
__device__ __forceinline__ void load_chunk(const char* row, int64_t c0, int V, ChunkRegs<C>& w) {
  const int lane = threadIdx.x & 63;
  if (c0 + C::N <= V) {  // a whole chunk (wave-uniform): no masking
    load_tile<DT, VEC, C::U, false, 64, false>(row, c0, V, w, lane);
  } else {
    const bool live = c0 < V;
    load_tile<DT, VEC, C::U, false, 64>(row, live ? c0 : 0, live ? V : 0, w, lane);
  }
}

// Sources of the part masses of the sampled distribution: the statistics
// partials per tile (q or p: each tile's share of the normaliser), the
// statistics and eta partials together (a token rule's target), or the
// residual masses per SampChunk computed by the sampling pass.
enum MassSrc : int { kSrcStatsQ = 0, kSrcStatsP = 1, kSrcPass = 3, kSrcTokPi = 4,
                     kSrcDraft = 5 };

template <int SRC>
__device__ __forceinline__ double part_mass(const Params& P, int64_t row, int b, int k,
                                            const RowStat& rs) {
  if constexpr (SRC == kSrcStatsQ) {
    const TilePart& t = P.tiles[row * P.nt + k];
    return t.s_q * exp2_acc((double)t.r_q - rs.lz_q);
  } else if constexpr (SRC == kSrcStatsP) {
    const TilePart& t = P.tiles[row * P.nt + k];
    return t.s_p * exp2_acc((double)t.r_p - rs.lz_p);
  } else if constexpr (SRC == kSrcTokPi) {
    // Alg. 6's target over a tile: its q mass less the eta partial (the q
    // mass where r = 1), plus eta times its p mass
    const TilePart& t = P.tiles[row * P.nt + k];
    const double qm = t.s_q * exp2_acc((double)t.r_q - rs.lz_q);
    const double pm = t.s_p * exp2_acc((double)t.r_p - rs.lz_p);
    return fmax(qm - P.tvpart[row * P.nt + k], 0.0) + rs.tv * pm;
  } else if constexpr (SRC == kSrcDraft) {
    // the q statistics partials of the drafter kernel's own launch
    const TilePart t = ld_tile(P.tiles + row * P.nt + k);
    return t.s_q * exp2_acc((double)t.r_q - rs.lz_q);
  } else {
    return ld_dev_f64(P.masses + (int64_t)b * P.nc + k);
  }
}

// Wave 0: the part (tile or chunk) of the inverse-CDF draw -- the first part
// k with C_k > u W, C_k the running mass through part k in vocabulary order
// and W the total -- and the target mass left at its start.  Returns W.
// Parts are read kFindGroup per lane at a time, all loads in flight
// together; for at most 64 * kFindGroup parts both passes use one read.
constexpr int kFindGroup = 4;

template <int SRC>
__device__ __forceinline__ void load_parts(const Params& P, int64_t row, int b, int K, int k0,
                                           const RowStat& rs, double (&m)[kFindGroup]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < kFindGroup; ++j) {
    const int k = k0 + j * 64 + lane;
    m[j] = k < K ? part_mass<SRC>(P, row, b, k, rs) : 0.0;
  }
}

template <int SRC>
__device__ __forceinline__ double find_part(const Params& P, int64_t row, int b, int K,
                                            const RowStat& rs, float u, int* ks_out,
                                            double* rem_out) {
  constexpr int GN = 64 * kFindGroup;
  double m0[kFindGroup];
  load_parts<SRC>(P, row, b, K, 0, rs, m0);
  double W = 0.0;
#pragma unroll
  for (int j = 0; j < kFindGroup; ++j) W += wave_sum(m0[j]);
  for (int k0 = GN; k0 < K; k0 += GN) {
    double m[kFindGroup];
    load_parts<SRC>(P, row, b, K, k0, rs, m);
#pragma unroll
    for (int j = 0; j < kFindGroup; ++j) W += wave_sum(m[j]);
  }
  const double target = (double)u * W;
  double carry = 0.0, rem = 0.0;
  int ks = -1, klast = -1;
  for (int k0 = 0; k0 < K && ks < 0; k0 += GN) {
    double m[kFindGroup];
    if (k0 == 0) {
#pragma unroll
      for (int j = 0; j < kFindGroup; ++j) m[j] = m0[j];
    } else {
      load_parts<SRC>(P, row, b, K, k0, rs, m);
    }
#pragma unroll
    for (int j = 0; j < kFindGroup; ++j) {
      const double incl = carry + wave_incl_scan(m[j]);
      const unsigned long long pos = __ballot(m[j] > 0.0);
      const unsigned long long hit = __ballot(m[j] > 0.0 && incl > target);
      if (pos) klast = k0 + j * 64 + 63 - __clzll(pos);
      if (ks < 0 && hit) {
        const int l = __ffsll(hit) - 1;
        ks = k0 + j * 64 + l;
        rem = target - (lane_f64(incl, l) - lane_f64(m[j], l));
      }
      carry = lane_f64(incl, 63);
    }
  }
  if (ks < 0) {  // rounding left u W at or past the end: the last part with mass
    ks = klast;
    rem = __builtin_huge_val();
  }
  *ks_out = ks;
  *rem_out = rem;
  return W;
}

// Whole block: residual masses (KIND) of the SampChunks of a row (K
// sampling workgroups per sequence): wave w of workgroup kw takes chunks
// kw * kSampWaves + w, then + K * kSampWaves, ...; the next chunk loads while
// one is summed, and chunk c's mass goes to masses[c].  No block barrier:
// every wave drains its own stores.
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ void residual_masses(const char* qrow, const char* prow, int V, int nc,
                                                int K, int kw, const ProbScale& ps,
                                                double* masses) {
  using C = SampChunk<DT, VEC>;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int step = K * kSampWaves;
  ChunkRegs<C> wq, wp, nq = {}, np = {};
  {
    const int c = kw * kSampWaves + wv;
    const int64_t c0 = c < nc ? (int64_t)c * C::N : (int64_t)V;
    load_chunk<DT, VEC, C>(qrow, c0, V, wq);
    load_chunk<DT, VEC, C>(prow, c0, V, wp);
  }
  for (int b0 = kw * kSampWaves; b0 < nc; b0 += step) {  // block-uniform
    const int c = b0 + wv;
    if (b0 + step < nc) {  // prefetch the next batch
      const int cn = c + step;
      const int64_t c0 = cn < nc ? (int64_t)cn * C::N : (int64_t)V;
      load_chunk<DT, VEC, C>(qrow, c0, V, nq);
      load_chunk<DT, VEC, C>(prow, c0, V, np);
    }
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < C::U; ++i) {
      float t = 0.0f;
#pragma unroll
      for (int e = 0; e < C::VW; ++e)
        t += weight_of<KIND>(elem<DT, VEC>(wq[i], e), elem<DT, VEC>(wp[i], e), ps);
      acc += (double)t;
    }
    acc = wave_sum(acc);
    if (lane == 0 && c < nc) st_dev_f64(masses + c, acc);
#pragma unroll
    for (int i = 0; i < C::U; ++i)
#pragma unroll
      for (int j = 0; j < C::NW; ++j) {
        wq[i][j] = nq[i][j];
        wp[i][j] = np[i][j];
      }
  }
  vmem_drain();
}

// Wave 0: the in-chunk draw in the chunk starting at entry c0.  Lane loads
// are scanned in entry order -- lane load i, then lane -- for the first one
// where the running mass exceeds rem; its lane then walks its VW entries.
// Rounding that leaves rem unreached takes the last entry with mass.
template <int DT, bool VEC, class C, int KIND>
__device__ __forceinline__ void pick_wave(const Params& P, int b, int64_t row, int64_t c0,
                                          double rem, const ProbScale& ps) {
  constexpr int EB = StatTile<DT, VEC>::EB;
  const int lane = threadIdx.x & 63;
  const int V = P.V;
  const char* qrow = (const char*)P.q + row * V * EB;
  const char* prow = (const char*)P.p + row * V * EB;
  ChunkRegs<C> cq = {}, cp = {};
  if (KIND != kP) load_chunk<DT, VEC, C>(qrow, c0, V, cq);
  if (KIND != kQ) load_chunk<DT, VEC, C>(prow, c0, V, cp);
  double carry = 0.0, before = 0.0;
  int hlane = -1, last_pos = -1;
  int64_t hbase = 0;
  uint32_t sq[C::NW] = {}, sp_[C::NW] = {};
#pragma unroll
  for (int i = 0; i < C::U; ++i) {
    const int64_t base = c0 + (int64_t)(i * 64 + lane) * C::VW;
    double m = 0.0;
#pragma unroll
    for (int e = 0; e < C::VW; ++e) {
      const float w = weight_of<KIND>(elem<DT, VEC>(cq[i], e), elem<DT, VEC>(cp[i], e), ps);
      m += (double)w;
      if (w > 0.0f) last_pos = max(last_pos, (int)(base + e));
    }
    const double incl = carry + wave_incl_scan(m);
    if (hlane < 0) {  // wave-uniform
      const unsigned long long hit = __ballot(m > 0.0 && incl > rem);
      if (hit) {
        hlane = __ffsll(hit) - 1;
        before = lane_f64(incl, hlane) - lane_f64(m, hlane);
        hbase = base;
#pragma unroll
        for (int j = 0; j < C::NW; ++j) {
          sq[j] = cq[i][j];
          sp_[j] = cp[i][j];
        }
      }
    }
    carry = lane_f64(incl, 63);
  }
  if (hlane < 0) {
    const int lp = -wave_min(-last_pos);
    if (lane == 0) P.out_token[b] = lp;
    return;
  }
  if (lane != hlane) return;
  double run = before;
  int hit = -1, lastw = -1;
#pragma unroll
  for (int e = 0; e < C::VW; ++e) {
    const float w = weight_of<KIND>(elem<DT, VEC>(sq, e), elem<DT, VEC>(sp_, e), ps);
    run += (double)w;
    if (w > 0.0f) lastw = (int)(hbase + e);
    if (hit < 0 && run > rem && w > 0.0f) hit = (int)(hbase + e);
  }
  P.out_token[b] = hit >= 0 ? hit : lastw;  // rounding inside the lane load
}

// Whole block: the draw inside statistics tile t0 (entry offset).  Each
// wavefront sums the weights of one SubChunk; wave 0 scans the kSampWaves
// sums for the sub-chunk where rem is crossed and draws inside it.
template <int DT, bool VEC, int KIND, int NWV, int TN = StatTile<DT, VEC>::N>
__device__ __forceinline__ void pick_tile(const Params& P, int b, int64_t row, int64_t t0,
                                          double rem, const ProbScale& ps, SharedT<NWV>& sh) {
  using C = SubChunk<DT, VEC, NWV, TN>;
  constexpr int NS = TN / C::N;  // sub-chunks of the tile
  static_assert(NS * C::N == TN && NS % NWV == 0 && NS <= 64,
                "a tile is a whole number of sub-chunks per wavefront");
  constexpr int EB = StatTile<DT, VEC>::EB;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int V = P.V;
  const char* qrow = (const char*)P.q + row * V * EB;
  const char* prow = (const char*)P.p + row * V * EB;
  for (int sc = wv; sc < NS; sc += NWV) {  // wave wv sums sub-chunks wv, wv + NWV, ...
    ChunkRegs<C> cq = {}, cp = {};
    if (KIND != kP) load_chunk<DT, VEC, C>(qrow, t0 + sc * C::N, V, cq);
    if (KIND != kQ) load_chunk<DT, VEC, C>(prow, t0 + sc * C::N, V, cp);
    double m = 0.0;
#pragma unroll
    for (int i = 0; i < C::U; ++i) {
      float t = 0.0f;
#pragma unroll
      for (int e = 0; e < C::VW; ++e)
        t += weight_of<KIND>(elem<DT, VEC>(cq[i], e), elem<DT, VEC>(cp[i], e), ps);
      m += (double)t;
    }
    m = wave_sum(m);
    if (lane == 0) sh.dv[sc] = m;
  }
  __syncthreads();
  if (wv != 0) return;
  const double ml = lane < NS ? sh.dv[lane] : 0.0;
  const double incl = wave_incl_scan(ml);
  const unsigned long long hit = __ballot(ml > 0.0 && incl > rem);
  const unsigned long long pos = __ballot(ml > 0.0);
  int c;
  double r;
  if (hit) {
    c = __ffsll(hit) - 1;
    r = rem - (lane_f64(incl, c) - lane_f64(ml, c));
  } else {  // rounding: the last sub-chunk with mass, its last entry with mass
    c = pos ? 63 - __clzll(pos) : 0;
    r = __builtin_huge_val();
  }
  pick_wave<DT, VEC, C, KIND>(P, b, row, t0 + c * C::N, r, ps);
}

// Whole block: the inverse-CDF draw of sequence b at row `row` (the row of
// j*) from the distribution `kind`, whose part masses come from `src`.  Wave 0
// finds the part; the draw inside a residual chunk runs in wave 0, the draw
// inside a statistics tile uses every wavefront.  An empty residual (possible
// only through rounding) is replaced by p.
template <int DT, bool VEC>
__device__ __forceinline__ void draw(const Params& P, int b, int64_t row, int kind, int src,
                                     float u, const SeqParam& sp, const RowStat& rs,
                                     SeqShared& ss, SampShared& sh) {
  if (threadIdx.x < 64) {
    int ks;
    double rem, W;
    if (src == kSrcStatsQ) W = find_part<kSrcStatsQ>(P, row, b, P.nt, rs, u, &ks, &rem);
    else if (src == kSrcStatsP) W = find_part<kSrcStatsP>(P, row, b, P.nt, rs, u, &ks, &rem);
    else if (src == kSrcTokPi) W = find_part<kSrcTokPi>(P, row, b, P.nt, rs, u, &ks, &rem);
    else W = find_part<kSrcPass>(P, row, b, P.nc, rs, u, &ks, &rem);
    if ((kind == kResidual || kind == kTokRes) && !(W > 0.0)) {
      kind = kP;
      src = kSrcStatsP;
      W = find_part<kSrcStatsP>(P, row, b, P.nt, rs, u, &ks, &rem);
    }
    if (threadIdx.x == 0) {
      ss.pk = PickState{ks, kind, src, rem};
      if (P.out_norm) P.out_norm[b] = (float)W;
      if (ks < 0) P.out_token[b] = -1;
    }
  }
  __syncthreads();
  const PickState pk = ss.pk;
  if (pk.k < 0) return;  // block-uniform
  const ProbScale ps = prob_scale(sp, rs, pk.kind == kTokRes || pk.kind == kTokPi);
  constexpr int TN = StatTile<DT, VEC>::N;
  if (pk.src == kSrcPass) {
    using SC = SampChunk<DT, VEC>;
    if (threadIdx.x < 64) {
      if (pk.kind == kTokRes)
        pick_wave<DT, VEC, SC, kTokRes>(P, b, row, (int64_t)pk.k * SC::N, pk.rem, ps);
      else
        pick_wave<DT, VEC, SC, kResidual>(P, b, row, (int64_t)pk.k * SC::N, pk.rem, ps);
    }
  } else if (pk.kind == kQ) {
    pick_tile<DT, VEC, kQ, kSampWaves>(P, b, row, (int64_t)pk.k * TN, pk.rem, ps, sh);
  } else if (pk.kind == kP) {
    pick_tile<DT, VEC, kP, kSampWaves>(P, b, row, (int64_t)pk.k * TN, pk.rem, ps, sh);
  } else if (pk.kind == kTokPi) {
    pick_tile<DT, VEC, kTokPi, kSampWaves>(P, b, row, (int64_t)pk.k * TN, pk.rem, ps, sh);
  } else {
    pick_tile<DT, VEC, kResidual, kSampWaves>(P, b, row, (int64_t)pk.k * TN, pk.rem, ps, sh);
  }
}

// ================================================================ kernels

// Statistics pass.  grid (nt, R): stats tile k of row r.  Each thread takes
// the exact max of its entries and the sum of 2^(z c - r_t), r_t = max * c_hi
// (a reference near its largest z c); each wave combines its threads against
// the wave max, and thread 0 the waves against the tile max.  With ARGMAX
// (batches that may hold greedy rows) the lowest entry attaining the max is
// found as well.
// Thread sums of one statistics tile: s = sum 2^a over the thread's entries,
// a = z c - r (r the thread reference); with MOM (a set of kMom* bits) also
// the first moments it names: hq = sum 2^a_q a_q, hp = sum 2^a_p a_p and
// x = sum 2^a_q a_p (entries of zero weight contribute nothing, so -inf
// logits never meet an infinite factor; a finite-weight q entry facing a -inf
// p logit makes x = -inf).  Moments outside the set stay 0.
template <int DT, bool VEC, int MOM>
__device__ __forceinline__ void tile_sums(const uint32_t (&wq)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                          const uint32_t (&wp)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                          const SeqParam& sp, float rq, float rp, float& sq,
                                          float& spp, float& hq, float& hp, float& xq) {
  using T = StatTile<DT, VEC>;
  if constexpr (MOM) {
    // one running sum per quantity: the moments' extra values stay short-lived
#pragma unroll
    for (int i = 0; i < T::U; ++i)
#pragma unroll
      for (int e = 0; e < T::VW; ++e) {
        const float zq = elem<DT, VEC>(wq[i], e), zp = elem<DT, VEC>(wp[i], e);
        const float aq = fmaf(zq, sp.c_lo, fmaf(zq, sp.c_hi, -rq));
        const float ap = fmaf(zp, sp.c_lo, fmaf(zp, sp.c_hi, -rp));
        const float tq = exp2_hw(aq), tp = exp2_hw(ap);
        const bool wq_pos = tq > 0.0f;
        sq += tq;
        spp += tp;
        if constexpr ((MOM & kMomHQ) != 0) hq = fmaf(tq, wq_pos ? aq : 0.0f, hq);
        if constexpr ((MOM & kMomX) != 0) xq = fmaf(tq, wq_pos ? ap : 0.0f, xq);
        if constexpr ((MOM & kMomHP) != 0) hp = fmaf(tp, tp > 0.0f ? ap : 0.0f, hp);
        // keep the scheduler from hoisting every exponential of the tile
        if ((e & 3) == 3) __builtin_amdgcn_sched_barrier(0);
      }
  } else {
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
  }
}

// The partial of statistics tile k of row r from its loaded entries (wq, wp),
// written by thread 0: with DEV through agent-scope stores, for readers in
// the same launch.
template <int DT, bool VEC, bool ARGMAX, int MOM, bool DEV>
__device__ __forceinline__ void tile_partial(const Params& P, int r, int k, const SeqParam& sp,
                                             const uint32_t (&wq)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                             const uint32_t (&wp)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                             Shared& sh) {
  using T = StatTile<DT, VEC>;
  const int64_t t0 = (int64_t)k * T::N;
  // Thread max, from the maxima of its lane loads; with ARGMAX also the
  // lowest entry attaining it (indices fit 32 bits: V < 2^31).
  float gq[T::U], gp[T::U];
#pragma unroll
  for (int i = 0; i < T::U; ++i) {
    float a = kNegInf, b = kNegInf;
#pragma unroll
    for (int e = 0; e < T::VW; ++e) {
      a = fmaxf(a, elem<DT, VEC>(wq[i], e));
      b = fmaxf(b, elem<DT, VEC>(wp[i], e));
    }
    gq[i] = a;
    gp[i] = b;
  }
  float mq = gq[0], mp = gp[0];
#pragma unroll
  for (int i = 1; i < T::U; ++i) {
    mq = fmaxf(mq, gq[i]);
    mp = fmaxf(mp, gp[i]);
  }
  int iq = 0x7fffffff, ip = 0x7fffffff;
  const int base = (int)t0 + (int)threadIdx.x * T::VW;
  if constexpr (ARGMAX && !MOM) {
    iq = first_max_index<DT, VEC, T::U, kThreads>(wq, gq, mq, base);
    ip = first_max_index<DT, VEC, T::U, kThreads>(wp, gp, mp, base);
  }
  const float rq = (mq == kNegInf) ? 0.0f : mq * sp.c_hi;
  const float rp = (mp == kNegInf) ? 0.0f : mp * sp.c_hi;
  if constexpr (DEV) {
    // the packed words outlive this tile's statistics (the one-read second
    // pass uses them): unpack again below rather than hold all the entries
#pragma unroll
    for (int i = 0; i < T::U; ++i)
#pragma unroll
      for (int j = 0; j < T::NW; ++j)
        asm volatile("" : "+v"(const_cast<uint32_t&>(wq[i][j])), "+v"(const_cast<uint32_t&>(wp[i][j])));
  }
  float sq = 0.0f, spp = 0.0f, hq = 0.0f, hp = 0.0f, xq = 0.0f;
  constexpr bool mom = MOM;
  tile_sums<DT, VEC, MOM>(wq, wp, sp, rq, rp, sq, spp, hq, hp, xq);
  // the moments are complete here: left free, the compiler sinks their
  // accumulation into the conditional combine below and keeps every
  // exponential of the tile live until then
  if constexpr (MOM) asm volatile("" : "+v"(hq), "+v"(hp), "+v"(xq), "+v"(sq), "+v"(spp));
  if constexpr (ARGMAX && MOM) {
    // the lowest entry equal to the thread max, in a pass of its own after
    // the sums
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = T::U - 1; i >= 0; --i)
#pragma unroll
      for (int e = T::VW - 1; e >= 0; --e) {
        const int idx = base + i * kThreads * T::VW + e;
        if (elem<DT, VEC>(wq[i], e) == mq) iq = idx;
        if (elem<DT, VEC>(wp[i], e) == mp) ip = idx;
      }
    asm volatile("" : "+v"(iq), "+v"(ip));
  }
  // Wave partials against the wave max (r_t - r_w is exact in fp64; only its
  // rounding to float is inexact), then one barrier and thread 0 combines the
  // waves in order against the tile max.
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const float Wq = wave_max(mq), Wp = wave_max(mp);
  const double eq = (double)rq - (double)(Wq * sp.c_hi), ep = (double)rp - (double)(Wp * sp.c_hi);
  const double fq = (double)exp2_hw((float)eq), fp = (double)exp2_hw((float)ep);
  double dq = (mq == kNegInf) ? 0.0 : (double)sq * fq;
  double dp = (mp == kNegInf) ? 0.0 : (double)spp * fp;
  dq = wave_sum(dq);
  dp = wave_sum(dp);
  double mhq = 0.0, mhp = 0.0, mx = 0.0;
  if constexpr (mom) {
    mhq = wave_sum(mq == kNegInf ? 0.0 : mom_move(hq, sq, fq, eq));
    mhp = wave_sum(mp == kNegInf ? 0.0 : mom_move(hp, spp, fp, ep));
    mx = wave_sum(mq == kNegInf ? 0.0 : mom_move(xq, sq, fq, ep));
  }
  if constexpr (ARGMAX) {
    iq = wave_min((mq == Wq) ? iq : 0x7fffffff);
    ip = wave_min((mp == Wp) ? ip : 0x7fffffff);
  }
  if (lane == 0) {
    sh.m[wv][0] = Wq;
    sh.m[wv][1] = Wp;
    sh.d[wv][0] = dq;
    sh.d[wv][1] = dp;
    sh.i[wv][0] = iq;
    sh.i[wv][1] = ip;
    if constexpr (mom) {
      sh.h[wv][0] = mhq;
      sh.h[wv][1] = mhp;
      sh.h[wv][2] = mx;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float Mq = sh.m[0][0], Mp = sh.m[0][1];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) {
      Mq = fmaxf(Mq, sh.m[w][0]);
      Mp = fmaxf(Mp, sh.m[w][1]);
    }
    const float Rq = Mq * sp.c_hi, Rp = Mp * sp.c_hi;
    double tq = 0.0, tp = 0.0;
    int aq = 0x7fffffff, ap = 0x7fffffff;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float wq_ = sh.m[w][0], wp_ = sh.m[w][1];
      if (wq_ != kNegInf)
        tq += sh.d[w][0] * (double)exp2_hw((float)((double)(wq_ * sp.c_hi) - (double)Rq));
      if (wp_ != kNegInf)
        tp += sh.d[w][1] * (double)exp2_hw((float)((double)(wp_ * sp.c_hi) - (double)Rp));
      if (ARGMAX && wq_ == Mq) aq = min(aq, sh.i[w][0]);
      if (ARGMAX && wp_ == Mp) ap = min(ap, sh.i[w][1]);
    }
    TilePart t;
    t.s_q = tq;
    t.s_p = tp;
    t.r_q = (Mq == kNegInf) ? kNegInf : Rq;
    t.r_p = (Mp == kNegInf) ? kNegInf : Rp;
    t.zmax_q = Mq;
    t.zmax_p = Mp;
    t.amax_q = ARGMAX ? aq : -1;
    t.amax_p = ARGMAX ? ap : -1;
    if constexpr (DEV)
      st_tile(P.tiles + (int64_t)r * P.nt + k, t);
    else
      P.tiles[(int64_t)r * P.nt + k] = t;
    if constexpr (mom) {
      // the waves' moments against the tile references, in wave order
      TileMom m{0.0, 0.0, 0.0};
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float wq_ = sh.m[w][0], wp_ = sh.m[w][1];
        const double gq = (wq_ == kNegInf) ? 0.0 : (double)(wq_ * sp.c_hi) - (double)Rq;
        const double gp = (wp_ == kNegInf) ? 0.0 : (double)(wp_ * sp.c_hi) - (double)Rp;
        const double fq_ = (double)exp2_hw((float)gq), fp_ = (double)exp2_hw((float)gp);
        // a wave's sums d_w are against the wave max, as its moments are
        if (wq_ != kNegInf) mom_add(m.hq, sh.h[w][0], sh.d[w][0], fq_, gq);
        if (wp_ != kNegInf) mom_add(m.hp, sh.h[w][1], sh.d[w][1], fp_, gp);
        if (wq_ != kNegInf)
          mom_add(m.x, sh.h[w][2], sh.d[w][0], fq_, wp_ == kNegInf ? -__builtin_huge_val() : gp);
      }
      P.moms[(int64_t)r * P.nt + k] = m;
    }
  }
}

template <int DT, bool VEC, bool ARGMAX, int MOM>
__device__ __forceinline__ void stats_tile(const Params& P) {
  using T = StatTile<DT, VEC>;
  __shared__ Shared sh;
  const int k = blockIdx.x, r = blockIdx.y;
  const SeqParam sp = seq_param(P, r / (P.gamma + 1));
  // rows that need first moments belong to the moment kernel (block-uniform)
  if (MOM ? !needs_mom(sp) : (P.mom_split && needs_mom(sp))) return;
  const int V = P.V;
  const char* qrow = (const char*)P.q + (int64_t)r * V * T::EB;
  const char* prow = (const char*)P.p + (int64_t)r * V * T::EB;
  const int64_t t0 = (int64_t)k * T::N;
  uint32_t wq[T::U][T::NW], wp[T::U][T::NW];
  load_tile<DT, VEC, T::U, true>(qrow, t0, V, wq, threadIdx.x);
  load_tile<DT, VEC, T::U, true>(prow, t0, V, wp, threadIdx.x);
  tile_partial<DT, VEC, ARGMAX, MOM, false>(P, r, k, sp, wq, wp, sh);
}

template <int DT, bool VEC, bool ARGMAX>
__global__ __launch_bounds__(kThreads) void k_stats(Params P) {
  stats_tile<DT, VEC, ARGMAX, 0>(P);
}

// With first moments, for the rows of BiLD* (temperature > 0) and log-loss
// sequences only; the plain kernel takes every other row.  Held to
// SPC_MOM_OCCUPANCY resident workgroups per CU: left free, the compiler
// keeps every exponential of the tile live at once.
#ifndef SPC_MOM_OCCUPANCY
#define SPC_MOM_OCCUPANCY 6
#endif
template <int DT, bool VEC, bool ARGMAX, int MS>
__global__ __launch_bounds__(kThreads, SPC_MOM_OCCUPANCY) void k_stats_mom(Params P) {
  stats_tile<DT, VEC, ARGMAX, MS>(P);
}

template <int DT, bool VEC, int MS>
void launch_mom(const Params& P, bool argmax, dim3 grid, hipStream_t st) {
  if (argmax)
    hipLaunchKernelGGL((k_stats_mom<DT, VEC, true, MS>), grid, dim3(kThreads), 0, st, P);
  else
    hipLaunchKernelGGL((k_stats_mom<DT, VEC, false, MS>), grid, dim3(kThreads), 0, st, P);
}

// The second-pass weight summed over a thread's entries of one statistics
// tile: for a token rule eta's share (the q mass of the entries the rule
// marks), else max(0, p - q) (D_TV of Lemma 3) in float32.
template <int DT, bool VEC>
__device__ __forceinline__ double pass2_sum(const uint32_t (&wq)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                            const uint32_t (&wp)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                            const ProbScale& ps, bool tok) {
  using T = StatTile<DT, VEC>;
  double acc = 0.0;
#pragma unroll
  for (int i = 0; i < T::U; ++i) {
    float t = 0.0f;
#pragma unroll
    for (int e = 0; e < T::VW; ++e) {
      const float zq = elem<DT, VEC>(wq[i], e), zp = elem<DT, VEC>(wp[i], e);
      if (tok) {
        t += token_r(ps.tok, zq, zp) ? prob(zq, ps.c_hi, ps.c_lo, ps.q_hi, ps.q_lo) : 0.0f;
      } else {
        // D_TV for the deferral decision only, where an absolute error of
        // about 1e-7 is far inside the decision margin; the replacement draw
        // of a rejected row sums its own cancellation-free residual
        const float pq = prob(zq, ps.c_hi, ps.c_lo, ps.q_hi, ps.q_lo);
        const float pp = prob(zp, ps.c_hi, ps.c_lo, ps.p_hi, ps.p_lo);
        t += fmaxf(pp - pq, 0.0f);
      }
    }
    acc += (double)t;
    // one lane load at a time: with the whole tile already in registers the
    // scheduler would otherwise start every entry's exponentials at once
    __builtin_amdgcn_sched_barrier(0);
  }
  return acc;
}

// eta's share of a token-rule tile when the statistics already fix it: the
// rule marks every entry of a tile whose largest logit (p's for TokenV2/V3,
// q's for TokenV1) lies below the threshold, so the share is the tile's q
// mass -- the same expression the sampling pass evaluates for that tile's q
// mass, so the two cancel exactly there -- and a threshold of -inf marks no
// entry.  False when the tile's entries must be visited.
__device__ __forceinline__ bool eta_from_stats(const TokenRule& tr, const TilePart& t,
                                               double lz_q, double* out) {
  if (tr.theta == kNegInf) {
    *out = 0.0;
    return true;
  }
  if ((tr.on_p ? t.zmax_p : t.zmax_q) < tr.theta) {
    *out = t.s_q * exp2_acc((double)t.r_q - lz_q);
    return true;
  }
  return false;
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
  // D_TV rows only: token-rule rows take k_eta
  if (!needs_pass2(sp) || is_token(sp.rule)) return;  // block-uniform
  const int V = P.V;
  const char* qrow = (const char*)P.q + (int64_t)r * V * T::EB;
  const char* prow = (const char*)P.p + (int64_t)r * V * T::EB;
  const int64_t t0 = (int64_t)k * T::N;
  uint32_t wq[T::U][T::NW], wp[T::U][T::NW];
  // D_TV visits every tile: its loads overlap the merge
  load_tile<DT, VEC, T::U, true>(qrow, t0, V, wq, threadIdx.x);
  load_tile<DT, VEC, T::U, true>(prow, t0, V, wp, threadIdx.x);
  if (threadIdx.x < 64) {
    const RowStat rs = merge_row(P, r, false, false);
    if (threadIdx.x == 0) srow = rs;
  }
  __syncthreads();
  double acc = pass2_sum<DT, VEC>(wq, wp, prob_scale(sp, srow, false), false);
  double unused = 0.0;
  block_sum2(acc, unused, sh);
  if (threadIdx.x == 0) P.tvpart[(int64_t)r * P.nt + k] = acc;
}

// Eta pass (token-rule rows at temperature > 0).  grid (ceil(nt /
// kEtaTiles), R): a workgroup merges row r once and takes its tiles
// x kEtaTiles .. + kEtaTiles - 1 in turn.  A tile wholly below the rule's
// threshold takes its share from the statistics (eta_from_stats); any other
// tile is read again and summed exactly as by the TV pass's tile code.
constexpr int kEtaTiles = 8;

template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void k_eta(Params P) {
  using T = StatTile<DT, VEC>;
  __shared__ Shared sh;
  __shared__ RowStat srow;
  const int r = blockIdx.y;
  const SeqParam sp = seq_param(P, r / (P.gamma + 1));
  if (!needs_pass2(sp) || !is_token(sp.rule)) return;  // block-uniform
  const int V = P.V, nt = P.nt;
  const char* qrow = (const char*)P.q + (int64_t)r * V * T::EB;
  const char* prow = (const char*)P.p + (int64_t)r * V * T::EB;
  if (threadIdx.x < 64) {
    const RowStat rs = merge_row(P, r, false, false);
    if (threadIdx.x == 0) srow = rs;
  }
  __syncthreads();
  const ProbScale ps = prob_scale(sp, srow, true);
  const int k1 = min(nt, ((int)blockIdx.x + 1) * kEtaTiles);
  for (int k = (int)blockIdx.x * kEtaTiles; k < k1; ++k) {  // block-uniform
    double eta;
    if (eta_from_stats(ps.tok, P.tiles[(int64_t)r * nt + k], srow.lz_q, &eta)) {
      if (threadIdx.x == 0) P.tvpart[(int64_t)r * nt + k] = eta;
      continue;
    }
    uint32_t wq[T::U][T::NW], wp[T::U][T::NW];
    load_tile<DT, VEC, T::U, true>(qrow, (int64_t)k * T::N, V, wq, threadIdx.x);
    load_tile<DT, VEC, T::U, true>(prow, (int64_t)k * T::N, V, wp, threadIdx.x);
    double acc = pass2_sum<DT, VEC>(wq, wp, ps, true);
    double unused = 0.0;
    block_sum2(acc, unused, sh);
    if (threadIdx.x == 0) P.tvpart[(int64_t)r * nt + k] = acc;
    __syncthreads();  // the block's shared scratch is reused by the next tile
  }
}

// ------------------------------------------- one read for the second pass
// Statistics and the second pass in one launch, for batches whose rows need
// no first moments.  A resident grid of G workgroups (G a multiple of nt,
// all co-resident: a cooperative launch) takes tiles t = g, g + G, ... in
// row-major order, so the nt tiles of a row always fall in one round of G.
// A workgroup computes its tile's partial; on a row that needs the second
// pass it then waits for the row's other nt - 1 partials (a per-row arrival
// counter), merges them, and sums the TV or eta weight over the entries it
// still holds in registers, so the row is read from HBM once.  The wait is
// bounded: a workgroup that gives up writes a NaN partial, which makes its
// sequence invalid (the sampling pass reports -1), instead of hanging.
// Measured on MI355X it is slower than the second read it saves (each round
// of resident tiles waits through publish, arrival and merge with its loads
// idle, and a cooperative launch costs more to start), so it runs only on
// request.
constexpr uint32_t kRowSpinLimit = 1u << 16;  // about 0.1 s

// Thread 0 has written the tile's partial (agent-scope stores).  Arrive on
// the row's counter and wait until all n tiles have; returns false after the
// spin limit.
__device__ __forceinline__ bool row_arrive_wait(uint32_t* cnt, uint32_t n, Shared& sh) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    vmem_drain();  // the partial's stores are complete
    uint32_t seen =
        __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u;
    uint32_t it = 0;
    while (seen < n && it < kRowSpinLimit) {
      __builtin_amdgcn_s_sleep(2);
      seen = __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      ++it;
    }
    sh.flag = seen >= n;
  }
  __syncthreads();
  const bool ok = sh.flag;
  vmem_drain();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  return ok;
}

// Leave the row: the last of its n tiles to leave resets both counters
// (every tile has arrived and stopped waiting by then).
__device__ __forceinline__ void row_depart(uint32_t* cnt, uint32_t n) {
  if (threadIdx.x == 0) {
    const uint32_t prev =
        __hip_atomic_fetch_add(cnt + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == n - 1) {
      __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(cnt + 1, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Held to SPC_RES_OCCUPANCY resident workgroups per CU (no spill at 5).
#ifndef SPC_RES_OCCUPANCY
#define SPC_RES_OCCUPANCY 5
#endif
template <int DT, bool VEC, bool ARGMAX>
__global__ __launch_bounds__(kThreads, SPC_RES_OCCUPANCY) void k_stats_res(Params P) {
  using T = StatTile<DT, VEC>;
  __shared__ Shared sh;
  __shared__ RowStat srow;
  const int nt = P.nt, V = P.V;
  const int64_t ntiles = (int64_t)P.B * (P.gamma + 1) * nt;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {  // block-uniform
    const int r = (int)(t / nt), k = (int)(t - (int64_t)r * nt);
    const SeqParam sp = seq_param(P, r / (P.gamma + 1));
    const char* qrow = (const char*)P.q + (int64_t)r * V * T::EB;
    const char* prow = (const char*)P.p + (int64_t)r * V * T::EB;
    // the thread's load offsets are recomputed per tile rather than held
    // across the loop in registers
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    uint32_t wq[T::U][T::NW], wp[T::U][T::NW];
    load_tile<DT, VEC, T::U, true>(qrow, (int64_t)k * T::N, V, wq, tid);
    load_tile<DT, VEC, T::U, true>(prow, (int64_t)k * T::N, V, wp, tid);
    tile_partial<DT, VEC, ARGMAX, 0, true>(P, r, k, sp, wq, wp, sh);
    if (needs_pass2(sp)) {  // block-uniform
      // only the packed words stay live across the wait: left free, the
      // compiler keeps every unpacked entry of the statistics for reuse
#pragma unroll
      for (int i = 0; i < T::U; ++i)
#pragma unroll
        for (int j = 0; j < T::NW; ++j) asm volatile("" : "+v"(wq[i][j]), "+v"(wp[i][j]));
      uint32_t* cnt = P.row_cnt + (int64_t)r * kRowCntStride;
      const bool ok = row_arrive_wait(cnt, (uint32_t)nt, sh);
      if (threadIdx.x < 64) {
        const RowStat rs = merge_row<true>(P, r, false, false, 0, load_head<true>(P, r, false, false));
        if (threadIdx.x == 0) srow = rs;
      }
      __syncthreads();
      const bool tok = is_token(sp.rule);
      const ProbScale ps = prob_scale(sp, srow, tok);
      double eta;
      if (tok && eta_from_stats(ps.tok, ld_tile(P.tiles + (int64_t)r * nt + k), srow.lz_q,
                                &eta)) {
        if (threadIdx.x == 0) P.tvpart[(int64_t)r * nt + k] = ok ? eta : __builtin_nan("");
      } else {
        double acc = pass2_sum<DT, VEC>(wq, wp, ps, tok);
        double unused = 0.0;
        block_sum2(acc, unused, sh);
        if (threadIdx.x == 0)
          P.tvpart[(int64_t)r * nt + k] = ok ? acc : __builtin_nan("");
      }
      row_depart(cnt, (uint32_t)nt);
    }
    __syncthreads();  // the block's shared scratch is reused by the next tile
  }
}

// Sampling pass.  grid (K, B) of 1024-thread workgroups: every workgroup of
// sequence b merges the sequence's rows and decides it (workgroup 0 writes
// the outputs).  A replacement drawn from a residual needs that row's
// residual masses: the K workgroups sum them chunk by chunk, and the last to
// finish draws.  Every other draw -- the extra token from q, p or a token
// rule's target, whose per-tile masses the earlier passes left -- is made by
// workgroup 0 alone.
template <int DT, bool VEC>
__global__ __launch_bounds__(kSampThreads) void k_sample(Params P) {
  __shared__ SampShared sh;
  __shared__ SeqShared ss;
  const int k = blockIdx.x, b = blockIdx.y;
  const SeqParam sp = seq_param(P, b);
  decide_seq<DT>(P, b, sp, ss, k == 0);
  const SeqState s = ss.seq;
  if (s.kind == kNone) return;  // block-uniform
  const int64_t row = (int64_t)b * (P.gamma + 1) + s.row;
  const RowStat rs = ss.rows[s.row].rs;
  const bool pass = s.kind == kTokRes || s.kind == kResidual;
  if (!pass) {
    if (k != 0) return;  // block-uniform
    const int src = s.kind == kQ ? kSrcStatsQ : s.kind == kP ? kSrcStatsP : kSrcTokPi;
    draw<DT, VEC>(P, b, row, s.kind, src, s.u, sp, rs, ss, sh);
    return;
  }
  constexpr int EB = StatTile<DT, VEC>::EB;
  const ProbScale ps = prob_scale(sp, rs, s.kind == kTokRes);
  const char* qrow = (const char*)P.q + row * P.V * EB;
  const char* prow = (const char*)P.p + row * P.V * EB;
  double* masses = P.masses + (int64_t)b * P.nc;
  if (s.kind == kTokRes)
    residual_masses<DT, VEC, kTokRes>(qrow, prow, P.V, P.nc, P.K, k, ps, masses);
  else
    residual_masses<DT, VEC, kResidual>(qrow, prow, P.V, P.nc, P.K, k, ps, masses);
  if (!arrive_last(P.samp_cnt + b, (uint32_t)P.K, sh)) return;
  draw<DT, VEC>(P, b, row, s.kind, kSrcPass, s.u, sp, rs, ss, sh);
}

// Drafter sampling step (Alg. 4: x_{t+j} ~ q_{t+j}), one launch.  grid
// (nt, B): statistics tile k of row b of the drafter's logits, as in k_stats
// for one tensor.  The last tile of a row to finish (a per-row counter on a
// line of its own) merges the row's partials and draws the token: the tile
// masses give the tile where u W falls, then the tile's sub-chunks and
// lanes are scanned in vocabulary order.  A greedy row (temperature 0)
// takes the lowest index attaining its max instead.
template <int DT, bool VEC, bool ARGMAX, int TM>
__global__ __launch_bounds__(kThreads) void k_draft(Params P) {
  using T = DraftTile<DT, VEC, TM>;
  __shared__ Shared sh;
  __shared__ RowStat srow;
  __shared__ PickState pks;
  const int k = blockIdx.x, b = blockIdx.y;
  const SeqParam sp = seq_param(P, b);
  const int V = P.V;
  const char* row = (const char*)P.q + (int64_t)b * V * T::EB;
  const int64_t t0 = (int64_t)k * T::N;
  uint32_t w[T::U][T::NW];
  load_tile<DT, VEC, T::U, true>(row, t0, V, w, threadIdx.x);
  float g[T::U];
#pragma unroll
  for (int i = 0; i < T::U; ++i) {
    float a = kNegInf;
#pragma unroll
    for (int e = 0; e < T::VW; ++e) a = fmaxf(a, elem<DT, VEC>(w[i], e));
    g[i] = a;
  }
  float m = g[0];
#pragma unroll
  for (int i = 1; i < T::U; ++i) m = fmaxf(m, g[i]);
  int im = 0x7fffffff;
  const int base = (int)t0 + (int)threadIdx.x * T::VW;
  if constexpr (ARGMAX) {
    im = first_max_index<DT, VEC, T::U, kThreads>(w, g, m, base);
    // unpack again for the sums rather than hold every entry with the words
#pragma unroll
    for (int i = 0; i < T::U; ++i)
#pragma unroll
      for (int j = 0; j < T::NW; ++j) asm volatile("" : "+v"(w[i][j]));
  }
  const float r = (m == kNegInf) ? 0.0f : m * sp.c_hi;
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < T::U; ++i) {
    float t[T::VW];
#pragma unroll
    for (int e = 0; e < T::VW; ++e) {
      const float z = elem<DT, VEC>(w[i], e);
      t[e] = exp2_hw(fmaf(z, sp.c_lo, fmaf(z, sp.c_hi, -r)));
    }
#pragma unroll
    for (int h = 1; h < T::VW; h <<= 1)
#pragma unroll
      for (int e = 0; e + h < T::VW; e += 2 * h) t[e] += t[e + h];
    s += t[0];
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const float Wm = wave_max(m);
  double d = (m == kNegInf)
                 ? 0.0
                 : (double)s * (double)exp2_hw((float)((double)r - (double)(Wm * sp.c_hi)));
  d = wave_sum(d);
  if constexpr (ARGMAX) im = wave_min((m == Wm) ? im : 0x7fffffff);
  if (lane == 0) {
    sh.m[wv][0] = Wm;
    sh.d[wv][0] = d;
    sh.i[wv][0] = im;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float M = sh.m[0][0];
#pragma unroll
    for (int x = 1; x < kWaves; ++x) M = fmaxf(M, sh.m[x][0]);
    const float R = M * sp.c_hi;
    double tot = 0.0;
    int am = 0x7fffffff;
#pragma unroll
    for (int x = 0; x < kWaves; ++x) {
      const float wm = sh.m[x][0];
      if (wm != kNegInf)
        tot += sh.d[x][0] * (double)exp2_hw((float)((double)(wm * sp.c_hi) - (double)R));
      if (ARGMAX && wm == M) am = min(am, sh.i[x][0]);
    }
    TilePart t{tot, 0.0, (M == kNegInf) ? kNegInf : R, kNegInf, M, kNegInf,
               ARGMAX ? am : -1, -1};
    st_tile(P.tiles + (int64_t)b * P.nt + k, t);
  }
  if (!arrive_last(P.samp_cnt + (int64_t)b * kDraftCntStride, (uint32_t)P.nt, sh)) return;
  // the last tile of row b: merge the row (wave 0, a tile per lane)
  if (threadIdx.x < 64) {
    TilePart h{0.0, 0.0, kNegInf, kNegInf, kNegInf, kNegInf, 0x7fffffff, 0x7fffffff};
    float zq = kNegInf, rq = kNegInf;
    for (int kk = lane; kk < P.nt; kk += 64) {
      const TilePart tk = ld_tile(P.tiles + (int64_t)b * P.nt + kk);
      zq = fmaxf(zq, tk.zmax_q);
      rq = fmaxf(rq, tk.r_q);
    }
    zq = wave_max(zq);
    rq = wave_max(rq);
    double sq = 0.0;
    int aq = 0x7fffffff;
    for (int kk = lane; kk < P.nt; kk += 64) {
      h = ld_tile(P.tiles + (int64_t)b * P.nt + kk);
      sq += h.s_q * exp2_acc((double)h.r_q - (double)rq);
      if (ARGMAX && h.zmax_q == zq) aq = min(aq, h.amax_q);
    }
    sq = wave_sum(sq);
    if constexpr (ARGMAX) aq = wave_min(aq);
    if (threadIdx.x == 0) {
      RowStat rs{};
      rs.lz_q = (double)rq + log2_acc(sq);
      rs.zmax_q = zq;
      rs.amax_q = ARGMAX ? aq : -1;
      srow = rs;
    }
  }
  __syncthreads();
  const RowStat rs = srow;
  if (!sp.valid || sp.greedy) {  // block-uniform
    if (threadIdx.x == 0) P.out_token[b] = sp.valid ? rs.amax_q : -1;
    return;
  }
  if (threadIdx.x < 64) {
    int ks;
    double rem;
    find_part<kSrcDraft>(P, b, b, P.nt, rs, P.uniforms[b], &ks, &rem);
    if (threadIdx.x == 0) {
      pks = PickState{ks, kQ, kSrcDraft, rem};
      if (ks < 0) P.out_token[b] = -1;
    }
  }
  __syncthreads();
  const PickState pk = pks;
  if (pk.k < 0) return;  // block-uniform
  pick_tile<DT, VEC, kQ, kWaves, T::N>(P, b, b, (int64_t)pk.k * T::N, pk.rem, prob_scale(sp, rs),
                                       sh);
}

template <int DT, bool VEC, int TM>
hipError_t launch_draft_t(const Params& P, bool argmax, hipStream_t st) {
  const dim3 grid(P.nt, P.B);
  if (argmax)
    hipLaunchKernelGGL((k_draft<DT, VEC, true, TM>), grid, dim3(kThreads), 0, st, P);
  else
    hipLaunchKernelGGL((k_draft<DT, VEC, false, TM>), grid, dim3(kThreads), 0, st, P);
  return hipGetLastError();
}

template <int DT, bool VEC, bool ARGMAX>
const void* res_kernel() {
  return reinterpret_cast<const void*>(&k_stats_res<DT, VEC, ARGMAX>);
}

template <int DT, bool VEC>
const void* res_kernel(bool argmax) {
  return argmax ? res_kernel<DT, VEC, true>() : res_kernel<DT, VEC, false>();
}

template <int DT, bool VEC>
hipError_t launch_t(const Params& P, int tv_kinds, bool need_sample, bool need_argmax,
                    bool need_plain, bool need_mom, int res_grid, hipEvent_t e0, hipEvent_t e1,
                    hipStream_t st) {
  const unsigned R = (unsigned)(P.B * (P.gamma + 1));
  const dim3 grid(P.nt, R);
  hipError_t err;
  if (e0 && (err = hipEventRecord(e0, st)) != hipSuccess) return err;
  if (res_grid > 0 && tv_kinds && !need_mom) {
    // statistics and second pass, one read: every workgroup must be resident
    void* args[] = {const_cast<Params*>(&P)};
    err = hipLaunchCooperativeKernel(res_kernel<DT, VEC>(need_argmax), dim3((unsigned)res_grid),
                                     dim3(kThreads), args, 0, st);
    if (err == hipSuccess) {
      if (e1 && (err = hipEventRecord(e1, st)) != hipSuccess) return err;
      hipLaunchKernelGGL((k_sample<DT, VEC>), dim3(need_sample ? P.K : 1, P.B),
                         dim3(kSampThreads), 0, st, P);
      return hipGetLastError();
    }
    if (err != hipErrorCooperativeLaunchTooLarge && err != hipErrorNotSupported) return err;
    (void)hipGetLastError();  // not launchable here: the two-kernel path below
  }
  if (need_plain) {
    if (need_argmax)
      hipLaunchKernelGGL((k_stats<DT, VEC, true>), grid, dim3(kThreads), 0, st, P);
    else
      hipLaunchKernelGGL((k_stats<DT, VEC, false>), grid, dim3(kThreads), 0, st, P);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  if (need_mom) {
    // the moments the batch's rules read: x alone (BiLD*), H_q alone
    // (ChowLog), or all three
    if (P.mom_set == kMomX)
      launch_mom<DT, VEC, kMomX>(P, need_argmax, grid, st);
    else if (P.mom_set == kMomHQ)
      launch_mom<DT, VEC, kMomHQ>(P, need_argmax, grid, st);
    else
      launch_mom<DT, VEC, kMomX | kMomHQ | kMomHP>(P, need_argmax, grid, st);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  if (e1 && (err = hipEventRecord(e1, st)) != hipSuccess) return err;
  if (tv_kinds & kPassTv) {
    hipLaunchKernelGGL((k_tv<DT, VEC>), dim3(P.nt, R), dim3(kThreads), 0, st, P);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  if (tv_kinds & kPassEta) {
    hipLaunchKernelGGL((k_eta<DT, VEC>), dim3((P.nt + kEtaTiles - 1) / kEtaTiles, R),
                       dim3(kThreads), 0, st, P);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  // a batch with no sequence at temperature > 0 only needs the decisions
  hipLaunchKernelGGL((k_sample<DT, VEC>), dim3(need_sample ? P.K : 1, P.B), dim3(kSampThreads), 0,
                     st, P);
  return hipGetLastError();
}

}  // namespace

int stat_tile_elems(int dtype, bool vec) {
  if (dtype == 1) return vec ? StatTile<1, true>::N : StatTile<1, false>::N;
  return vec ? StatTile<0, true>::N : StatTile<0, false>::N;
}

int draft_tile_elems(int dtype, bool vec, bool long_tiles) {
  if (long_tiles) {
    if (dtype == 1) return vec ? DraftTile<1, true, 2>::N : DraftTile<1, false, 2>::N;
    return vec ? DraftTile<0, true, 2>::N : DraftTile<0, false, 2>::N;
  }
  if (dtype == 1) return vec ? DraftTile<1, true, 1>::N : DraftTile<1, false, 1>::N;
  return vec ? DraftTile<0, true, 1>::N : DraftTile<0, false, 1>::N;
}

int samp_chunk_elems(int dtype, bool vec) {
  if (dtype == 1) return vec ? SampChunk<1, true>::N : SampChunk<1, false>::N;
  return vec ? SampChunk<0, true>::N : SampChunk<0, false>::N;
}

// Enough workgroups to give every compute unit one (a sampling workgroup
// fills a CU), but no more than one chunk per wavefront: small batches spread
// a row over several workgroups, large ones take one per sequence and loop.
int samp_groups(int64_t nc, int B, int cus) {
  const int64_t by_chunks = (nc + kSampWaves - 1) / kSampWaves;
  const int64_t by_cus = (cus + B - 1) / B;
  const int64_t k = by_chunks < by_cus ? by_chunks : by_cus;
  return (int)(k < 1 ? 1 : k);
}

hipError_t launch_draft(const Params& P, int dtype, bool vec, bool argmax, bool long_tiles,
                        hipStream_t st) {
  if (long_tiles) {
    if (dtype == 1)
      return vec ? launch_draft_t<1, true, 2>(P, argmax, st)
                 : launch_draft_t<1, false, 2>(P, argmax, st);
    return vec ? launch_draft_t<0, true, 2>(P, argmax, st)
               : launch_draft_t<0, false, 2>(P, argmax, st);
  }
  if (dtype == 1)
    return vec ? launch_draft_t<1, true, 1>(P, argmax, st)
               : launch_draft_t<1, false, 1>(P, argmax, st);
  return vec ? launch_draft_t<0, true, 1>(P, argmax, st) : launch_draft_t<0, false, 1>(P, argmax, st);
}

hipError_t launch_verify(const Params& P, int dtype, bool vec, int tv_kinds, bool need_sample,
                         bool need_argmax, bool need_plain, bool need_mom, int res_grid,
                         hipEvent_t e0, hipEvent_t e1, hipStream_t st) {
  if (dtype == 1) {
    return vec ? launch_t<1, true>(P, tv_kinds, need_sample, need_argmax, need_plain, need_mom,
                                   res_grid, e0, e1, st)
               : launch_t<1, false>(P, tv_kinds, need_sample, need_argmax, need_plain, need_mom,
                                    res_grid, e0, e1, st);
  }
  return vec ? launch_t<0, true>(P, tv_kinds, need_sample, need_argmax, need_plain, need_mom,
                                 res_grid, e0, e1, st)
             : launch_t<0, false>(P, tv_kinds, need_sample, need_argmax, need_plain, need_mom,
                                  res_grid, e0, e1, st);
}

int res_blocks_per_cu(int dtype, bool vec, bool argmax) {
  // per variant; queried once per process (every device here is the same part)
  static int cache[2][2][2] = {{{-1, -1}, {-1, -1}}, {{-1, -1}, {-1, -1}}};
  int& c = cache[dtype == 1][vec][argmax];
  if (c < 0) {
    const void* f = dtype == 1 ? (vec ? res_kernel<1, true>(argmax) : res_kernel<1, false>(argmax))
                               : (vec ? res_kernel<0, true>(argmax) : res_kernel<0, false>(argmax));
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, f, kThreads, 0) != hipSuccess) {
      (void)hipGetLastError();
      nb = 0;
    }
    c = nb;
  }
  return c;
}

}  // namespace spc
