// spc_kernels.hip -- gfx950 kernels of the speculative-cascade verify step.
//
// The step (GenSpecSample, Alg. 4, with the cascade target T_delta of eq. (6)
// and the deferral rules of Table 1) runs as a statistics launch and one or
// two job launches; no workgroup ever waits for another.  A row is one
// position (b, j) of the logit pair (q, p); rows are cut into statistics
// tiles of consecutive vocabulary entries.
//
//   k_tiles      grid (tile, row).  A tile reduces its entries of q and p to
//                {max z, sum 2^(z c - r)} (c = log2(e) / T); its first
//                wavefront then arrives on the row's counter, and the last
//                tile of the row merges the row.  Then, per row:
//                  OPT / OPTLOG at T > 0   publishes a TV job (D_TV of Lemma 3
//                                          needs both normalisers: one chunk
//                                          per tile, the row read again);
//                  token rules at T > 0    settles eta (Alg. 6) for the tiles
//                                          wholly below the rule's threshold
//                                          from their statistics and
//                                          publishes a job for the others;
//                  T = 0                   publishes the two halves of its
//                                          argmax (the lowest index of a row
//                                          maximum lies in the first tile
//                                          whose maximum it is);
//                  otherwise               decides the row at once.
//   row decision delta_j and a_j of the row, then an atomic OR of the row into
//                its sequence's decided-row mask.  The decision that completes
//                the prefix 0..j* of decided rows containing the first
//                rejection j* finishes the sequence: the greedy token, or a
//                draw published to the next job pass (from the statistics
//                partials, for an extra token from q, p or a token rule's
//                target; else a residual job over row j*).
//   k_jobs       a static walk over the jobs the launches before it
//                published: every chunk of every row job, then the single
//                jobs.  The last chunk of a job continues it (the row's
//                decision, which may publish to the next pass, or the
//                residual draw).
//
// Draws are inverse CDF in vocabulary order.  Merges and sums run in fixed
// orders, so results do not depend on scheduling.  Counters sit in a zeroed
// region of the workspace and every launch leaves them at zero: arrival
// counters are reset by their last arrival, a pass's job counts by the last
// of its workgroups to read them.  So a call replayed from a graph finds the
// counters as the captured call did.
#include <math.h>

#include <algorithm>

#include "spc_internal.h"

namespace spc {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr double kLog2e = 1.4426950408889634074;  // log2(e)
constexpr double kLn2 = 0.69314718055994530942;   // ln(2)

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = kThreads / 64;

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
// Entries at or past `end` read as -inf; a lane past the end re-reads the
// tile's first entry and discards the value, so the loads are branch-free.
// With MASK false the caller guarantees a whole tile before `end`.  Addresses
// are a uniform tile base plus a 32-bit lane offset.
template <int DT, bool VEC, int U, bool NT, int GT = kThreads, bool MASK = true>
__device__ __forceinline__ void load_tile(const char* row, int64_t t0, int64_t end,
                                          uint32_t (&w)[U][Tile<DT, VEC, U>::NW], int tid) {
  using T = Tile<DT, VEC, U>;
  constexpr uint32_t kPad = (DT == 1) ? 0xff80ff80u : 0xff800000u;
  constexpr int kSpan = GT * U * T::VW;  // entries of a whole tile
  const char* base = row + t0 * T::EB;
  const int left = (int)(end - t0 < (int64_t)kSpan ? end - t0 : (int64_t)kSpan);
  const bool full = !MASK || left == kSpan;
#pragma unroll
  for (int i = 0; i < U; ++i) {
    const int e = (i * GT + tid) * T::VW;
    const bool ok = full || e < left;
    const char* a = base + (uint32_t)((ok ? e : 0) * T::EB);
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

// First moments of a tile, written and read within one launch.
static_assert(sizeof(TileMom) == 24, "TileMom is three doubles");
__device__ __forceinline__ void st_mom(TileMom* dst, const TileMom& m) {
  st_dev_f64(&dst->hq, m.hq);
  st_dev_f64(&dst->hp, m.hp);
  st_dev_f64(&dst->x, m.x);
}
__device__ __forceinline__ TileMom ld_mom(const TileMom* src) {
  return TileMom{ld_dev_f64(&src->hq), ld_dev_f64(&src->hp), ld_dev_f64(&src->x)};
}

// Merged row statistics, written and read within one launch: six 64-bit words.
static_assert(sizeof(RowStat) == 48, "RowStat is six 64-bit words");
__device__ __forceinline__ void st_rowstat(RowStat* dst, const RowStat& s) {
  uint64_t w[6];
  __builtin_memcpy(w, &s, sizeof w);
#pragma unroll
  for (int i = 0; i < 6; ++i)
    __hip_atomic_store(reinterpret_cast<uint64_t*>(dst) + i, w[i], __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ RowStat ld_rowstat(const RowStat* src) {
  uint64_t w[6];
#pragma unroll
  for (int i = 0; i < 6; ++i)
    w[i] = __hip_atomic_load(reinterpret_cast<uint64_t*>(const_cast<RowStat*>(src)) + i,
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  RowStat s;
  __builtin_memcpy(&s, w, sizeof w);
  return s;
}

// 32- and 64-bit words shared within one launch (agent scope, relaxed).
__device__ __forceinline__ uint32_t ld_u32(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_u32(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_u64(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_u64(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t ld_i32(const int32_t* p) {
  return (int32_t)ld_u32(reinterpret_cast<const uint32_t*>(p));
}
__device__ __forceinline__ void st_i32(int32_t* p, int32_t v) {
  st_u32(reinterpret_cast<uint32_t*>(p), (uint32_t)v);
}
__device__ __forceinline__ uint32_t add_u32(uint32_t* p, uint32_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t xchg_u32(uint32_t* p, uint32_t v) {
  return __hip_atomic_exchange(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void max_u32(uint32_t* p, uint32_t v) {
  (void)__hip_atomic_fetch_max(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t or_u64(uint64_t* p, uint64_t v) {
  return __hip_atomic_fetch_or(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
__device__ __forceinline__ RowStat lane_rowstat(const RowStat& x, int l) {
  RowStat y;
  y.lz_q = lane_f64(x.lz_q, l);
  y.lz_p = lane_f64(x.lz_p, l);
  y.tv = lane_f64(x.tv, l);
  y.slog = lane_f64(x.slog, l);
  y.zmax_q = lane_f32(x.zmax_q, l);
  y.zmax_p = lane_f32(x.zmax_p, l);
  y.amax_q = lane_i32(x.amax_q, l);
  y.amax_p = lane_i32(x.amax_p, l);
  return y;
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

// Merged statistics and decision of one row of a sequence.
struct RowDecision {
  RowStat rs;
  float maxq, maxp, tv;  // inputs of the deferral rule
  float u;               // the row's uniform
  int delta, keep;       // delta_j and a_j
};

// The part of a draw found by wave 0, for the whole workgroup.
struct PickState {
  int k;       // part holding the sample (-1: nothing to draw)
  int kind;    // SampleKind actually sampled
  int src;     // MassSrc of the part masses
  double rem;  // target mass remaining at the start of that part
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
// Temperatures below 2^-107 are taken as 2^-107: z / T then stays finite in
// float32 for logits up to about 10^6 in magnitude, and the tempered softmax
// is already the T -> 0 limit (uniform over the tied maxima) for any logits
// whose distinct values differ by more than about 10^-30.
constexpr double kTempFloor = 0x1p-107;

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
            isfinite(T) && T >= 0.0f && (s.rule != SPC_RULE_LOSSY || alpha < 1.0f) &&
            (!P.rule_ps || !P.rule_mask || ((P.rule_mask >> s.rule) & 1u));
  s.greedy = P.force_greedy || T == 0.0f;
  s.c = kLog2e / ((s.greedy || !s.valid) ? 1.0 : fmax((double)T, kTempFloor));
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
  return ps;
}

__device__ __forceinline__ float prob(float z, float c_hi, float c_lo, float l_hi, float l_lo) {
  return exp2_hw(fmaf(z, c_hi, -l_hi) + fmaf(z, c_lo, -l_lo));
}

// Residual weight max(0, p_v - q_v) of a replacement draw, as the plain
// difference of the two probabilities.  Where p_v ~ q_v the difference loses
// relative precision, but its absolute error stays at a float32 ulp of p_v:
// over a draw's cumulative masses that is far below the errors the shared
// log-normalisers already carry (about 2e-8 of the mass).  A form through
// the log-ratio keeps full relative precision per entry but costs a
// polynomial and two selects more per entry, in the pass that sums every
// entry of row j*.  A masked logit (-inf) gives probability 0 on its side
// (c_lo > 0), so the weight is p_v or 0 as it should be.
template <int DT>
__device__ __forceinline__ float residual_weight(float zq, float zp, const ProbScale& s) {
  const float pq = prob(zq, s.c_hi, s.c_lo, s.q_hi, s.q_lo);
  const float pp = prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
  return fmaxf(pp - pq, 0.0f);
}

// Weight of one entry under a sampled distribution.  With a token rule the p
// scale carries eta (prob_scale): the residual max(0, pi - q) of Alg. 6's
// target is p eta where r = 0 and max(0, p eta - q) where r = 1 (the plain
// difference, as in residual_weight), and the target itself is p eta where
// r = 1 and q + p eta where r = 0.
template <int DT, int KIND>
__device__ __forceinline__ float weight_of(float zq, float zp, const ProbScale& s) {
  if constexpr (KIND == kQ) {
    return prob(zq, s.c_hi, s.c_lo, s.q_hi, s.q_lo);
  } else if constexpr (KIND == kP) {
    return prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
  } else if constexpr (KIND == kResidual) {
    return residual_weight<DT>(zq, zp, s);
  } else if constexpr (KIND == kTokRes) {
    const float pe = prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
    return token_r(s.tok, zq, zp) ? fmaxf(pe - prob(zq, s.c_hi, s.c_lo, s.q_hi, s.q_lo), 0.0f)
                                  : pe;
  } else {
    const float pe = prob(zp, s.c_hi, s.c_lo, s.p_hi, s.p_lo);
    const float qe = prob(zq, s.c_hi, s.c_lo, s.q_hi, s.q_lo);
    return token_r(s.tok, zq, zp) ? pe : qe + pe;
  }
}

template <int DT, int KIND>
__device__ __forceinline__ float weight_k(float zq, float zp, const ProbScale& s, int) {
  return weight_of<DT, KIND>(zq, zp, s);
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

// The deferral decision of an OPT or OPTLOG row at T > 0 when D_TV cannot
// change it, else -1.  D_TV lies in [lo, 1] (lo a lower bound that the
// computed D_TV cannot undercut), so the threshold of eq. (11) (max p -
// alpha D_TV) or of OPTLog (alpha D_TV) ranges between its values at the two
// ends; rounding is monotone, so the comparison decide_row makes with any
// D_TV in [lo, 1] agrees with the one made at both ends.
__device__ __forceinline__ int tv_free_decision(const SeqParam& sp, const RowStat& rs,
                                                double lo) {
  const double a = sp.alpha;
  if (sp.rule == SPC_RULE_OPT) {
    const double maxq = exp2_acc((double)rs.zmax_q * sp.c - rs.lz_q);
    const double maxp = exp2_acc((double)rs.zmax_p * sp.c - rs.lz_p);
    const double t0 = maxp - a * lo, t1 = maxp - a * 1.0;
    if (maxq < fmin(t0, t1)) return 1;
    if (!(maxq < fmax(t0, t1))) return 0;
    return -1;
  }
  const double t0 = a * lo, t1 = a * 1.0;  // OPTLOG: slog > alpha D_TV
  if (rs.slog > fmax(t0, t1)) return 1;
  if (!(rs.slog > fmin(t0, t1))) return 0;
  return -1;
}

// ------------------------------------------------------------- row merge
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

// Wave 0 merges the nt tile partials of row r (written earlier in the same
// launch) in a fixed order: lane l takes tiles l, l + 64, ...; butterflies
// combine the lanes.  With mrule (a log-loss rule or BiLD*) it also forms the
// rule's statistic from the tiles' first moments: against the row references,
//   H(q) = ln 2 (log2 S_q - H_q / S_q),  H(p) = ln 2 (log2 S_p - H_p / S_p),
//   D(q, p) = -sum q log p = ln 2 (log2 S_p - X / S_q),
// each a sum of two non-negative terms.  kq / kp: the first tile whose
// largest logit is the row's (it holds the lowest index of the row maximum),
// as k * 16 + the mask of the tile's slices that attain it.
// tv_low (rows of at most 64 tiles, else 0): half the L1 distance between
// the tile masses of p and q, a lower bound on D_TV (merging entries into
// tiles can only shrink the distance).
// Every lane returns the same RowStat.
__device__ __forceinline__ RowStat merge_row(const Params& P, int r, int mrule, int* kq_out,
                                             int* kp_out, bool want_low, double& tv_low) {
  const int lane = threadIdx.x & 63;
  const int nt = P.nt;
  const TilePart* tp = P.tiles + (int64_t)r * nt;
  const TileMom* mp = P.moms + (int64_t)r * nt;
  TilePart t0{0.0, 0.0, kNegInf, kNegInf, kNegInf, kNegInf, -1, -1};
  TileMom m0{0.0, 0.0, 0.0};
  if (lane < nt) {
    t0 = ld_tile(tp + lane);
    if (mrule) m0 = ld_mom(mp + lane);
  }
  float zq = t0.zmax_q, zp = t0.zmax_p, rq = t0.r_q, rp = t0.r_p;
  for (int k = lane + 64; k < nt; k += 64) {
    const TilePart tk = ld_tile(tp + k);
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
  int kq = 0x7fffffff, kp = 0x7fffffff;
  auto add = [&](const TilePart& tk, const TileMom& mk, int k) {
    // r_k - r is exact in fp64; an all -inf tile has s = 0
    const double gq = (double)tk.r_q - (double)rq, gp = (double)tk.r_p - (double)rp;
    const double fq = exp2_acc(gq), fp = exp2_acc(gp);
    sq += tk.s_q * fq;
    sp += tk.s_p * fp;
    if (tk.zmax_q == zq) kq = min(kq, k);
    if (tk.zmax_p == zp) kp = min(kp, k);
    if (mrule) {
      mom_add(mhq, mk.hq, tk.s_q, fq, gq);
      mom_add(mhp, mk.hp, tk.s_p, fp, gp);
      mom_add(mx, mk.x, tk.s_q, fq, gp);
    }
  };
  if (lane < nt) add(t0, m0, lane);
  for (int k = lane + 64; k < nt; k += 64)
    add(ld_tile(tp + k), mrule ? ld_mom(mp + k) : TileMom{0.0, 0.0, 0.0}, k);
  sq = wave_sum(sq);
  sp = wave_sum(sp);
  tv_low = 0.0;
  if (want_low && nt <= 64) {  // wave-uniform
    // lane l's tile masses under q and p (tile l)
    double d = 0.0;
    if (lane < nt)
      d = fabs(t0.s_p * exp2_acc((double)t0.r_p - (double)rp) / sp -
               t0.s_q * exp2_acc((double)t0.r_q - (double)rq) / sq);
    tv_low = 0.5 * wave_sum(d);
  }
  kq = wave_min(kq);
  kp = wave_min(kp);
  // with the slice masks of those tiles (statistics tiles record them)
  const auto mask_of = [&](int k, bool pq) {
    if (k >= nt) return 15;
    if (k < 64) return lane_i32(pq ? t0.amax_p : t0.amax_q, k) & 15;
    const TilePart tk = ld_tile(tp + k);
    return (pq ? tk.amax_p : tk.amax_q) & 15;
  };
  *kq_out = kq < nt ? kq * 16 + mask_of(kq, false) : kq;
  *kp_out = kp < nt ? kp * 16 + mask_of(kp, true) : kp;
  RowStat rs;
  const double lq2 = log2_acc(sq), lp2 = log2_acc(sp);
  rs.lz_q = (double)rq + lq2;
  rs.lz_p = (double)rp + lp2;
  rs.tv = 0.0;
  rs.slog = 0.0;
  if (mrule) {
    mhq = wave_sum(mhq);
    mhp = wave_sum(mhp);
    mx = wave_sum(mx);
    rs.slog = log_stat(mrule, lq2, lp2, sq, sp, mhq, mhp, mx);
  }
  rs.zmax_q = zq;
  rs.zmax_p = zp;
  rs.amax_q = -1;
  rs.amax_p = -1;
  return rs;
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

// ------------------------------------------------------------- sampling
// A chunk is what one wavefront covers reading wave-contiguously: lane l's
// lane load i covers entries (i * 64 + l) * VW .. + VW - 1 of it.  A
// statistics tile is a whole number of SubChunks; the residual job and the
// in-tile draw sum them in the same order.
template <int DT, bool VEC, int U_>
struct Chunk {
  static constexpr int U = U_;
  static constexpr int NW = Tile<DT, VEC, U_>::NW, VW = Tile<DT, VEC, U_>::VW;
  static constexpr int N = 64 * U * VW;  // entries per chunk
};
// A sub-chunk of a TN-entry tile drawn from by NWV wavefronts: one per
// wavefront, or several of at most 2 lane loads each (few registers: the
// draw shares its launch with the statistics tiles).
template <int DT, bool VEC, int NWV, int TN = StatTile<DT, VEC>::N>
using SubChunk = Chunk<DT, VEC, (TN / (64 * NWV * Tile<DT, VEC, 1>::VW) < 2)
                                    ? TN / (64 * NWV * Tile<DT, VEC, 1>::VW)
                                    : 2>;

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
// residual masses per tile summed by the residual job.
enum MassSrc : int { kSrcStatsQ = 0, kSrcStatsP = 1, kSrcPass = 3, kSrcTokPi = 4,
                     kSrcDraft = 5 };

template <int SRC>
__device__ __forceinline__ double part_mass(const Params& P, int64_t row, int b, int k,
                                            const RowStat& rs) {
  // every partial was written earlier in the same launch: agent-scope loads
  if constexpr (SRC == kSrcStatsQ || SRC == kSrcDraft) {
    const TilePart t = ld_tile(P.tiles + row * P.nt + k);
    return t.s_q * exp2_acc((double)t.r_q - rs.lz_q);
  } else if constexpr (SRC == kSrcStatsP) {
    const TilePart t = ld_tile(P.tiles + row * P.nt + k);
    return t.s_p * exp2_acc((double)t.r_p - rs.lz_p);
  } else if constexpr (SRC == kSrcTokPi) {
    // Alg. 6's target over a tile: its q mass less the eta partial (the q
    // mass where r = 1), plus eta times its p mass
    const TilePart t = ld_tile(P.tiles + row * P.nt + k);
    const double qm = t.s_q * exp2_acc((double)t.r_q - rs.lz_q);
    const double pm = t.s_p * exp2_acc((double)t.r_p - rs.lz_p);
    const double* ep = P.tvpart + (row * P.nt + k) * kSlices;  // the tile's eta partials
    const double eta_k = (ld_dev_f64(ep) + ld_dev_f64(ep + 1)) + (ld_dev_f64(ep + 2) + ld_dev_f64(ep + 3));
    return fmax(qm - eta_k, 0.0) + rs.tv * pm;
  } else {
    return ld_dev_f64(P.submass + (int64_t)b * P.nsub + k);
  }
}

// Wave 0: the part (tile or chunk) of the inverse-CDF draw -- the first part
// k with C_k > u W, C_k the running mass through part k in vocabulary order
// and W the total -- and the target mass left at its start.  Returns W.
// Parts are read G per lane at a time, all loads in flight together; for at
// most 64 G parts both passes use one read.
constexpr int kFindGroup = 4;

template <int SRC, int G>
__device__ __forceinline__ void load_parts(const Params& P, int64_t row, int b, int K, int k0,
                                           const RowStat& rs, double (&m)[G]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const int k = k0 + j * 64 + lane;
    m[j] = k < K ? part_mass<SRC>(P, row, b, k, rs) : 0.0;
  }
}

template <int SRC, int G = kFindGroup>
__device__ __forceinline__ double find_part(const Params& P, int64_t row, int b, int K,
                                            const RowStat& rs, float u, int* ks_out,
                                            double* rem_out) {
  constexpr int GN = 64 * G;
  double m0[G];
  load_parts<SRC, G>(P, row, b, K, 0, rs, m0);
  double W = 0.0;
#pragma unroll
  for (int j = 0; j < G; ++j) W += wave_sum(m0[j]);
  for (int k0 = GN; k0 < K; k0 += GN) {
    double m[G];
    load_parts<SRC, G>(P, row, b, K, k0, rs, m);
#pragma unroll
    for (int j = 0; j < G; ++j) W += wave_sum(m[j]);
  }
  const double target = (double)u * W;
  double carry = 0.0, rem = 0.0;
  int ks = -1, klast = -1;
  for (int k0 = 0; k0 < K && ks < 0; k0 += GN) {
    double m[G];
    if (k0 == 0) {
#pragma unroll
      for (int j = 0; j < G; ++j) m[j] = m0[j];
    } else {
      load_parts<SRC, G>(P, row, b, K, k0, rs, m);
    }
#pragma unroll
    for (int j = 0; j < G; ++j) {
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

// Wave 0: the in-chunk draw in the chunk starting at entry c0.  Lane loads
// are scanned in entry order -- lane load i, then lane -- for the first one
// where the running mass exceeds rem; its lane then walks its VW entries.
// Rounding that leaves rem unreached takes the last entry with mass.
template <int DT, bool VEC, class C, int KIND>
__device__ __forceinline__ void pick_wave(const Params& P, int b, int64_t row, int64_t c0,
                                          double rem, const ProbScale& ps, int kind = -1) {
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
      const float w = weight_k<DT, KIND>(elem<DT, VEC>(cq[i], e), elem<DT, VEC>(cp[i], e), ps, kind);
      m += (double)w;
      if (w > 0.0f) last_pos = max(last_pos, (int)(base + e));
      if (e & 1) __builtin_amdgcn_sched_barrier(0);
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
    const float w = weight_k<DT, KIND>(elem<DT, VEC>(sq, e), elem<DT, VEC>(sp_, e), ps, kind);
    run += (double)w;
    if (w > 0.0f) lastw = (int)(hbase + e);
    if (hit < 0 && run > rem && w > 0.0f) hit = (int)(hbase + e);
    if (e & 1) __builtin_amdgcn_sched_barrier(0);
  }
  P.out_token[b] = hit >= 0 ? hit : lastw;  // rounding inside the lane load
}

// Whole block: the masses of the sub-chunks of the TN-entry tile at entry t0
// of a row under the distribution KIND, in sh.dv[0 .. NS-1] (wave w sums
// sub-chunks w, w + NWV, ...).  Ends with a block barrier.
template <int DT, bool VEC, int KIND, int NWV, int TN = StatTile<DT, VEC>::N>
__device__ __forceinline__ void subchunk_masses(const Params& P, int64_t row, int64_t t0,
                                                const ProbScale& ps, SharedT<NWV>& sh) {
  using C = SubChunk<DT, VEC, NWV, TN>;
  constexpr int NS = TN / C::N;  // sub-chunks of the tile
  static_assert(NS * C::N == TN && NS % NWV == 0 && NS <= 64,
                "a tile is a whole number of sub-chunks per wavefront");
  constexpr int EB = StatTile<DT, VEC>::EB;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int V = P.V;
  const char* qrow = (const char*)P.q + row * V * EB;
  const char* prow = (const char*)P.p + row * V * EB;
  for (int sc = wv; sc < NS; sc += NWV) {
    ChunkRegs<C> cq = {}, cp = {};
    if (KIND != kP) load_chunk<DT, VEC, C>(qrow, t0 + sc * C::N, V, cq);
    if (KIND != kQ) load_chunk<DT, VEC, C>(prow, t0 + sc * C::N, V, cp);
    double m = 0.0;
#pragma unroll
    for (int i = 0; i < C::U; ++i) {
      float t = 0.0f;
#pragma unroll
      for (int e = 0; e < C::VW; ++e) {
        t += weight_of<DT, KIND>(elem<DT, VEC>(cq[i], e), elem<DT, VEC>(cp[i], e), ps);
        // two entries at a time keep the weights' temporaries few
        if (e & 1) __builtin_amdgcn_sched_barrier(0);
      }
      m += (double)t;
    }
    m = wave_sum(m);
    if (lane == 0) sh.dv[sc] = m;
  }
  __syncthreads();
}

// Wave 0: the total of a tile's sub-chunk masses (after subchunk_masses),
// summed by the same scan the in-tile draw runs, so a draw whose target falls
// in this tile by the tile masses finds it among the sub-chunks.
template <int DT, bool VEC, int NWV, int TN = StatTile<DT, VEC>::N>
__device__ __forceinline__ double tile_mass(const SharedT<NWV>& sh) {
  constexpr int NS = TN / SubChunk<DT, VEC, NWV, TN>::N;
  const int lane = threadIdx.x & 63;
  return lane_f64(wave_incl_scan(lane < NS ? sh.dv[lane] : 0.0), NS - 1);
}

// Whole block: the draw inside the tile at entry t0.  Wave 0 scans the
// sub-chunk masses for the sub-chunk where rem is crossed and draws inside it.
template <int DT, bool VEC, int KIND, int NWV, int TN = StatTile<DT, VEC>::N>
__device__ __forceinline__ void pick_tile(const Params& P, int b, int64_t row, int64_t t0,
                                          double rem, const ProbScale& ps, SharedT<NWV>& sh) {
  using C = SubChunk<DT, VEC, NWV, TN>;
  constexpr int NS = TN / C::N;
  subchunk_masses<DT, VEC, KIND, NWV, TN>(P, row, t0, ps, sh);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
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

// ================================================================ statistics tiles
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
// written by thread 0 through agent-scope stores, for readers in the same
// launch.
template <int DT, bool VEC, int MOM>
__device__ __forceinline__ void tile_partial(const Params& P, int r, int k, const SeqParam& sp,
                                             const uint32_t (&wq)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                             const uint32_t (&wp)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                             Shared& sh) {
  using T = StatTile<DT, VEC>;
  // Thread max, from the maxima of its lane loads.
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
  const float rq = (mq == kNegInf) ? 0.0f : mq * sp.c_hi;
  const float rp = (mp == kNegInf) ? 0.0f : mp * sp.c_hi;
  float sq = 0.0f, spp = 0.0f, hq = 0.0f, hp = 0.0f, xq = 0.0f;
  constexpr bool mom = MOM;
  tile_sums<DT, VEC, MOM>(wq, wp, sp, rq, rp, sq, spp, hq, hp, xq);
  // the moments are complete here: left free, the compiler sinks their
  // accumulation into the conditional combine below and keeps every
  // exponential of the tile live until then
  if constexpr (MOM) asm volatile("" : "+v"(hq), "+v"(hp), "+v"(xq), "+v"(sq), "+v"(spp));
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
  if (lane == 0) {
    sh.m[wv][0] = Wq;
    sh.m[wv][1] = Wp;
    sh.d[wv][0] = dq;
    sh.d[wv][1] = dp;
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
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float wq_ = sh.m[w][0], wp_ = sh.m[w][1];
      if (wq_ != kNegInf)
        tq += sh.d[w][0] * (double)exp2_hw((float)((double)(wq_ * sp.c_hi) - (double)Rq));
      if (wp_ != kNegInf)
        tp += sh.d[w][1] * (double)exp2_hw((float)((double)(wp_ * sp.c_hi) - (double)Rp));
    }
    TilePart t;
    t.s_q = tq;
    t.s_p = tp;
    t.r_q = (Mq == kNegInf) ? kNegInf : Rq;
    t.r_p = (Mp == kNegInf) ? kNegInf : Rp;
    t.zmax_q = Mq;
    t.zmax_p = Mp;
    // the slices (waves) whose entries attain the tile maximum
    int mq = 0, mp = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      mq |= (sh.m[w][0] == Mq) ? 1 << w : 0;
      mp |= (sh.m[w][1] == Mp) ? 1 << w : 0;
    }
    t.amax_q = mq;
    t.amax_p = mp;
    st_tile(P.tiles + (int64_t)r * P.nt + k, t);
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
      st_mom(P.moms + (int64_t)r * P.nt + k, m);
    }
  }
}


// The second-pass weight summed over a thread's entries of one statistics
// tile: for a token rule eta's share (the q mass of the entries the rule
// marks), else max(0, p - q) (D_TV of Lemma 3) in float32.
template <int DT, bool VEC, bool TOK>
__device__ __forceinline__ double pass2_sum(const uint32_t (&wq)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                            const uint32_t (&wp)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                            const ProbScale& ps) {
  using T = StatTile<DT, VEC>;
  double acc = 0.0;
#pragma unroll
  for (int i = 0; i < T::U; ++i) {
    float t = 0.0f;
#pragma unroll
    for (int e = 0; e < T::VW; ++e) {
      const float zq = elem<DT, VEC>(wq[i], e), zp = elem<DT, VEC>(wp[i], e);
      if constexpr (TOK) {
        t += token_r(ps.tok, zq, zp) ? prob(zq, ps.c_hi, ps.c_lo, ps.q_hi, ps.q_lo) : 0.0f;
      } else {
        // D_TV for the deferral decision, where an absolute error of about
        // 1e-7 is far inside the decision margin (the replacement draw sums
        // the same difference: residual_weight)
        const float pq = prob(zq, ps.c_hi, ps.c_lo, ps.q_hi, ps.q_lo);
        const float pp = prob(zp, ps.c_hi, ps.c_lo, ps.p_hi, ps.p_lo);
        t += fmaxf(pp - pq, 0.0f);
      }
      if (e & 1) __builtin_amdgcn_sched_barrier(0);
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


// ---------------------------------------------------------------- slices
// A slice is wavefront w's share of a statistics tile in the tile's own
// layout: lane loads i = 0 .. U-1 of threads w*64 .. w*64+63, lane load i
// covering the 64 VW consecutive entries at t0 + (i * 4 + w) * 64 VW -- the
// tile's sub-chunk i * 4 + w.  A statistics workgroup that takes a second
// pass over a tile (its wavefront w computing slice w) and a job-pass
// wavefront that takes one slice compute the same partial with the same
// arithmetic, so a row's result does not depend on which did it.
static_assert(kSlices == kWaves, "a tile has one slice per wavefront of its workgroup");
template <int DT, bool VEC>
using PartC = Chunk<DT, VEC, 2 * StatTile<DT, VEC>::U>;  // half a tile, wave-contiguous
template <int DT, bool VEC>
using SubC = Chunk<DT, VEC, 1>;

// Wave: "am I the last of n arrivals on cnt?" after this wavefront's item
// (its results stored by its own lanes), arriving with weight w.  On true
// the counter is reset and the wavefront reads the other items' results with
// ld_dev_*.
__device__ __forceinline__ bool arrive_last_w(uint32_t* cnt, uint32_t n, uint32_t w = 1u) {
  uint32_t prev = 0;
  if ((threadIdx.x & 63) == 0) {
    vmem_drain();  // every lane's stores of this item are complete
    prev = add_u32(cnt, w);
    if (prev == n - w) st_u32(cnt, 0u);
  }
  const bool last = (uint32_t)lane_i32((int)prev, 0) == n - w;
  if (last) vmem_drain();
  return last;
}

// Wave: the slice's sub-chunk masses from its loaded entries (lane i < U
// returns sub-chunk i * 4 + w's).
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ double slice_masses_of(const uint32_t (&cq)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                                  const uint32_t (&cp)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
                                                  const ProbScale& ps, int kind) {
  using T = StatTile<DT, VEC>;
  const int lane = threadIdx.x & 63;
  double mine = 0.0;
#pragma unroll
  for (int i = 0; i < T::U; ++i) {
    float t = 0.0f;
#pragma unroll
    for (int e = 0; e < T::VW; ++e) {
      t += weight_k<DT, KIND>(elem<DT, VEC>(cq[i], e), elem<DT, VEC>(cp[i], e), ps, kind);
      if (e & 1) __builtin_amdgcn_sched_barrier(0);
    }
    const double s = wave_sum((double)t);
    if (lane == i) mine = s;
    __builtin_amdgcn_sched_barrier(0);
  }
  return mine;
}

// Wave: the masses of the sub-chunks of slice w of the tile at entry t0 of
// a row under the distribution KIND; lane i < U returns sub-chunk i * 4 + w's
// (float sums per lane load, fp64 across lanes), other lanes 0.
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ double slice_masses_w(const Params& P, int64_t row, int64_t t0, int w,
                                                 const ProbScale& ps, int kind = -1) {
  using T = StatTile<DT, VEC>;
  const int lane = threadIdx.x & 63, V = P.V;
  uint32_t cq[T::U][T::NW] = {}, cp[T::U][T::NW] = {};
  if (KIND != kP)
    load_tile<DT, VEC, T::U, true>((const char*)P.q + row * V * T::EB, t0, V, cq, w * 64 + lane);
  if (KIND != kQ)
    load_tile<DT, VEC, T::U, true>((const char*)P.p + row * V * T::EB, t0, V, cp, w * 64 + lane);
  return slice_masses_of<DT, VEC, KIND>(cq, cp, ps, kind);
}


// Wave: the second-pass partial of slice w of tile k of row r -- the TV
// weight max(0, p - q), or eta's share (the q mass of the entries the rule
// marks) -- into tvpart[r][k * 4 + w].
template <int DT, bool VEC, bool TOK, bool NT = true>
__device__ __forceinline__ void pass2_slice_w(const Params& P, int r, int k, int w,
                                              const SeqParam& sp) {
  using T = StatTile<DT, VEC>;
  const int lane = threadIdx.x & 63, V = P.V;
  const int64_t t0 = (int64_t)k * T::N;
  // the row's statistics and the slice's entries are requested together,
  // the statistics first: waiting for them (a wait for a load is a wait for
  // every load issued before it) leaves the entries in flight while the
  // probability scales are formed -- one round trip, not two.  Only the
  // words prob_scale reads are loaded (a load whose value is never used
  // would still hold its register, and reusing that register would wait for
  // every load before it).
  const uint64_t* rw = reinterpret_cast<const uint64_t*>(P.rowstat + r);
  RowStat rs{};
  rs.lz_q = __longlong_as_double((long long)ld_u64(rw));
  rs.lz_p = __longlong_as_double((long long)ld_u64(rw + 1));
  if constexpr (TOK) {  // eta's rule: the row's TV word and maxima too
    rs.tv = __longlong_as_double((long long)ld_u64(rw + 2));
    const uint64_t m = ld_u64(rw + 4);
    __builtin_memcpy(&rs.zmax_q, &m, sizeof m);
  }
  __builtin_amdgcn_sched_barrier(0);
  uint32_t wq[T::U][T::NW], wp[T::U][T::NW];
  load_tile<DT, VEC, T::U, NT>((const char*)P.q + (int64_t)r * V * T::EB, t0, V, wq, w * 64 + lane);
  load_tile<DT, VEC, T::U, NT>((const char*)P.p + (int64_t)r * V * T::EB, t0, V, wp, w * 64 + lane);
  __builtin_amdgcn_sched_barrier(0);
  const ProbScale ps = prob_scale(sp, rs, TOK);
  double acc = pass2_sum<DT, VEC, TOK>(wq, wp, ps);
  acc = wave_sum(acc);
  if (lane == 0) st_dev_f64(P.tvpart + ((int64_t)r * P.nt + k) * kSlices + w, acc);
}

// Wave: the TV partial of slice w of tile k of row r from the slice's entries
// already in registers (the statistics tile's own loads), into
// tvpart[r][k * 4 + w].
template <int DT, bool VEC>
__device__ __forceinline__ void tv_slice_regs_w(
    const Params& P, int r, int k, int w, const SeqParam& sp,
    const uint32_t (&wq)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
    const uint32_t (&wp)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW]) {
  const ProbScale ps = prob_scale(sp, ld_rowstat(P.rowstat + r), false);
  const double acc = wave_sum(pass2_sum<DT, VEC, false>(wq, wp, ps));
  if ((threadIdx.x & 63) == 0) st_dev_f64(P.tvpart + ((int64_t)r * P.nt + k) * kSlices + w, acc);
}

// ================================================================ the step
// Jobs a row or a sequence publishes for the job pass that follows: a TV or
// eta second pass over a row and the residual masses of row j* of a sequence
// are "row jobs" of nt chunks (one per tile); the two halves of a greedy
// row's argmax and the draws from statistics partials are single chunks.
enum JobKind : int { kJobTv = 1, kJobEta = 2, kJobArg = 4, kJobTvTile = 6, kJobTvSlice = 7 };

// A job entry: kind (bits 60..63), an extra field (bits 32..59: the argmax
// tensor, or a draw's sample kind and j*) and the row or sequence it belongs
// to (bits 0..31).
__device__ __forceinline__ uint64_t job_entry(int kind, uint32_t extra, uint32_t id) {
  return ((uint64_t)kind << 60) | ((uint64_t)(extra & 0x0fffffffu) << 32) | (uint64_t)id;
}
__device__ __forceinline__ int job_kind(uint64_t e) { return (int)(e >> 60); }
__device__ __forceinline__ uint32_t job_extra(uint64_t e) {
  return (uint32_t)(e >> 32) & 0x0fffffffu;
}
__device__ __forceinline__ uint32_t job_id(uint64_t e) { return (uint32_t)e; }

// Job counters: jobs published per pass and list, workgroups per pass that
// have read them.
__device__ __forceinline__ uint32_t* hdr_word(const Params& P, int line) {
  return P.hdr + (int64_t)line * kLineWords;
}
// The header line holding the count of jobs published for the job pass.
constexpr int kHdrJobs = 1;
// The job entries of the job pass.
__device__ __forceinline__ uint64_t* job_list(const Params& P) { return P.jobs; }
__device__ __forceinline__ uint32_t* row_word(const Params& P, int64_t r, int w) {
  return P.rowline + r * kLineWords + w;
}
__device__ __forceinline__ uint64_t* seq_mask(const Params& P, int64_t b) {
  return reinterpret_cast<uint64_t*>(row_word(P, b, kSeqMask));
}
__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int l) {
  return ((uint64_t)(uint32_t)lane_i32((int)(v >> 32), l) << 32) |
         (uint64_t)(uint32_t)lane_i32((int)(uint32_t)v, l);
}

// Publish a job (whose inputs are stored) for the job pass, a later launch.
// The pass never holds more jobs than its list has slots; the bound only
// keeps a broken count from writing past it.
__device__ __forceinline__ void publish_single(const Params& P, int kind, uint32_t extra,
                                               uint32_t id) {
  const uint32_t s = add_u32(hdr_word(P, kHdrJobs), 1u);
  if ((int64_t)s >= P.single_slots) return;
  st_u64(job_list(P) + s, job_entry(kind, extra, id));
}
// Wave: n jobs (kind, extra = 0 .. n-1, id), one reservation.
__device__ __forceinline__ void publish_singles_w(const Params& P, int kind, uint32_t id,
                                                  uint32_t n) {
  if (n == 0u) return;
  const int lane = threadIdx.x & 63;
  uint32_t s0 = 0;
  if (lane == 0) s0 = add_u32(hdr_word(P, kHdrJobs), n);
  s0 = (uint32_t)lane_i32((int)s0, 0);
  for (uint32_t x = (uint32_t)lane; x < n; x += 64u) {
    if ((int64_t)s0 + x >= P.single_slots) break;
    st_u64(job_list(P) + s0 + x, job_entry(kind, x, id));
  }
}

// Shared state of a job workgroup.
struct StepShared {
  Shared sh;
  RowStat rs;
  PickState pk;
  int a[4];  // values thread 0 or wave 0 hands to the block
};

// Wave: sequence b's first rejection is j* = f.  Writes its accept length,
// then the greedy token; or, for a draw (from the statistics partials, or
// from the residual of row f), records it in the sequence's outcome word for
// the draw pass (k_res) that follows the launch finishing the sequence: the
// statistics kernel's, or the job pass's.
template <int DT>
__device__ __forceinline__ void seq_finish_w(const Params& P, int b, int f, const SeqParam& sp,
                                             int rec) {
  const int gamma = P.gamma, g1 = gamma + 1;
  const int64_t row = (int64_t)b * g1 + f;
  if ((threadIdx.x & 63) != 0) return;
  if (!sp.valid) {
    P.out_accept[b] = -1;
    P.out_token[b] = -1;
    if (P.out_norm) P.out_norm[b] = 0.0f;
    return;
  }
  P.out_accept[b] = f;
  const int dstar = (rec >> 1) & 1;
  if (sp.greedy) {
    const RowStat rs = ld_rowstat(P.rowstat + row);
    P.out_token[b] = (dstar || sp.rule == SPC_RULE_LOSSY) ? rs.amax_p : rs.amax_q;
    if (P.out_norm) P.out_norm[b] = 1.0f;
    return;
  }
  int kind;
  if (is_token(sp.rule)) {
    kind = (f < gamma) ? kTokRes : kTokPi;
  } else if (sp.rule == SPC_RULE_LOSSY) {
    // residual max(0, pi - q) = max(0, p - q); extra token from p
    kind = (f < gamma) ? kResidual : kP;
  } else {
    // a rejection with delta = 0 only happens for an out-of-range draft; its
    // residual max(0, q - q) is empty, so p is sampled instead
    kind = (f < gamma) ? (dstar ? kResidual : kP) : (dstar ? kP : kQ);
  }
  st_u32(row_word(P, b, kSeqInfo), kSeqInfoSet | ((uint32_t)kind << 8) | (uint32_t)f);
}

// Lane 0: write the outputs and the record of decided row r (d from
// decide_row; an invalid sequence's rows record "reject, no deferral"),
// with `extra` in the record's bits 4 and up.
__device__ __forceinline__ void row_record(const Params& P, int r, const SeqParam& sp,
                                           const RowDecision& d, int extra) {
  P.out_defer[r] = sp.valid ? (uint8_t)d.delta : (uint8_t)0;
  if (sp.valid && P.out_stats) {
    const double T = sp.greedy ? 1.0 : kLog2e / sp.c;
    float* o = P.out_stats + (int64_t)r * 8;
    o[0] = (float)((double)d.rs.zmax_q / T);
    o[1] = (float)(d.rs.lz_q * kLn2);
    o[2] = d.maxq;
    o[3] = (float)((double)d.rs.zmax_p / T);
    o[4] = (float)(d.rs.lz_p * kLn2);
    o[5] = d.maxp;
    o[6] = d.tv;
    o[7] = (float)d.rs.slog;
  }
  if (sp.valid && P.out_argmax) {
    P.out_argmax[(int64_t)r * 2 + 0] = d.rs.amax_q;
    P.out_argmax[(int64_t)r * 2 + 1] = d.rs.amax_p;
  }
  if (sp.valid) st_rowstat(P.rowstat + r, d.rs);
  st_i32(P.rowdec + r, (sp.valid ? d.keep | (d.delta << 1) : 0) | (extra << 4));
}

// The inputs of a sampled row's decision besides its statistics: the draft
// token, its logits and the row's uniform.
struct DraftIn {
  int x;
  float zqx, zpx, u;
};

// The draft token of row r = (b, j); -1 at the bonus position.
__device__ __forceinline__ int draft_token(const Params& P, int b, int j) {
  return j < P.gamma ? P.draft[(int64_t)b * P.gamma + j] : -1;
}

// Wave: the draft inputs of row r with draft token x (logits only for an
// in-range draft of a sampled row).
template <int DT>
__device__ __forceinline__ DraftIn draft_in(const Params& P, int r, int x, const SeqParam& sp) {
  DraftIn in{x, 0.0f, 0.0f, 0.0f};
  if (sp.valid && !sp.greedy) {
    in.u = P.uniforms[r];
    if (in.x >= 0 && in.x < P.V) {
      in.zqx = load_logit<DT>(P.q, r, P.V, in.x);
      in.zpx = load_logit<DT>(P.p, r, P.V, in.x);
    }
  }
  return in;
}

// Blocks of at most kPackRows rows of a sampled sequence carry their
// decisions in the sequence's 64-bit mask word (three bits a row).
constexpr int kPackRows = 21;

// Wave: decide row r = (b, j) from its statistics rs (delta_j by the rule,
// a_j by the acceptance test), write its outputs and add it to the
// sequence's decided-row mask.  Returns j* when this decision completes the
// prefix of decided rows 0 .. j* (j* the first rejection; row gamma always
// rejects), else -1; every lane returns the same value.
// rec_f: j*'s record (bit 0 a_j*, bit 1 delta_j*).
template <int DT>
__device__ __forceinline__ int row_decide_w(const Params& P, int r, int b, int j,
                                            const SeqParam& sp, const RowStat& rs,
                                            const DraftIn* pre, int* rec_f) {
  const int gamma = P.gamma, g1 = gamma + 1, V = P.V;
  const int lane = threadIdx.x & 63;
  RowDecision d{};
  if (sp.valid) {
    const DraftIn in = pre ? *pre : draft_in<DT>(P, r, draft_token(P, b, j), sp);
    const int x = in.x;
    float zqx = in.zqx, zpx = in.zpx;
    const float u = in.u;
    if (sp.greedy &&
        ((is_token(sp.rule) && sp.rule != SPC_RULE_TOKEN_V1) || sp.rule == SPC_RULE_BILD) &&
        rs.amax_q >= 0 && rs.amax_q < V) {
      // greedy TokenV2/V3 and BiLD* read p at the drafter's argmax
      zpx = load_logit<DT>(P.p, r, V, rs.amax_q);
    }
    d = decide_row(sp, rs, j, gamma, V, x, zqx, zpx, u);
  }
  if (g1 <= kPackRows && !sp.greedy) {
    // the decision travels in the mask word itself: bit j (row decided),
    // bit kPackRows + j (a_j = 0), bit 2 kPackRows + j (delta_j); no row
    // reads another's record, so none waits for its stores
    // (an invalid sequence's rows reject, as their records say)
    const uint64_t mine = (1ull << j) | ((uint64_t)!(sp.valid && d.keep) << (kPackRows + j)) |
                          ((uint64_t)(sp.valid && d.delta) << (2 * kPackRows + j));
    uint64_t old = 0;
    if (lane == 0) {
      row_record(P, r, sp, d, 0);
      old = or_u64(seq_mask(P, b), mine);
    }
    old = lane_u64(old, 0);
    const uint64_t rows = (1ull << g1) - 1ull;
    const uint64_t now = old | mine;
    if (lane == 0 && (now & rows) == rows) st_u64(seq_mask(P, b), 0ull);  // the last row resets it
    const int p_old = __builtin_ctzll(~(old & rows));
    const int p_now = __builtin_ctzll(~(now & rows));
    if (p_now <= p_old) return -1;
    const uint64_t rej = (now >> kPackRows) & ((1ull << p_now) - 1ull);
    if (!rej) return -1;
    const int f = __builtin_ctzll(rej);
    *rec_f = (int)((now >> (2 * kPackRows + f)) & 1ull) << 1;  // a_f = 0, delta_f
    return f >= p_old ? f : -1;
  }
  uint64_t old = 0;
  if (lane == 0) {
    row_record(P, r, sp, d, 0);
    vmem_drain();  // the row's record is stored before its bit is set
    old = or_u64(seq_mask(P, b), 1ull << j);
  }
  old = lane_u64(old, 0);
  const uint64_t full = (g1 == 64) ? ~0ull : ((1ull << g1) - 1ull);
  const uint64_t now = old | (1ull << j);
  if (lane == 0 && now == full) st_u64(seq_mask(P, b), 0ull);  // the last row resets it
  const int p_old = __builtin_ctzll(~old);
  const int p_now = (now == ~0ull) ? 64 : __builtin_ctzll(~now);
  if (p_now <= p_old) return -1;
  // rows 0 .. p_now - 1 are decided (their records were stored before their
  // bits were set); the first rejection among them, if it lies in the rows
  // this decision added to the prefix, is j*
  const int rec = lane < p_now ? ld_i32(P.rowdec + (int64_t)b * g1 + lane) : 1;
  const unsigned long long rej = __ballot(!(rec & 1));
  if (!rej) return -1;
  const int f = __ffsll(rej) - 1;
  *rec_f = lane_i32(rec, f);
  return f >= p_old ? f : -1;
}

// Wave, after the last tile of row r = (b, j) arrived: merge the row, then
// publish its second pass (TV, or eta for the tiles its statistics leave
// open) or its argmax to the job pass, or decide it and, when that settles
// j*, finish the sequence.
template <int DT, int MS>
__device__ __forceinline__ void row_merged_w(const Params& P, int r, int b, int j,
                                             const SeqParam& sp, int x) {
  const int lane = threadIdx.x & 63;
  const int nt = P.nt;
  // the decision's draft inputs, requested together with the tile partials
  const DraftIn in = draft_in<DT>(P, r, x, sp);
  int kq, kp;
  double tv_low;
  RowStat rs = merge_row(P, r, (MS != 0 && needs_mom(sp)) ? sp.rule : 0, &kq, &kp,
                         sp.valid && !sp.greedy && has_tv_parts(sp.rule) && !P.out_stats, tv_low);
  if (sp.valid && sp.greedy) {
    // the lowest index of each row maximum, from the first tile holding it
    if (lane == 0) {
      st_rowstat(P.rowstat + r, rs);
      st_i32(P.argres + (int64_t)r * 4 + 0, kq);
      st_i32(P.argres + (int64_t)r * 4 + 1, kp);
      publish_single(P, kJobArg, 0u, (uint32_t)r);
      publish_single(P, kJobArg, 1u, (uint32_t)r);
    }
    return;
  }
  if (sp.valid && has_tv_parts(sp.rule)) {
    // Without row statistics to report, a row whose decision D_TV cannot
    // change is decided now and takes no TV pass: its ready flag says 2 to
    // its own waiting workgroups (tv_self) and stays 0 for the TV pass
    // kernel.  Every other row is published as merged (flag 1).
    // (the tile-mass bound, lowered by 1e-5 relative and 1e-6 absolute: the
    // computed D_TV, whose error is ~1e-7 of the mass summed, stays above it)
    const double lo = fmax(0.0, tv_low * (1.0 - 1e-5) - 1e-6);
    const bool free = !P.out_stats && tv_free_decision(sp, rs, lo) >= 0;
    if (lane == 0 && !free) {
      st_rowstat(P.rowstat + r, rs);
      if (!P.tv_jobs) {
        vmem_drain();
        st_u32(row_word(P, r, kRowReady), 1u);
      }
    }
    // (with tv_jobs the row's TV slices are jobs of the job pass)
    if (!free && P.tv_jobs)
      publish_singles_w(P, kJobTvSlice, (uint32_t)r, (uint32_t)(nt * kSlices));
    if (lane == 0 && free && P.tv_self) st_u32(row_word(P, r, kRowReady), 2u);
    if (!free) return;
    rs.tv = 1.0;  // any D_TV in [lo, 1] decides it alike
  }
  if (sp.valid && is_token(sp.rule)) {
    // eta's share of every tile wholly below the rule's threshold comes from
    // its statistics; the other tiles are listed for a second look (the job's
    // chunks past the list do nothing).  With none listed, eta is summed
    // here in the order the job's last chunk would sum it.
    const TokenRule tr = token_rule(sp, rs, exp2_acc((double)rs.zmax_p * sp.c - rs.lz_p));
    double eta = 0.0;
    uint32_t count = 0;
    for (int k0 = 0; k0 < nt; k0 += 64) {
      const int k = k0 + lane;
      double e = 0.0;
      bool need = false;
      if (k < nt) {
        need = !eta_from_stats(tr, ld_tile(P.tiles + (int64_t)r * nt + k), rs.lz_q, &e);
        if (!need) {  // the tile's share, on its first slice
          double* ep = P.tvpart + ((int64_t)r * nt + k) * kSlices;
          st_dev_f64(ep, e);
          st_dev_f64(ep + 1, 0.0);
          st_dev_f64(ep + 2, 0.0);
          st_dev_f64(ep + 3, 0.0);
        }
      }
      const unsigned long long nm = __ballot(need);
      if (need)
        st_i32(P.etalist + (int64_t)r * nt + count + __popcll(nm & ((1ull << lane) - 1ull)), k);
      count += (uint32_t)__popcll(nm);
      if (k < nt) eta += e;
    }
    if (count != 0) {
      if (lane == 0) {
        st_rowstat(P.rowstat + r, rs);
        st_i32(P.etacnt + r, (int32_t)count);
      }
      // a job per slice of every listed tile (the job pass)
      publish_singles_w(P, kJobEta, (uint32_t)r, count * (uint32_t)kSlices);
      return;
    }
    rs.tv = wave_sum(eta);
  }
  int rec = 0;
  const int f = row_decide_w<DT>(P, r, b, j, sp, rs, &in, &rec);
  if (f >= 0) seq_finish_w<DT>(P, b, f, sp, rec);
}

// Wave: the row's decision once its TV, eta or argmax is known; when it
// settles j*, the sequence's finish publishes to the next job pass.
template <int DT>
__device__ __forceinline__ void row_job_decide(const Params& P, int kind, int r) {
  const int g1 = P.gamma + 1, np = P.nt * kSlices;
  const int b = r / g1, j = r - b * g1;
  RowStat rs = ld_rowstat(P.rowstat + r);
  if (kind == kJobArg) {
    rs.amax_q = ld_i32(P.argres + (int64_t)r * 4 + 2);
    rs.amax_p = ld_i32(P.argres + (int64_t)r * 4 + 3);
  } else {
    // the TV or eta partials of every slice, in slice order
    double s = 0.0;
    for (int k = threadIdx.x & 63; k < np; k += 64)
      s += ld_dev_f64(P.tvpart + (int64_t)r * np + k);
    rs.tv = wave_sum(s);
  }
  const SeqParam sp = seq_param(P, b);
  int rec = 0;
  const int f = row_decide_w<DT>(P, r, b, j, sp, rs, nullptr, &rec);
  if (f >= 0) seq_finish_w<DT>(P, b, f, sp, rec);
}

// The wait of a workgroup for a TV row's merge is bounded by P.wait_ticks of
// the 100 MHz real-time clock (by default 4000: 40 us, far beyond the usual
// wait); past it the tile goes to the job pass.

// Wave: the last of the 4 nt slices of TV row rv arrived: its decision (and
// the sequence's finish), then the row's ready
// flag is cleared for the next call.
template <int DT>
__device__ __forceinline__ void tv_row_done(const Params& P, int rv) {
  row_job_decide<DT>(P, kJobTv, rv);
  if ((threadIdx.x & 63) == 0) st_u32(row_word(P, rv, kRowReady), 0u);
}

// Wait (bounded, thread 0) for the ready flag of TV row rv; block-uniform
// result: 1 (merged, take the TV pass), 2 (decided without one) or 0 (timed
// out: the job pass takes tile k of the row's TV pass).
__device__ __forceinline__ uint32_t tv_wait_ready(const Params& P, int rv, int k, Shared& sh) {
  if (threadIdx.x == 0) {
    const uint32_t* flag = row_word(P, rv, kRowReady);
    uint32_t f = ld_u32(flag);
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (f == 0u && __builtin_amdgcn_s_memrealtime() - t0 < (uint64_t)P.wait_ticks) {
      __builtin_amdgcn_s_sleep(4);
      f = ld_u32(flag);
    }
    sh.flag = (int)f;
    if (f == 0u) publish_single(P, kJobTvTile, (uint32_t)k, (uint32_t)rv);
  }
  __syncthreads();
  return (uint32_t)sh.flag;
}

// Wave 0: a tile of TV row rv arrives (weight kSlices) without a TV pass,
// the row having been decided without one (flag 2); the last arrival
// clears the flag for the next call.
__device__ __forceinline__ void tv_skip_arrive_w(const Params& P, int rv) {
  if (arrive_last_w(row_word(P, rv, kRowTvArrive), (uint32_t)(kSlices * P.nt), kSlices) &&
      (threadIdx.x & 63) == 0)
    st_u32(row_word(P, rv, kRowReady), 0u);
}


// Whole block: the TV pass over tile k of the block's own row r from the
// registers that hold the tile (small batches: every tile of the grid is
// resident at once, so the row's last tile arrives while the others wait).
// Once the row's merge has set its ready flag each wavefront sums its slice;
// the last of the row's slices decides the row.
template <int DT, bool VEC>
__device__ __forceinline__ void tv_self(
    const Params& P, int r, int k, const SeqParam& sp, Shared& sh,
    const uint32_t (&wq)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW],
    const uint32_t (&wp)[StatTile<DT, VEC>::U][StatTile<DT, VEC>::NW]) {
  const uint32_t f = tv_wait_ready(P, r, k, sh);  // block-uniform
  if (f == 0u) return;
  if (f == 2u) {
    if (threadIdx.x < 64) tv_skip_arrive_w(P, r);
    return;
  }
  tv_slice_regs_w<DT, VEC>(P, r, k, threadIdx.x >> 6, sp, wq, wp);
  vmem_drain();
  __syncthreads();  // all four slices are stored
  if (threadIdx.x < 64 &&
      arrive_last_w(row_word(P, r, kRowTvArrive), (uint32_t)(kSlices * P.nt), kSlices))
    tv_row_done<DT>(P, r);
}

// How the statistics tiles serve the TV pass (OPT / OPTLOG rows at T > 0):
// not at all (the TV pass kernel takes it, or there is no TV row), or, in a
// grid resident at once, on their own row from registers (tv_self).
enum TvMode : int { kTvNone = 0, kTvSelf = 2 };

// The statistics tiles.  grid (nt, R): tile k of row r, its logits read
// non-temporally; with PAIR, grid (ceil(nt / 2), R) and tiles 2x and 2x + 1,
// both loaded at once (large batches: half the arrivals, twice the bytes in
// flight per workgroup).  After the tile partials wave 0 arrives on the
// row's counter, and the last tile of the row merges and decides it (a TV
// row: marks it merged).  With kTvSelf the block then takes its share of its
// own row's TV pass; otherwise waves 1-3 leave after the partials.
// With first moments the block is held to 96 VGPRs (five workgroups per
// SIMD); the two-tile form keeps its registers (capped, it spills in the
// streaming loop).
template <int DT, bool VEC, int MS, int TVM, bool PAIR = false>
__global__ __launch_bounds__(kThreads)
__attribute__((amdgpu_waves_per_eu(MS != 0 ? 5 : 1))) void k_tiles(Params P) {
  static_assert(!PAIR || TVM == kTvNone, "a pair of tiles takes no TV pass");
  constexpr bool NT = true;
  using T = StatTile<DT, VEC>;
  __shared__ Shared shs[PAIR ? 2 : 1];
  Shared& sh = shs[0];
  const int k = PAIR ? 2 * (int)blockIdx.x : (int)blockIdx.x, r = blockIdx.y;
  const int nt = P.nt, g1 = P.gamma + 1, V = P.V;
  const int b = r / g1, j = r - b * g1;
  const SeqParam sp = seq_param(P, b);
  // the row's draft token, for the decision should this be its last tile
  const int x = draft_token(P, b, j);
  const char* qrow = (const char*)P.q + (int64_t)r * V * T::EB;
  const char* prow = (const char*)P.p + (int64_t)r * V * T::EB;
  const int64_t t0 = (int64_t)k * T::N;
  const bool two = PAIR && k + 1 < nt;  // block-uniform
  uint32_t wq[T::U][T::NW], wp[T::U][T::NW], vq[T::U][T::NW], vp[T::U][T::NW];
  load_tile<DT, VEC, T::U, NT>(qrow, t0, V, wq, threadIdx.x);
  load_tile<DT, VEC, T::U, NT>(prow, t0, V, wp, threadIdx.x);
  if (two) {
    load_tile<DT, VEC, T::U, NT>(qrow, t0 + T::N, V, vq, threadIdx.x);
    load_tile<DT, VEC, T::U, NT>(prow, t0 + T::N, V, vp, threadIdx.x);
  }
  if (MS != 0 && needs_mom(sp))
    tile_partial<DT, VEC, MS>(P, r, k, sp, wq, wp, sh);
  else
    tile_partial<DT, VEC, 0>(P, r, k, sp, wq, wp, sh);
  if constexpr (PAIR) {
    if (two) {
      if (MS != 0 && needs_mom(sp))
        tile_partial<DT, VEC, MS>(P, r, k + 1, sp, vq, vp, shs[PAIR ? 1 : 0]);
      else
        tile_partial<DT, VEC, 0>(P, r, k + 1, sp, vq, vp, shs[PAIR ? 1 : 0]);
    }
  }
  const uint32_t n = two ? 2u : 1u;  // tiles this block adds to its row
  if (threadIdx.x < 64) {
    // wave 0: thread 0 stored the partials; arrive on the row's counter
    uint32_t prev = 0;
    if (threadIdx.x == 0) {
      vmem_drain();
      prev = add_u32(row_word(P, r, kRowArrive), n);
      if (prev + n == (uint32_t)nt) st_u32(row_word(P, r, kRowArrive), 0u);
    }
    if ((uint32_t)lane_i32((int)prev, 0) + n == (uint32_t)nt) {
      vmem_drain();
      row_merged_w<DT, MS>(P, r, b, j, sp, x);
    }
  }
  if constexpr (TVM == kTvSelf) {
    if (sp.valid && !sp.greedy && has_tv_parts(sp.rule)) tv_self<DT, VEC>(P, r, k, sp, sh, wq, wp);
  }
}

// The TV passes of a batch too large for its statistics workgroups to take
// them: grid (nt, R), after the statistics kernel (every TV row is merged).
// Workgroup (k, r) of a TV row (OPT / OPTLOG at T > 0) sums the TV partials
// of tile k (wavefront w its slice w, the logits read non-temporally: this
// is their last read); the last of the row's slices decides the row, and a
// sequence that decision finishes is drawn by the draw pass that follows.
// Other rows' workgroups leave at once.
template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void k_tvpass(Params P) {
  const int k = blockIdx.x, r = blockIdx.y;
  const SeqParam sp = seq_param(P, r / (P.gamma + 1));
  if (!(sp.valid && !sp.greedy && has_tv_parts(sp.rule))) return;  // block-uniform
  // rows decided without a TV pass have no ready flag
  if (ld_u32(row_word(P, r, kRowReady)) != 1u) return;  // block-uniform
  pass2_slice_w<DT, VEC, false>(P, r, k, threadIdx.x >> 6, sp);
  vmem_drain();
  __syncthreads();  // all four slices are stored
  if (threadIdx.x < 64 &&
      arrive_last_w(row_word(P, r, kRowTvArrive), (uint32_t)(kSlices * P.nt), kSlices))
    tv_row_done<DT>(P, r);
}

// ---------------------------------------------------------------- job pass
// Wave: the masses of the NS sub-chunks of the part at entry e0 of a row
// under the distribution KIND; lane base + i returns sub-chunk i's (float
// sums per lane load, fp64 across lanes), other lanes 0.
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ double part_masses_w(const Params& P, int64_t row, int64_t e0,
                                                const ProbScale& ps, int base = 0, int kind = -1) {
  using C = PartC<DT, VEC>;
  constexpr int EB = StatTile<DT, VEC>::EB;
  const int lane = threadIdx.x & 63, V = P.V;
  ChunkRegs<C> cq = {}, cp = {};
  if (KIND != kP) load_chunk<DT, VEC, C>((const char*)P.q + row * V * EB, e0, V, cq);
  if (KIND != kQ) load_chunk<DT, VEC, C>((const char*)P.p + row * V * EB, e0, V, cp);
  double mine = 0.0;
#pragma unroll
  for (int i = 0; i < C::U; ++i) {
    float t = 0.0f;
#pragma unroll
    for (int e = 0; e < C::VW; ++e) {
      t += weight_k<DT, KIND>(elem<DT, VEC>(cq[i], e), elem<DT, VEC>(cp[i], e), ps, kind);
      if (e & 1) __builtin_amdgcn_sched_barrier(0);
    }
    const double s = wave_sum((double)t);
    if (lane == base + i) mine = s;
    __builtin_amdgcn_sched_barrier(0);  // one lane load's weights at a time
  }
  return mine;
}

// Wave: the draw inside the NSUB sub-chunks starting at entry e0 whose
// masses lane i < NSUB holds: the first sub-chunk where the running mass
// exceeds rem (rounding that leaves rem unreached takes the last sub-chunk
// with mass), then the entry inside it.
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ void draw_in_subs_w(const Params& P, int b, int64_t row, int64_t e0,
                                               double ml, int nsub, double rem,
                                               const ProbScale& ps, int kind = -1) {
  const int lane = threadIdx.x & 63;
  ml = lane < nsub ? ml : 0.0;
  const double incl = wave_incl_scan(ml);
  const unsigned long long hit = __ballot(ml > 0.0 && incl > rem);
  const unsigned long long pos = __ballot(ml > 0.0);
  int c;
  double r;
  if (hit) {
    c = __ffsll(hit) - 1;
    r = rem - (lane_f64(incl, c) - lane_f64(ml, c));
  } else {
    c = pos ? 63 - __clzll(pos) : 0;
    r = __builtin_huge_val();
  }
  pick_wave<DT, VEC, SubC<DT, VEC>, KIND>(P, b, row, e0 + (int64_t)c * SubC<DT, VEC>::N, r, ps,
                                          kind);
}

// Wave: the inverse-CDF draw of sequence b at row `row` (the row of j*) from
// the distribution `kind`, its part masses from `src`: the statistics
// partials per tile (then the tile's sub-chunk masses are summed here), or
// the residual job's sub-chunk masses, searched directly.  An empty residual
// (possible only through rounding) is replaced by p.
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ void draw_kind_w(const Params& P, int b, int64_t row, int ks,
                                            double rem, const ProbScale& ps) {
  if constexpr (KIND == kResidual || KIND == kTokRes) {
    // the residual job's sub-chunk masses were searched: ks is a sub-chunk
    pick_wave<DT, VEC, SubC<DT, VEC>, KIND>(P, b, row, (int64_t)ks * SubC<DT, VEC>::N, rem, ps);
  } else {
    // a statistics tile: the masses of its sub-chunks (its two
    // wave-contiguous halves, in order), then the sub-chunk's entry
    const int64_t t0 = (int64_t)ks * StatTile<DT, VEC>::N;
    constexpr int NS = PartC<DT, VEC>::U;
    double m = 0.0;
#pragma unroll 1
    for (int half = 0; half < 2; ++half)
      m += part_masses_w<DT, VEC, KIND>(P, row, t0 + half * PartC<DT, VEC>::N, ps, half * NS);
    draw_in_subs_w<DT, VEC, KIND>(P, b, row, t0, m, 2 * NS, rem, ps);
  }
}

template <int DT, bool VEC>
__device__ __forceinline__ void draw_w(const Params& P, int b, int64_t row, int kind, int src,
                                       const SeqParam& sp, const RowStat& rs) {
  const int lane = threadIdx.x & 63;
  const float u = P.uniforms[(int64_t)b * (P.gamma + 1) + P.gamma];
  int ks;
  double rem, W;
  if (src == kSrcStatsQ) W = find_part<kSrcStatsQ>(P, row, b, P.nt, rs, u, &ks, &rem);
  else if (src == kSrcStatsP) W = find_part<kSrcStatsP>(P, row, b, P.nt, rs, u, &ks, &rem);
  else if (src == kSrcTokPi) W = find_part<kSrcTokPi>(P, row, b, P.nt, rs, u, &ks, &rem);
  else W = find_part<kSrcPass, 8>(P, row, b, P.nsub, rs, u, &ks, &rem);
  if ((kind == kResidual || kind == kTokRes) && !(W > 0.0)) {
    kind = kP;
    src = kSrcStatsP;
    W = find_part<kSrcStatsP>(P, row, b, P.nt, rs, u, &ks, &rem);
  }
  if (lane == 0) {
    if (P.out_norm) P.out_norm[b] = (float)W;
    if (ks < 0) P.out_token[b] = -1;
  }
  if (ks < 0) return;  // wave-uniform
  const ProbScale ps = prob_scale(sp, rs, kind == kTokRes || kind == kTokPi);
  if (kind == kQ) draw_kind_w<DT, VEC, kQ>(P, b, row, ks, rem, ps);
  else if (kind == kP) draw_kind_w<DT, VEC, kP>(P, b, row, ks, rem, ps);
  else if (kind == kTokPi) draw_kind_w<DT, VEC, kTokPi>(P, b, row, ks, rem, ps);
  else if (kind == kTokRes) draw_kind_w<DT, VEC, kTokRes>(P, b, row, ks, rem, ps);
  else draw_kind_w<DT, VEC, kResidual>(P, b, row, ks, rem, ps);
}

// Wave: item c = k * 4 + w of a TV or eta row job of row r: slice w of tile
// k (for eta, of the k-th listed tile; an item past the list does nothing).
template <int DT, bool VEC, bool TOK>
__device__ __forceinline__ void pass2_item_w(const Params& P, int r, int c) {
  int k = c / kSlices;
  const int w = c % kSlices;
  if (TOK) {
    if (k >= ld_i32(P.etacnt + r)) return;  // wave-uniform
    k = ld_i32(P.etalist + (int64_t)r * P.nt + k);
  }
  pass2_slice_w<DT, VEC, TOK>(P, r, k, w, seq_param(P, r / (P.gamma + 1)));
}

// Wave: half h of the argmax of greedy row r: the lowest index of the row
// maximum of q (h = 0) or p (h = 1), in the first tile holding it, read only
// in the slices of that tile that attain it (usually one; a slice's lane
// loads interleave with the other slices', so the minimum is taken over
// every slice read).
template <int DT, bool VEC>
__device__ __forceinline__ void arg_half_w(const Params& P, int r, int h) {
  using T = StatTile<DT, VEC>;
  const int V = P.V;
  const int lane = threadIdx.x & 63;
  const int packed = ld_i32(P.argres + (int64_t)r * 4 + h);
  int k = packed >> 4, mask = packed & 15;
  if (packed < 0 || k >= P.nt) {  // a broken record: search the whole first tile
    k = 0;
    mask = 15;
  }
  if (mask == 0) mask = 15;
  const RowStat rs = ld_rowstat(P.rowstat + r);
  const float z = h ? rs.zmax_p : rs.zmax_q;
  const char* row = (const char*)(h ? P.p : P.q) + (int64_t)r * V * T::EB;
  const int64_t t0 = (int64_t)k * T::N;
  int idx = 0x7fffffff;
#pragma unroll 1
  for (int w = 0; w < kSlices; ++w) {
    if (!((mask >> w) & 1)) continue;  // wave-uniform
    uint32_t c[T::U][T::NW];
    load_tile<DT, VEC, T::U, true>(row, t0, V, c, w * 64 + lane);
#pragma unroll
    for (int i = T::U - 1; i >= 0; --i) {
      const int base = (int)t0 + ((i * kSlices + w) * 64 + lane) * T::VW;
#pragma unroll
      for (int e = T::VW - 1; e >= 0; --e)
        if (elem<DT, VEC>(c[i], e) == z && base + e < V) idx = min(idx, base + e);
    }
  }
  idx = wave_min(idx);
  if (lane == 0) st_i32(P.argres + (int64_t)r * 4 + 2 + h, idx);
}

// Wave: item c = k * 4 + w of sequence b's residual job over row f (= j*),
// sampling kind KIND: the residual masses of the sub-chunks of slice w of
// tile k, stored at their place in the row's sub-chunk order, which the draw
// searches directly.
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ void res_slice_w(const Params& P, int b, int c, int f,
                                            const RowStat& rs) {
  constexpr int U = StatTile<DT, VEC>::U;
  using T = StatTile<DT, VEC>;
  const int k = c / kSlices, w = c % kSlices;
  const int lane = threadIdx.x & 63, V = P.V;
  const int64_t row = (int64_t)b * (P.gamma + 1) + f;
  const int64_t t0 = (int64_t)k * T::N;
  const SeqParam sp = seq_param(P, b);
  const ProbScale ps = prob_scale(sp, rs, KIND == kTokRes);
  __builtin_amdgcn_sched_barrier(0);
  uint32_t cq[T::U][T::NW], cp[T::U][T::NW];
  load_tile<DT, VEC, T::U, true>((const char*)P.q + row * V * T::EB, t0, V, cq, w * 64 + lane);
  load_tile<DT, VEC, T::U, true>((const char*)P.p + row * V * T::EB, t0, V, cp, w * 64 + lane);
  const double ml = slice_masses_of<DT, VEC, KIND>(cq, cp, ps, -1);
  if (lane < U)
    st_dev_f64(P.submass + (int64_t)b * P.nsub + (int64_t)k * (U * kSlices) + lane * kSlices + w,
               ml);
}


// ---------------------------------------------------------------- draw pass
// k_res: grid (nt, B), the step's last kernel.  For a sequence finished with
// a residual draw, workgroup (k, b) sums the residual masses of the
// sub-chunks of tile k of row j* (wavefront w its slice w); the last of the
// sequence's workgroups to arrive draws.  A draw from the statistics
// partials is made by workgroup (0, b).  The last arrival clears the
// sequence's outcome word for the next call.  Sequences without a draw
// (greedy or invalid) have no outcome word and are skipped.
// bfloat16: held to 80 VGPRs, six resident workgroups per SIMD, so that in
// large batches (256 sequences: 8192 workgroups) one workgroup's loads
// overlap another's residual weights.  What spills is the draw's own code,
// which only the last arrival of a sequence runs.
template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads)
__attribute__((amdgpu_waves_per_eu(DT == SPC_BF16 ? 6 : 1))) void k_res(Params P) {
  const int k = blockIdx.x, b = blockIdx.y;
  const int g1 = P.gamma + 1, lane = threadIdx.x & 63;
  // the statistics of every row of the sequence (lane j: row j), requested
  // together with the outcome word that names the row the draw needs
  RowStat mine{};
  if (lane < g1) mine = ld_rowstat(P.rowstat + (int64_t)b * g1 + lane);
  const uint32_t info = ld_u32(row_word(P, b, kSeqInfo));
  if (!(info & kSeqInfoSet)) return;  // block-uniform
  const int f = (int)(info & 0xffu), kind = (int)((info >> 8) & 0xffu);
  const int64_t row = (int64_t)b * g1 + f;
  const RowStat rs = lane_rowstat(mine, f);
  const SeqParam sp = seq_param(P, b);
  const bool residual = kind == kResidual || kind == kTokRes;
  if (residual) {
    const int w = threadIdx.x >> 6;
    if (kind == kTokRes) res_slice_w<DT, VEC, kTokRes>(P, b, k * kSlices + w, f, rs);
    else res_slice_w<DT, VEC, kResidual>(P, b, k * kSlices + w, f, rs);
    vmem_drain();
  }
  __syncthreads();  // every wavefront's masses are stored
  if (threadIdx.x >= 64) return;
  if (!residual && k == 0) {
    const int src = kind == kQ ? kSrcStatsQ : kind == kP ? kSrcStatsP : kSrcTokPi;
    draw_w<DT, VEC>(P, b, row, kind, src, sp, ld_rowstat(P.rowstat + row));
    vmem_drain();
  }
  if (arrive_last_w(row_word(P, b, kSeqResArrive), (uint32_t)P.nt)) {
    if (residual) draw_w<DT, VEC>(P, b, row, kind, kSrcPass, sp, ld_rowstat(P.rowstat + row));
    if ((threadIdx.x & 63) == 0) st_u32(row_word(P, b, kSeqInfo), 0u);
  }
}

// Thread 0 of each workgroup, after reading the pass's job counts: arrive
// on one of kExitLeaves leaf counters; the last of a leaf arrives on the
// top counter, and the last there clears the pass's counts (every workgroup
// has read them by then).  Two levels keep the arrivals on one line few.
__device__ __forceinline__ void exit_tree(const Params& P) {
  const uint32_t G = gridDim.x, g = blockIdx.x;
  const uint32_t leaf = g % kExitLeaves;
  const uint32_t n_leaf = (G - leaf + kExitLeaves - 1) / kExitLeaves;
  const uint32_t n_top = G < (uint32_t)kExitLeaves ? G : (uint32_t)kExitLeaves;
  uint32_t* lc = hdr_word(P, kHdrExit + (int)leaf);
  uint32_t* tc = hdr_word(P, kHdrExit + kExitLeaves);
  if (add_u32(lc, 1u) != n_leaf - 1u) return;
  st_u32(lc, 0u);
  if (add_u32(tc, 1u) != n_top - 1u) return;
  st_u32(tc, 0u);
  st_u32(hdr_word(P, kHdrJobs), 0u);
}

// The job pass: a static walk over the jobs the statistics kernel of this
// call published: a slice of a TV row (batches of mixed rules), a slice of
// a tile a token row listed for eta, a TV tile whose wait timed out, an
// argmax half.  Wavefront w of the grid takes
// items w, w + W, ...  The item that completes a job decides its row; a
// sequence that decision finishes is drawn by the draw pass that follows.
// Held to 128 VGPRs: two workgroups per compute unit.
template <int DT, bool VEC>
__global__ __launch_bounds__(kJobThreads) __attribute__((amdgpu_waves_per_eu(4))) void k_jobs(
    Params P) {
  __shared__ uint32_t count;
  const int nt = P.nt, g1 = P.gamma + 1;
  if (threadIdx.x == 0) {
    if (gridDim.x == 1) {
      count = xchg_u32(hdr_word(P, kHdrJobs), 0u);  // the only reader takes and clears it
    } else {
      count = ld_u32(hdr_word(P, kHdrJobs));
      vmem_drain();  // the count has arrived before this workgroup counts itself
      exit_tree(P);
    }
  }
  __syncthreads();
  const int64_t n_items = min((int64_t)count, P.single_slots);
  const uint64_t* singles = job_list(P);
  constexpr int kW = kJobThreads / 64;
  const int64_t W = (int64_t)gridDim.x * kW;
  const int lane = threadIdx.x & 63;
  // this wavefront's items are g0, g0 + W, ...; the entries of up to 64 of
  // them are requested at once (lane l: item base + l W), so that an item's
  // work starts without a round trip for its entry
  for (int64_t base = (int64_t)blockIdx.x * kW + (threadIdx.x >> 6); base < n_items;
       base += 64 * W) {
    const int64_t gl = base + (int64_t)lane * W;
    const uint64_t mine = gl < n_items ? ld_u64(singles + gl) : 0ull;
    const int cnt = (int)min<int64_t>(64, (n_items - base + W - 1) / W);
#pragma unroll 1
    for (int i = 0; i < cnt; ++i) {
      const uint64_t e = lane_u64(mine, i);
      const int kind = job_kind(e);
      const int id = (int)job_id(e);
      if (kind == kJobTvTile) {
        // a tile whose wait for its row's merge timed out: its four slices,
        // unless the row was decided without a TV pass
        if (ld_u32(row_word(P, id, kRowReady)) == 2u) {  // wave-uniform
          tv_skip_arrive_w(P, id);
          continue;
        }
        const SeqParam spt = seq_param(P, id / g1);
#pragma unroll 1
        for (int w = 0; w < kSlices; ++w)
          pass2_slice_w<DT, VEC, false>(P, id, (int)job_extra(e), w, spt);
        if (arrive_last_w(row_word(P, id, kRowTvArrive), (uint32_t)(kSlices * nt), kSlices))
          tv_row_done<DT>(P, id);
      } else if (kind == kJobTvSlice) {
        // slice x % 4 of tile x / 4 of TV row id
        const int x = (int)job_extra(e);
        pass2_slice_w<DT, VEC, false>(P, id, x / kSlices, x % kSlices, seq_param(P, id / g1));
        if (arrive_last_w(row_word(P, id, kRowTvArrive), (uint32_t)(kSlices * nt)))
          tv_row_done<DT>(P, id);
      } else if (kind == kJobEta) {
        // slice c % 4 of the (c / 4)-th listed tile of token row id
        const uint32_t n = (uint32_t)ld_i32(P.etacnt + id) * (uint32_t)kSlices;
        pass2_item_w<DT, VEC, true>(P, id, (int)job_extra(e));
        if (arrive_last_w(row_word(P, id, kRowTvArrive), n)) row_job_decide<DT>(P, kind, id);
      } else {  // kJobArg
        arg_half_w<DT, VEC>(P, id, (int)job_extra(e));
        if (arrive_last_w(row_word(P, id, kRowJobDone), 2u)) row_job_decide<DT>(P, kind, id);
      }
    }
  }
}

template <int DT, bool VEC>
hipError_t launch_step_t(const Params& P, hipStream_t st, bool draw_pass, bool tv_pass,
                         bool job_pass, int job_groups, hipEvent_t ev_begin, hipEvent_t ev_end) {
  const dim3 grid((unsigned)P.nt, (unsigned)(P.B * (P.gamma + 1))), block(kThreads);
  if (ev_begin) {
    const hipError_t e = hipEventRecord(ev_begin, st);
    if (e != hipSuccess) return e;
  }
  constexpr int kAll = kMomX | kMomHQ | kMomHP;
  if (!P.tv_self && P.pair && P.mom_set == 0) {
    const dim3 grid2((unsigned)((P.nt + 1) / 2), (unsigned)(P.B * (P.gamma + 1)));
    hipLaunchKernelGGL((k_tiles<DT, VEC, 0, kTvNone, true>), grid2, block, 0, st, P);
  } else if (!P.tv_self) {
    if (P.mom_set == 0)
      hipLaunchKernelGGL((k_tiles<DT, VEC, 0, kTvNone>), grid, block, 0, st, P);
    else if (P.mom_set == kMomX)
      hipLaunchKernelGGL((k_tiles<DT, VEC, kMomX, kTvNone>), grid, block, 0, st, P);
    else if (P.mom_set == kMomHQ)
      hipLaunchKernelGGL((k_tiles<DT, VEC, kMomHQ, kTvNone>), grid, block, 0, st, P);
    else
      hipLaunchKernelGGL((k_tiles<DT, VEC, kAll, kTvNone>), grid, block, 0, st, P);
  } else {
    if (P.mom_set == 0)
      hipLaunchKernelGGL((k_tiles<DT, VEC, 0, kTvSelf>), grid, block, 0, st, P);
    else
      hipLaunchKernelGGL((k_tiles<DT, VEC, kAll, kTvSelf>), grid, block, 0, st, P);
  }
  hipError_t err = hipGetLastError();
  if (err == hipSuccess && ev_end) err = hipEventRecord(ev_end, st);
  if (err == hipSuccess && tv_pass) {
    hipLaunchKernelGGL((k_tvpass<DT, VEC>), grid, block, 0, st, P);
    err = hipGetLastError();
  }
  if (err == hipSuccess && job_pass) {
    hipLaunchKernelGGL((k_jobs<DT, VEC>), dim3((unsigned)job_groups), dim3(kJobThreads), 0, st,
                       P);
    err = hipGetLastError();
  }
  if (err == hipSuccess && draw_pass) {  // every sequence is finished by now
    hipLaunchKernelGGL((k_res<DT, VEC>), dim3((unsigned)P.nt, (unsigned)P.B), block, 0, st, P);
    err = hipGetLastError();
  }
  return err;
}

// ================================================================ small problems
// k_small: one launch for a batch whose rows fit in one workgroup's registers
// (V up to kSmallThreads * kSmallU lane loads of VW entries).  grid (R),
// 1024 threads: workgroup r holds row r of q and p (thread t's lane load i
// covers entries (i * 1024 + t) * VW ..), reduces it to the row statistics,
// takes the second pass (TV or eta) from the same registers, decides the row,
// and computes, also from registers, the sub-chunk masses of the
// distribution it would be sampled from if it were the sequence's j*.  The
// last row of a sequence to arrive finds j* and draws: a search over row j*'s
// stored masses, then one sub-chunk read again.  No tile is read twice.
constexpr int kSmallThreads = 1024;
constexpr int kSmallWaves = kSmallThreads / 64;
constexpr int kSmallU = 4;
static_assert(kSmallU * kSmallWaves == kSmallSub, "sub-chunks per row of the small path");

template <int DT, bool VEC>
struct SmallRow {
  using T = Tile<DT, VEC, kSmallU>;  // element geometry (EB, VW, NW)
  static constexpr int N = kSmallThreads * kSmallU * T::VW;  // entries a workgroup holds
};

// The packed words stay live across the passes over a row; each pass unpacks
// them again (otherwise the compiler keeps every unpacked entry of the
// previous pass, twice the registers).
template <int NW>
__device__ __forceinline__ void small_fence(uint32_t (&wq)[kSmallU][NW], uint32_t (&wp)[kSmallU][NW]) {
#pragma unroll
  for (int i = 0; i < kSmallU; ++i)
#pragma unroll
    for (int k = 0; k < NW; ++k) asm volatile("" : "+v"(wq[i][k]), "+v"(wp[i][k]));
}

struct SmallShared {
  float m[kSmallWaves][2];
  double d[kSmallWaves][2];
  double h[kSmallWaves][3];
  int i[kSmallWaves][2];
  double a[kSmallWaves];
  RowStat rs;
  float zx[2];  // q and p logits at the draft token (or p at the drafter's argmax)
  int delta, kind;
};

// Whole block: sum of one double per thread, combined in wave order.
__device__ __forceinline__ double small_sum(double v, SmallShared& sh) {
  v = wave_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh.a[threadIdx.x >> 6] = v;
  __syncthreads();
  double t = sh.a[0];
#pragma unroll
  for (int w = 1; w < kSmallWaves; ++w) t += sh.a[w];
  return t;
}

// Whole block: the row statistics from the registers, as the statistics
// tiles and the row merge compute them: per thread against its own maximum,
// per wavefront against the wavefront's, then (fp64) against the row's; with
// ARG the lowest index of each row maximum, with MOM the first moments.
template <int DT, bool VEC>
using SmallRegs = uint32_t[kSmallU][Tile<DT, VEC, kSmallU>::NW];

// Thread t's lane load i of a row (entries (i * 1024 + t) * VW ..), raw: a
// lane load past the row reads the row's first entries instead, and every
// pass reads it as -inf through small_elem (a lane load is wholly inside or
// wholly outside the row).  Keeping the raw words, rather than selecting
// the padding once, spares the registers of a second copy.
template <int DT, bool VEC>
__device__ __forceinline__ void small_load(const char* row, int V, SmallRegs<DT, VEC>& w) {
  using T = Tile<DT, VEC, kSmallU>;
#pragma unroll
  for (int i = 0; i < kSmallU; ++i) {
    const int e = (i * kSmallThreads + (int)threadIdx.x) * T::VW;
    const char* a = row + (uint32_t)((e < V ? e : 0) * T::EB);
    if constexpr (VEC) {
      const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(a));
      w[i][0] = v.x;
      w[i][1] = v.y;
      w[i][2] = v.z;
      w[i][3] = v.w;
    } else if constexpr (DT == 1) {
      w[i][0] = *reinterpret_cast<const uint16_t*>(a);
    } else {
      w[i][0] = *reinterpret_cast<const uint32_t*>(a);
    }
  }
}

template <int DT, bool VEC>
__device__ __forceinline__ bool small_ok(int i, int V) {
  return (i * kSmallThreads + (int)threadIdx.x) * Tile<DT, VEC, kSmallU>::VW < V;
}

// Whether any lane of this wavefront holds entries of lane load i
// (wavefront-uniform): lane loads wholly past the row are skipped.
template <int DT, bool VEC>
__device__ __forceinline__ bool small_live(int i, int V) {
  return (i * kSmallThreads + (int)(threadIdx.x & ~63)) * Tile<DT, VEC, kSmallU>::VW < V;
}

template <int DT, bool VEC>
__device__ __forceinline__ float small_elem(const uint32_t* w, int e, bool ok) {
  return ok ? elem<DT, VEC>(w, e) : kNegInf;
}

template <int DT, bool VEC, int MOM, bool ARG>
__device__ __forceinline__ RowStat small_stats(SmallRegs<DT, VEC>& wq, SmallRegs<DT, VEC>& wp,
                                               int V, const SeqParam& sp, int mrule,
                                               SmallShared& sh) {
  using T = Tile<DT, VEC, kSmallU>;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  float mq = kNegInf, mp = kNegInf;
#pragma unroll
  for (int i = 0; i < kSmallU; ++i) {
    if (!small_live<DT, VEC>(i, V)) continue;  // wavefront-uniform
    const bool ok = small_ok<DT, VEC>(i, V);
#pragma unroll
    for (int e = 0; e < T::VW; ++e) {
      mq = fmaxf(mq, small_elem<DT, VEC>(wq[i], e, ok));
      mp = fmaxf(mp, small_elem<DT, VEC>(wp[i], e, ok));
    }
  }
  small_fence(wq, wp);
  int iq = 0x7fffffff, ip = 0x7fffffff;
  if constexpr (ARG) {
    // the first entry equal to the thread maximum, entries in index order
#pragma unroll
    for (int i = kSmallU - 1; i >= 0; --i) {
      if (!small_live<DT, VEC>(i, V)) continue;  // wavefront-uniform
      const bool ok = small_ok<DT, VEC>(i, V);
#pragma unroll
      for (int e = T::VW - 1; e >= 0; --e) {
        const int idx = (i * kSmallThreads + (int)threadIdx.x) * T::VW + e;
        if (small_elem<DT, VEC>(wq[i], e, ok) == mq) iq = idx;
        if (small_elem<DT, VEC>(wp[i], e, ok) == mp) ip = idx;
      }
    }
    if (mq == kNegInf) iq = 0x7fffffff;
    if (mp == kNegInf) ip = 0x7fffffff;
    small_fence(wq, wp);
  }
  const float rq = (mq == kNegInf) ? 0.0f : mq * sp.c_hi;
  const float rp = (mp == kNegInf) ? 0.0f : mp * sp.c_hi;
  float sq = 0.0f, spp = 0.0f, hq = 0.0f, hp = 0.0f, xq = 0.0f;
#pragma unroll
  for (int i = 0; i < kSmallU; ++i) {
    if (!small_live<DT, VEC>(i, V)) continue;  // wavefront-uniform
    const bool ok = small_ok<DT, VEC>(i, V);
#pragma unroll
    for (int e = 0; e < T::VW; ++e) {
      const float zq = small_elem<DT, VEC>(wq[i], e, ok), zp = small_elem<DT, VEC>(wp[i], e, ok);
      const float aq = fmaf(zq, sp.c_lo, fmaf(zq, sp.c_hi, -rq));
      const float ap = fmaf(zp, sp.c_lo, fmaf(zp, sp.c_hi, -rp));
      const float tq = exp2_hw(aq), tp = exp2_hw(ap);
      sq += tq;
      spp += tp;
      if constexpr (MOM) {
        hq = fmaf(tq, tq > 0.0f ? aq : 0.0f, hq);
        xq = fmaf(tq, tq > 0.0f ? ap : 0.0f, xq);
        hp = fmaf(tp, tp > 0.0f ? ap : 0.0f, hp);
      }
      if (e & 1) __builtin_amdgcn_sched_barrier(0);
    }
  }
  small_fence(wq, wp);
  // waves against the wave max, then the block against the row max (fp64)
  const float Wq = wave_max(mq), Wp = wave_max(mp);
  const double eq = (double)rq - (double)(Wq * sp.c_hi), ep = (double)rp - (double)(Wp * sp.c_hi);
  const double fq = exp2_acc(eq), fp = exp2_acc(ep);
  const double dq = wave_sum(mq == kNegInf ? 0.0 : (double)sq * fq);
  const double dp = wave_sum(mp == kNegInf ? 0.0 : (double)spp * fp);
  double mhq = 0.0, mhp = 0.0, mx = 0.0;
  if constexpr (MOM) {
    mhq = wave_sum(mq == kNegInf ? 0.0 : mom_move(hq, sq, fq, eq));
    mhp = wave_sum(mp == kNegInf ? 0.0 : mom_move(hp, spp, fp, ep));
    mx = wave_sum(mq == kNegInf ? 0.0 : mom_move(xq, sq, fq, ep));
  }
  if constexpr (ARG) {
    iq = wave_min(mq == Wq ? iq : 0x7fffffff);
    ip = wave_min(mp == Wp ? ip : 0x7fffffff);
  }
  if (lane == 0) {
    sh.m[wv][0] = Wq;
    sh.m[wv][1] = Wp;
    sh.d[wv][0] = dq;
    sh.d[wv][1] = dp;
    sh.h[wv][0] = mhq;
    sh.h[wv][1] = mhp;
    sh.h[wv][2] = mx;
    sh.i[wv][0] = iq;
    sh.i[wv][1] = ip;
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    // wave 0 combines the wavefronts, lane w taking wavefront w's partials
    const bool in = lane < kSmallWaves;
    const int w = in ? lane : 0;
    const float wq_ = in ? sh.m[w][0] : kNegInf, wp_ = in ? sh.m[w][1] : kNegInf;
    const float Mq = wave_max(wq_), Mp = wave_max(wp_);
    const double Rq = (double)(Mq * sp.c_hi), Rp = (double)(Mp * sp.c_hi);
    const double gq = wq_ == kNegInf ? 0.0 : (double)(wq_ * sp.c_hi) - Rq;
    const double gp = wp_ == kNegInf ? 0.0 : (double)(wp_ * sp.c_hi) - Rp;
    const double fq_ = exp2_acc(gq), fp_ = exp2_acc(gp);
    const double Sq = wave_sum(wq_ != kNegInf ? sh.d[w][0] * fq_ : 0.0);
    const double Sp = wave_sum(wp_ != kNegInf ? sh.d[w][1] * fp_ : 0.0);
    double Hq = 0.0, Hp = 0.0, X = 0.0;
    if constexpr (MOM) {
      Hq = wave_sum(wq_ != kNegInf ? mom_move(sh.h[w][0], sh.d[w][0], fq_, gq) : 0.0);
      Hp = wave_sum(wp_ != kNegInf ? mom_move(sh.h[w][1], sh.d[w][1], fp_, gp) : 0.0);
      X = wave_sum(wq_ != kNegInf ? mom_move(sh.h[w][2], sh.d[w][0], fq_,
                                             wp_ == kNegInf ? -__builtin_huge_val() : gp)
                                  : 0.0);
    }
    const int aq = wave_min(in && wq_ == Mq ? sh.i[w][0] : 0x7fffffff);
    const int ap = wave_min(in && wp_ == Mp ? sh.i[w][1] : 0x7fffffff);
    RowStat rs;
    const double lq2 = log2_acc(Sq), lp2 = log2_acc(Sp);
    rs.lz_q = (Mq == kNegInf ? (double)kNegInf : Rq) + lq2;
    rs.lz_p = (Mp == kNegInf ? (double)kNegInf : Rp) + lp2;
    rs.tv = 0.0;
    rs.slog = (MOM && mrule) ? log_stat(mrule, lq2, lp2, Sq, Sp, Hq, Hp, X) : 0.0;
    rs.zmax_q = Mq;
    rs.zmax_p = Mp;
    rs.amax_q = (ARG && aq != 0x7fffffff) ? aq : -1;
    rs.amax_p = (ARG && ap != 0x7fffffff) ? ap : -1;
    if (lane == 0) sh.rs = rs;
  }
  __syncthreads();
  return sh.rs;
}

// Thread: sum over its entries of the sampled distribution KIND's weights
// for lane load i (float, entry order).
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ float small_weight_row(const uint32_t (&wq)[Tile<DT, VEC, kSmallU>::NW],
                                                  const uint32_t (&wp)[Tile<DT, VEC, kSmallU>::NW],
                                                  bool ok, const ProbScale& ps, int kind) {
  float t = 0.0f;
#pragma unroll
  for (int e = 0; e < Tile<DT, VEC, kSmallU>::VW; ++e) {
    t += weight_k<DT, KIND>(small_elem<DT, VEC>(wq, e, ok), small_elem<DT, VEC>(wp, e, ok), ps, kind);
    if (e & 1) __builtin_amdgcn_sched_barrier(0);
  }
  return t;
}

// Whole block: the masses of the row's sub-chunks under KIND (sub-chunk
// i * 16 + w is wave w's lane load i), stored as set `set` of the row for
// the sequence's draw; returns their total.
template <int DT, bool VEC, int KIND>
__device__ __forceinline__ double small_masses(const Params& P, int r, int set, int kind,
                                               const uint32_t (&wq)[kSmallU][Tile<DT, VEC, kSmallU>::NW],
                                               const uint32_t (&wp)[kSmallU][Tile<DT, VEC, kSmallU>::NW],
                                               const ProbScale& ps, SmallShared& sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  double tot = 0.0;
#pragma unroll
  for (int i = 0; i < kSmallU; ++i) {
    double m = 0.0;
    if (small_live<DT, VEC>(i, P.V))  // wavefront-uniform
      m = wave_sum((double)small_weight_row<DT, VEC, KIND>(wq[i], wp[i], small_ok<DT, VEC>(i, P.V),
                                                           ps, kind));
    if (lane == 0)
      st_dev_f64(P.submass + ((int64_t)r * 2 + set) * kSmallSub + i * kSmallWaves + wv, m);
    tot += m;
    __builtin_amdgcn_sched_barrier(0);
  }
  return small_sum(lane == 0 ? tot : 0.0, sh);
}

template <int DT, bool VEC>
__device__ __forceinline__ double small_masses_kind(const Params& P, int r, int set, int kind,
                                                    const uint32_t (&wq)[kSmallU][Tile<DT, VEC, kSmallU>::NW],
                                                    const uint32_t (&wp)[kSmallU][Tile<DT, VEC, kSmallU>::NW],
                                                    const ProbScale& ps, SmallShared& sh) {
  if (kind == kResidual) return small_masses<DT, VEC, kResidual>(P, r, set, kind, wq, wp, ps, sh);
  if (kind == kTokRes) return small_masses<DT, VEC, kTokRes>(P, r, set, kind, wq, wp, ps, sh);
  if (kind == kQ) return small_masses<DT, VEC, kQ>(P, r, set, kind, wq, wp, ps, sh);
  if (kind == kP) return small_masses<DT, VEC, kP>(P, r, set, kind, wq, wp, ps, sh);
  return small_masses<DT, VEC, kTokPi>(P, r, set, kind, wq, wp, ps, sh);
}

// Wave: the draw of sequence b at row j* = f from that row's stored
// sub-chunk masses under `kind`: the sub-chunk where u W is crossed, then
// the entry inside it (read again).
template <int DT, bool VEC>
__device__ __forceinline__ void small_draw_w(const Params& P, int b, int f, int kind, int set,
                                             const SeqParam& sp) {
  const int64_t row = (int64_t)b * (P.gamma + 1) + f;
  const RowStat rs = ld_rowstat(P.rowstat + row);
  const float u = P.uniforms[(int64_t)b * (P.gamma + 1) + P.gamma];
  int ks;
  double rem;
  // set `set` of the row's masses, read as the residual search reads a
  // sequence's (nsub = kSmallSub)
  const double W = find_part<kSrcPass, kSmallSub / 64>(P, row, (int)(row * 2 + set), kSmallSub,
                                                       rs, u, &ks, &rem);
  if ((threadIdx.x & 63) == 0) {
    if (P.out_norm) P.out_norm[b] = (float)W;
    if (ks < 0) P.out_token[b] = -1;
  }
  if (ks < 0) return;  // wave-uniform
  const ProbScale ps = prob_scale(sp, rs, kind == kTokRes || kind == kTokPi);
  const int64_t c0 = (int64_t)ks * SubC<DT, VEC>::N;
  if (kind == kResidual) pick_wave<DT, VEC, SubC<DT, VEC>, kResidual>(P, b, row, c0, rem, ps);
  else if (kind == kTokRes) pick_wave<DT, VEC, SubC<DT, VEC>, kTokRes>(P, b, row, c0, rem, ps);
  else if (kind == kQ) pick_wave<DT, VEC, SubC<DT, VEC>, kQ>(P, b, row, c0, rem, ps);
  else if (kind == kP) pick_wave<DT, VEC, SubC<DT, VEC>, kP>(P, b, row, c0, rem, ps);
  else pick_wave<DT, VEC, SubC<DT, VEC>, kTokPi>(P, b, row, c0, rem, ps);
}

template <int DT, bool VEC, int MS>
__global__ __launch_bounds__(kSmallThreads) void k_small(Params P) {
  using T = Tile<DT, VEC, kSmallU>;
  __shared__ SmallShared sh;
  const int r = blockIdx.x, gamma = P.gamma, g1 = gamma + 1, V = P.V;
  const int b = r / g1, j = r - b * g1;
  const int lane = threadIdx.x & 63;
  const SeqParam sp = seq_param(P, b);
  const int x = (sp.valid && j < gamma) ? P.draft[(int64_t)b * gamma + j] : -1;
  const float u = (sp.valid && !sp.greedy) ? P.uniforms[r] : 0.0f;
  uint32_t wq[kSmallU][T::NW], wp[kSmallU][T::NW];
  small_load<DT, VEC>((const char*)P.q + (int64_t)r * V * T::EB, V, wq);
  small_load<DT, VEC>((const char*)P.p + (int64_t)r * V * T::EB, V, wp);
  const int mrule = (MS != 0 && needs_mom(sp)) ? sp.rule : 0;
  RowStat rs;
  if (sp.greedy)  // block-uniform
    rs = (MS != 0 && mrule) ? small_stats<DT, VEC, 1, true>(wq, wp, V, sp, mrule, sh)
                            : small_stats<DT, VEC, 0, true>(wq, wp, V, sp, 0, sh);
  else
    rs = (MS != 0 && mrule) ? small_stats<DT, VEC, 1, false>(wq, wp, V, sp, mrule, sh)
                            : small_stats<DT, VEC, 0, false>(wq, wp, V, sp, 0, sh);
  // the logits the decision reads, from the thread holding them: the draft
  // token's, or (greedy TokenV2/V3, BiLD*) p's at the drafter's argmax
  int xi = x;
  if (sp.valid && sp.greedy)
    xi = ((is_token(sp.rule) && sp.rule != SPC_RULE_TOKEN_V1) || sp.rule == SPC_RULE_BILD)
             ? rs.amax_q : -1;
  if (threadIdx.x == 0) {
    sh.zx[0] = 0.0f;
    sh.zx[1] = 0.0f;
  }
  __syncthreads();
  if (xi >= 0 && xi < V) {
    const int slot = xi / T::VW, e = xi - slot * T::VW;
    if (slot % kSmallThreads == (int)threadIdx.x) {
      const int i = slot / kSmallThreads;
      float zq = 0.0f, zp = 0.0f;
#pragma unroll
      for (int ii = 0; ii < kSmallU; ++ii)
        if (ii == i) {
#pragma unroll
          for (int ee = 0; ee < T::VW; ++ee)
            if (ee == e) {
              zq = elem<DT, VEC>(wq[ii], ee);
              zp = elem<DT, VEC>(wp[ii], ee);
            }
        }
      sh.zx[0] = sp.greedy ? 0.0f : zq;
      sh.zx[1] = zp;
    }
  }
  // the second pass from the registers: D_TV (OPT, OPTLOG) or eta (token
  // rules) at temperature > 0
  const bool tv = sp.valid && !sp.greedy && has_tv_parts(sp.rule);
  const bool eta = sp.valid && !sp.greedy && is_token(sp.rule);
  if (tv || eta) {  // block-uniform
    const ProbScale ps = prob_scale(sp, rs, eta);
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < kSmallU; ++i) {
      if (!small_live<DT, VEC>(i, V)) continue;  // wavefront-uniform
      const bool ok = small_ok<DT, VEC>(i, V);
      float t = 0.0f;
#pragma unroll
      for (int e = 0; e < T::VW; ++e) {
        const float zq = small_elem<DT, VEC>(wq[i], e, ok), zp = small_elem<DT, VEC>(wp[i], e, ok);
        if (eta) {
          t += token_r(ps.tok, zq, zp) ? prob(zq, ps.c_hi, ps.c_lo, ps.q_hi, ps.q_lo) : 0.0f;
        } else {
          const float pq = prob(zq, ps.c_hi, ps.c_lo, ps.q_hi, ps.q_lo);
          const float pp = prob(zp, ps.c_hi, ps.c_lo, ps.p_hi, ps.p_lo);
          t += fmaxf(pp - pq, 0.0f);
        }
        if (e & 1) __builtin_amdgcn_sched_barrier(0);
      }
      acc += (double)t;
    }
    rs.tv = small_sum(acc, sh);
    small_fence(wq, wp);
  }
  // The distributions this row may be drawn from if it is the sequence's
  // j*: set 0 for a deferring row (delta = 1) or the rule's fixed kind, set 1
  // for delta = 0 or for an empty residual (replaced by p).  Both come from
  // the registers before the decision, which then needs none of them.
  int kind0 = kNone, kind1 = kNone;
  if (sp.valid && !sp.greedy) {
    if (is_token(sp.rule)) {
      kind0 = j < gamma ? kTokRes : kTokPi;
      kind1 = j < gamma ? kP : kNone;
    } else if (sp.rule == SPC_RULE_LOSSY) {
      kind0 = j < gamma ? kResidual : kP;
      kind1 = j < gamma ? kP : kNone;
    } else {
      kind0 = j < gamma ? kResidual : kP;
      kind1 = j < gamma ? kP : kQ;
    }
  }
  double W0 = 0.0;
  if (kind0 != kNone)  // block-uniform
    W0 = small_masses_kind<DT, VEC>(P, r, 0, kind0, wq, wp,
                                    prob_scale(sp, rs, kind0 == kTokRes || kind0 == kTokPi), sh);
  small_fence(wq, wp);
  if (kind1 != kNone)
    (void)small_masses_kind<DT, VEC>(P, r, 1, kind1, wq, wp, prob_scale(sp, rs, false), sh);
  __syncthreads();  // the logits at the draft token are in shared memory
  // the decision (wave 0)
  if (threadIdx.x < 64) {
    RowDecision d{};
    if (sp.valid) d = decide_row(sp, rs, j, gamma, V, x, sh.zx[0], sh.zx[1], u);
    if (lane == 0) {
      int set = 0;
      if (sp.valid && !sp.greedy) {
        const bool empty = (kind0 == kResidual || kind0 == kTokRes) && !(W0 > 0.0);
        set = (is_token(sp.rule) || sp.rule == SPC_RULE_LOSSY) ? (empty ? 1 : 0)
                                                                : (d.delta && !empty ? 0 : 1);
      }
      const int kind = set ? kind1 : kind0;
      row_record(P, r, sp, d, (kind < 0 ? 0 : kind) | (set << 4));
    }
  }
  vmem_drain();
  __syncthreads();  // every store of this row is complete
  if (threadIdx.x >= 64) return;
  if (!arrive_last_w(row_word(P, b, kSeqResArrive), (uint32_t)g1)) return;
  // the last row of sequence b: j* is its first rejection
  const int rec = lane < g1 ? ld_i32(P.rowdec + (int64_t)b * g1 + lane) : 0;
  const unsigned long long rej = __ballot(lane < g1 && !(rec & 1));
  const int f = rej ? __ffsll(rej) - 1 : gamma;
  const int recf = lane_i32(rec, f);
  if (!sp.valid) {
    if (lane == 0) {
      P.out_accept[b] = -1;
      P.out_token[b] = -1;
      if (P.out_norm) P.out_norm[b] = 0.0f;
    }
    return;
  }
  if (lane == 0) P.out_accept[b] = f;
  if (sp.greedy) {
    if (lane == 0) {
      const RowStat rf = ld_rowstat(P.rowstat + (int64_t)b * g1 + f);
      const int dstar = (recf >> 1) & 1;
      P.out_token[b] = (dstar || sp.rule == SPC_RULE_LOSSY) ? rf.amax_p : rf.amax_q;
      if (P.out_norm) P.out_norm[b] = 1.0f;
    }
    return;
  }
  small_draw_w<DT, VEC>(P, b, f, (recf >> 4) & 0xf, (recf >> 8) & 1, sp);
}

template <int DT, bool VEC>
hipError_t launch_small_t(const Params& P, hipStream_t st, hipEvent_t ev_begin,
                          hipEvent_t ev_end) {
  if (ev_begin) {
    const hipError_t e = hipEventRecord(ev_begin, st);
    if (e != hipSuccess) return e;
  }
  // batches with first moments take the tile path (their registers would not
  // fit beside the row)
  if (P.mom_set != 0) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(P.B * (P.gamma + 1))), block(kSmallThreads);
  hipLaunchKernelGGL((k_small<DT, VEC, 0>), grid, block, 0, st, P);
  hipError_t err = hipGetLastError();
  if (err == hipSuccess && ev_end) err = hipEventRecord(ev_end, st);
  return err;
}

// Drafter sampling step (Alg. 4: x_{t+j} ~ q_{t+j}), one launch.  grid
// (nt, B): statistics tile k of row b of the drafter's logits, as in k_tiles
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


}  // namespace

int stat_tile_elems(int dtype, bool vec) {
  if (dtype == 1) return vec ? StatTile<1, true>::N : StatTile<1, false>::N;
  return vec ? StatTile<0, true>::N : StatTile<0, false>::N;
}

int tile_subchunks(int dtype, bool vec) {
  if (dtype == 1) return kSlices * (vec ? StatTile<1, true>::U : StatTile<1, false>::U);
  return kSlices * (vec ? StatTile<0, true>::U : StatTile<0, false>::U);
}

int draft_tile_elems(int dtype, bool vec, bool long_tiles) {
  if (long_tiles) {
    if (dtype == 1) return vec ? DraftTile<1, true, 2>::N : DraftTile<1, false, 2>::N;
    return vec ? DraftTile<0, true, 2>::N : DraftTile<0, false, 2>::N;
  }
  if (dtype == 1) return vec ? DraftTile<1, true, 1>::N : DraftTile<1, false, 1>::N;
  return vec ? DraftTile<0, true, 1>::N : DraftTile<0, false, 1>::N;
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

namespace {
// Zero fill with vector stores: a grid-stride loop over 32-bit words.
__global__ __launch_bounds__(256) void k_fill_zero(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
    p[i] = 0u;
}
}  // namespace

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t st) {
  const size_t n = bytes / 4;
  if (n == 0) return hipSuccess;
  const unsigned groups = (unsigned)std::min<size_t>((n + 255) / 256, 1024);
  hipLaunchKernelGGL(k_fill_zero, dim3(groups), dim3(256), 0, st, static_cast<uint32_t*>(ptr), n);
  return hipGetLastError();
}

int small_row_elems(int dtype, bool vec) {
  if (dtype == 1) return vec ? SmallRow<1, true>::N : SmallRow<1, false>::N;
  return vec ? SmallRow<0, true>::N : SmallRow<0, false>::N;
}

hipError_t launch_small(const Params& P, int dtype, bool vec, hipEvent_t ev_begin,
                        hipEvent_t ev_end, hipStream_t st) {
  if (dtype == 1)
    return vec ? launch_small_t<1, true>(P, st, ev_begin, ev_end)
               : launch_small_t<1, false>(P, st, ev_begin, ev_end);
  return vec ? launch_small_t<0, true>(P, st, ev_begin, ev_end)
             : launch_small_t<0, false>(P, st, ev_begin, ev_end);
}

hipError_t launch_step(const Params& P, int dtype, bool vec, bool draw_pass, bool tv_pass,
                       bool job_pass, int job_groups, hipEvent_t ev_begin, hipEvent_t ev_end,
                       hipStream_t st) {
  if (dtype == 1)
    return vec ? launch_step_t<1, true>(P, st, draw_pass, tv_pass, job_pass, job_groups, ev_begin,
                                        ev_end)
               : launch_step_t<1, false>(P, st, draw_pass, tv_pass, job_pass, job_groups,
                                         ev_begin, ev_end);
  return vec ? launch_step_t<0, true>(P, st, draw_pass, tv_pass, job_pass, job_groups, ev_begin,
                                      ev_end)
             : launch_step_t<0, false>(P, st, draw_pass, tv_pass, job_pass, job_groups, ev_begin,
                                       ev_end);
}

}  // namespace spc
