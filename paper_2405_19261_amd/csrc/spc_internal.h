// spc_internal.h -- structures shared by the C interface (spc_api.cpp) and the
// gfx950 kernels (spc_kernels.hip).  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "speccascade.h"

namespace spc {

constexpr int kThreads = 256;  // four 64-lane wavefronts per workgroup

// Sampling distribution at j* (Alg. 4): the residual max(0, p - q), or the
// extra-token target pi_{t+gamma}, which is q or p; for a token rule the
// residual max(0, pi - q) or pi_{t+gamma} of the target of Alg. 6.
enum SampleKind : int32_t { kNone = -1, kResidual = 0, kQ = 1, kP = 2, kTokRes = 3, kTokPi = 4 };

// Partial statistics of one (row, stats tile), both tensors.  With c the
// per-sequence log2(e)/T:  s = sum over the tile of 2^(z*c - r),  r the
// reference zmax * c_hi of the tile (-inf for an all -inf tile).
struct TilePart {
  double s_q, s_p;
  float r_q, r_p;
  float zmax_q, zmax_p;   // largest raw logit of the tile
  int32_t amax_q, amax_p; // lowest row index attaining it (greedy batches), else -1
};

// First moments of one (row, stats tile) for the log-loss rules and BiLD*,
// against the same references as its TilePart:  with a = z c - r,
//   hq = sum 2^a_q a_q,  hp = sum 2^a_p a_p,  x = sum 2^a_q a_p.
struct TileMom {
  double hq, hp, x;
};

// First moments (TileMom) a statistics pass may sum: x for BiLD*'s
// cross-entropy, hq for H(q), hp for H(p).
constexpr int kMomX = 1, kMomHQ = 2, kMomHP = 4;

// Per-row statistics after merging the tiles of a row.
struct RowStat {
  double lz_q, lz_p;      // log2 sum_v 2^(z_v * c)  (= lse / ln 2)
  double tv;              // D_TV(p, q) for OPT / OPTLOG rows, eta for token-rule rows, else 0
  double slog;            // a log-loss rule's statistic (nats): D(q,p), H(q) or H(q) - H(p)
  float zmax_q, zmax_p;
  int32_t amax_q, amax_p;
};

// Per-sequence decision, as the sampler needs it.
struct SeqState {
  int32_t row;   // j*
  int32_t kind;  // SampleKind
  float u;       // the sample's uniform u[b][gamma]
  int32_t pad;
};

struct Params {
  const void* q;
  const void* p;
  const int32_t* draft;
  const float* uniforms;
  int32_t B, gamma, V;
  int32_t nt;              // statistics tiles per row
  int32_t nc;              // residual chunks per row
  int32_t K;               // sampling workgroups per sequence
  int32_t rule;
  float alpha, temp;
  int32_t force_greedy;    // spc_greedy_verify: every sequence at temperature 0
  int32_t mom_split;       // the moment statistics kernel runs too: the plain one
                           // leaves it the rows that need first moments
  uint32_t rule_mask;      // rules per-sequence arrays may hold (0: any)
  int32_t mom_set;         // first moments the moment kernel sums (kMom* bits)
  const int32_t* rule_ps;
  const float* alpha_ps;
  const float* temp_ps;
  int32_t* out_accept;
  int32_t* out_token;
  uint8_t* out_defer;
  float* out_stats;
  int32_t* out_argmax;
  float* out_norm;
  // workspace
  uint32_t* samp_cnt;     // [B]   sampling workgroups of a sequence done
  uint32_t* row_cnt;      // [R][kRowCntStride] arrivals / departures per row (one read)
  TilePart* tiles;        // [R][nt] statistics partials
  double* tvpart;         // [R][nt] TV partials (OPT) or eta partials (token rules)
  double* masses;         // [B][nc] residual chunk masses of row j*
  TileMom* moms;          // [R][nt] first moments (log-loss rules and BiLD*)
};

// Entries per statistics tile and per residual chunk for a dtype and load
// path, and sampling workgroups per sequence for a row of nc chunks in a batch
// of B sequences on a device of `cus` compute units.
int stat_tile_elems(int dtype, bool vec);
int draft_tile_elems(int dtype, bool vec, bool long_tiles);
int samp_chunk_elems(int dtype, bool vec);
int samp_groups(int64_t nc, int B, int cus);

// Workspace layout for a shape; offsets in bytes from the base.
struct WsLayout {
  size_t samp_cnt, draft_cnt, row_cnt, zero_end;
  size_t tiles, tvpart, masses, moms, total;
};
WsLayout ws_layout(int64_t B, int64_t gamma, int64_t V, int dtype, bool vec);

// Words between the drafter kernel's per-row completion counters (one
// counter per 128-byte line: arrivals on a shared line serialise).
constexpr int kDraftCntStride = 32;

// The one-read statistics kernel's per-row counters (arrivals, departures),
// one 128-byte line per row, for batches of at most kResRows rows.
constexpr int kRowCntStride = 32;
constexpr int64_t kResRows = 8192;

// Workgroups of the one-read statistics kernel resident per compute unit
// (0 if it cannot run).
int res_blocks_per_cu(int dtype, bool vec, bool argmax);

// Enqueue the drafter sampling kernel (Params: q = the logits [B][V], nt,
// uniforms [B], temp_ps or temp, out_token, samp_cnt with kDraftCntStride,
// tiles).  argmax: some row may be at temperature 0.
// long_tiles: tiles of twice the statistics tile's lane loads (large
// batches) rather than the statistics tile's (small ones).
hipError_t launch_draft(const Params& P, int dtype, bool vec, bool argmax, bool long_tiles,
                        hipStream_t stream);

// Second passes a batch may need (bits of tv_kinds): D_TV of OPT and OPTLOG
// rows, eta of token-rule rows, each at temperature > 0.
constexpr int kPassTv = 1, kPassEta = 2;

// Enqueue the kernels of one verify call.  tv_kinds: the second passes the
// batch may need (kPassTv | kPassEta); need_sample: it may hold
// sequences at temperature > 0; need_argmax: it may hold greedy (temperature
// 0) sequences; need_plain / need_mom: it may hold rows that need no first
// moments / rows that do (log-loss rules, BiLD* at temperature > 0), each
// kind handled by its own statistics kernel.  res_grid > 0 (a multiple of
// nt; only with tv_kinds and without need_mom): statistics and second pass in
// one cooperative launch of res_grid workgroups instead of two kernels.
// Returns the first launch error.
hipError_t launch_verify(const Params& P, int dtype, bool vec, int tv_kinds, bool need_sample,
                         bool need_argmax, bool need_plain, bool need_mom, int res_grid,
                         hipEvent_t ev_begin, hipEvent_t ev_end, hipStream_t stream);

}  // namespace spc
