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
  int32_t amax_q, amax_p; // statistics tiles: bit w set when slice w attains zmax;
                          // drafter tiles: lowest row index attaining it, or -1
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

struct Params {
  const void* q;
  const void* p;
  const int32_t* draft;
  const float* uniforms;
  int32_t B, gamma, V;
  int32_t nt;              // statistics tiles per row
  int32_t rule;
  float alpha, temp;
  int32_t force_greedy;    // spc_greedy_verify: every sequence at temperature 0
  uint32_t rule_mask;      // rules per-sequence arrays may hold (0: any)
  int32_t mom_set;         // first moments the statistics tiles sum (kMom* bits; 0: none)
  const int32_t* rule_ps;
  const float* alpha_ps;
  const float* temp_ps;
  int32_t* out_accept;
  int32_t* out_token;
  uint8_t* out_defer;
  float* out_stats;
  int32_t* out_argmax;
  float* out_norm;
  // launch layout
  int64_t single_slots;    // jobs the job pass may hold: 2 R + B + R nt kSlices
  int32_t nsub;            // sub-chunks of a row: nt * tile_subchunks
  int32_t tv_self;         // TV rows get their TV pass from their own tiles' registers
  int32_t pair;            // statistics workgroups take two tiles each (large batches)
  int32_t tv_jobs;         // TV rows' slices are job-pass items (else the TV pass kernel)
  uint32_t wait_ticks;     // bound of a wait for a TV row's merge (100 MHz clock ticks)
  // workspace: zero region (counters; every launch leaves it as it found it)
  uint32_t* hdr;           // [kHdrLines][kLineWords] job counters
  uint32_t* rowline;       // [kMaxRows][kLineWords] per-row and per-sequence counters
  uint32_t* samp_cnt;      // drafter kernel: per-row completion counters (kDraftCntStride)
  // workspace: data (written before it is read in every launch)
  uint64_t* jobs;          // [single_slots] job entries of the job pass
  TilePart* tiles;         // [R][nt] statistics partials
  double* tvpart;          // [R][nt][kSlices] TV partials (OPT) or eta partials (token rules)
  double* submass;         // [B][nsub] residual masses per sub-chunk of row j*
  TileMom* moms;           // [R][nt] first moments (log-loss rules and BiLD*)
  RowStat* rowstat;        // [R] merged row statistics
  int32_t* rowdec;         // [R] bit 0 a_j, bit 1 delta_j
  int32_t* etalist;        // [R][nt] tiles whose eta share needs a second look
  int32_t* argres;         // [R][4] first tile of the q / p maximum (k * 16 + its slice
                           // mask), then the lowest index of the maximum
  int32_t* etacnt;         // [R] tiles listed in etalist
};

// Entries per statistics tile and per drafter tile for a dtype and load path.
int stat_tile_elems(int dtype, bool vec);
// Sub-chunks (lane-load rows of a wavefront) per statistics tile.
int tile_subchunks(int dtype, bool vec);
int draft_tile_elems(int dtype, bool vec, bool long_tiles);

// Counters live on 128-byte lines of 32-bit words: arrivals on a shared line
// serialise.
constexpr int kLineWords = 32;
constexpr int64_t kMaxRows = 16384;    // rows (and sequences) per launch
// Job passes: workgroups of kJobThreads threads whose wavefronts take items
// independently; a row job has kSlices items per statistics tile.
constexpr int kJobThreads = 512;
// A statistics tile splits into kSlices slices, one per wavefront of its
// workgroup (the unit of second-pass partials and residual jobs).
constexpr int kSlices = kThreads / 64;
// Header lines: the count of jobs published for the job pass (line 1; lines
// 0, 2 and 3 are spare), then kExitLeaves + 1 lines counting the workgroups
// of the pass that have read it (a two-level tree; the last arrival clears
// the count).
constexpr int kExitLeaves = 16;
constexpr int kHdrExit = 4;
constexpr int kHdrLines = kHdrExit + kExitLeaves + 1;

// Words of a row line (counters and flags, zero between calls): the row's
// tile arrivals, the decided-row mask of the sequence with the same index (64
// bits), the row's argmax-half arrivals, its "merged, TV pass open" flag and
// TV slice arrivals, the draw pass's arrivals for the sequence, the drafter
// kernel's per-row arrivals, and the sequence's outcome for the draw pass.
constexpr int kRowArrive = 0, kSeqMask = 2, kRowJobDone = 4, kRowReady = 5, kRowTvArrive = 6,
              kSeqResArrive = 7, kDraftArrive = 8, kSeqInfo = 9;
// A sequence's outcome word (kSeqInfo): kSeqInfoSet | sample kind << 8 | j*.
constexpr uint32_t kSeqInfoSet = 0x80000000u;

// Words between the drafter kernel's per-row completion counters.
constexpr int kDraftCntStride = kLineWords;

// Workspace layout for a shape; offsets in bytes from the base.  The zero
// region (header lines, row lines) has the same size for every shape.
struct WsLayout {
  size_t hdr, rowline, zero_end;
  size_t jobs, tiles, tvpart, submass, moms, rowstat, rowdec, etalist, argres, etacnt,
      total;
};
WsLayout ws_layout(int64_t B, int64_t gamma, int64_t V, int dtype, bool vec);

// Enqueue the drafter sampling kernel (Params: q = the logits [B][V], nt,
// uniforms [B], temp_ps or temp, out_token, samp_cnt with kDraftCntStride,
// tiles).  argmax: some row may be at temperature 0.
// long_tiles: tiles of twice the statistics tile's lane loads (large
// batches) rather than the statistics tile's (small ones).
hipError_t launch_draft(const Params& P, int dtype, bool vec, bool argmax, bool long_tiles,
                        hipStream_t stream);

// The small-problem path (k_small): a workgroup per row holding the row in
// registers; rows of at most small_row_elems entries, kSmallSub sub-chunks.
constexpr int kSmallSub = 64;
int small_row_elems(int dtype, bool vec);
hipError_t launch_small(const Params& P, int dtype, bool vec, hipEvent_t ev_begin,
                        hipEvent_t ev_end, hipStream_t stream);

// Enqueue one verify launch: the statistics tiles (k_tiles; with P.tv_self
// they also take their rows' TV passes), the TV pass kernel (k_tvpass) when
// `tv_pass`, the job pass (k_jobs, of `job_groups` workgroups) when
// `job_pass`, and last the draw pass (k_res) when `draw_pass`.
// ev_begin / ev_end (may be null): recorded right before and after k_tiles.
hipError_t launch_step(const Params& P, int dtype, bool vec, bool draw_pass, bool tv_pass,
                       bool job_pass, int job_groups, hipEvent_t ev_begin, hipEvent_t ev_end,
                       hipStream_t stream);

// Enqueue a kernel writing `bytes` zero bytes at `ptr` (a multiple of 4, ptr
// 4-byte aligned): a fill a graph capture may record.
hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream);

}  // namespace spc
