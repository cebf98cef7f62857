// spc_api.cpp -- the C interface of libspeccascade (declared in
// include/speccascade.h): argument checks, workspace, kernel dispatch.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "spc_internal.h"

namespace {

thread_local std::string g_err;

spc_status fail(spc_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// The internal workspace of each device.  A buffer that had to grow is kept
// (not freed) until spc_release: kernels already enqueued, or captured in a
// graph, may still refer to it.
struct DevWorkspace {
  void* ptr = nullptr;
  size_t bytes = 0;
  std::vector<void*> retired;
};
std::mutex g_ws_mu;
std::map<int, DevWorkspace> g_ws;

std::mutex g_cu_mu;
std::map<int, int> g_cus;

// Compute units of device dev, read once per device; 0 on failure.
int cu_count(int dev) {
  std::lock_guard<std::mutex> lk(g_cu_mu);
  auto it = g_cus.find(dev);
  if (it != g_cus.end()) return it->second;
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) n = 0;
  if (n > 0) g_cus[dev] = n;
  return n;
}

bool vec_path(int dtype, int64_t V) {
  const int64_t eb = dtype == SPC_BF16 ? 2 : 4;
  return (V * eb) % 16 == 0;  // every row starts on a 16-byte boundary
}

int64_t stat_tiles(int dtype, bool vec, int64_t V) {
  const int64_t n = spc::stat_tile_elems(dtype, vec);
  return (V + n - 1) / n;
}

// Sequences per launch: whole sequences, at most kMaxRows rows (the
// statistics grid is tiles x rows; a row of V < 2^31 entries has fewer than
// 2^31 tiles).
int64_t seqs_per_launch(int64_t B, int64_t gamma) {
  return std::max<int64_t>(1, std::min(B, spc::kMaxRows / (gamma + 1)));
}

}  // namespace

namespace spc {

WsLayout ws_layout(int64_t B, int64_t gamma, int64_t V, int dtype, bool vec) {
  // The zero region (job counter lines, per-row lines) has the same size
  // and offset for every shape, so one zeroed workspace serves calls of any
  // shape it is large enough for; launches leave it as found.
  const int64_t R = B * (gamma + 1);
  const int64_t nt = stat_tiles(dtype, vec, V);
  WsLayout L;
  size_t o = 0;
  L.hdr = o;
  o = align_up(o + 4 * (size_t)(kHdrLines * kLineWords), 256);
  L.rowline = o;
  o = align_up(o + 4 * (size_t)(kMaxRows * kLineWords), 256);
  L.zero_end = o;
  // the job pass's list: at most 2 R argmax halves, R nt TV tiles handed
  // back by their workgroups or R nt 4 eta slices (a row is one or the
  // other), and B spare
  L.jobs = o; o = align_up(o + 8 * (size_t)(2 * R + B + R * nt * kSlices), 256);
  L.tiles = o; o = align_up(o + sizeof(TilePart) * R * nt, 256);
  L.tvpart = o; o = align_up(o + sizeof(double) * R * nt * kSlices, 256);
  // residual sub-chunk masses per sequence, or (small path) two sets per row
  L.submass = o;
  o = align_up(o + sizeof(double) * std::max<int64_t>(B * nt * tile_subchunks(dtype, vec),
                                                       R * 2 * kSmallSub), 256);
  L.moms = o; o = align_up(o + sizeof(TileMom) * R * nt, 256);
  L.rowstat = o; o = align_up(o + sizeof(RowStat) * R, 256);
  L.rowdec = o; o = align_up(o + sizeof(int32_t) * R, 256);
  L.etalist = o; o = align_up(o + sizeof(int32_t) * R * nt, 256);
  L.argres = o; o = align_up(o + sizeof(int32_t) * 4 * R, 256);
  L.etacnt = o; o = align_up(o + sizeof(int32_t) * R, 256);
  L.total = o;
  return L;
}

}  // namespace spc

namespace {

// Bound of a statistics workgroup's wait for a TV row's merge, in ticks of
// the 100 MHz real-time clock: 4000 (40 us).  SPC_TV_WAIT_TICKS overrides it
// (read at every call); a test sets 0 so that every wait gives up at once
// and the job pass takes the tiles.
uint32_t tv_wait_ticks() {
  const char* e = getenv("SPC_TV_WAIT_TICKS");
  if (!e || !*e) return 4000u;
  char* end = nullptr;
  const unsigned long v = strtoul(e, &end, 10);
  return (end && *end == '\0' && v <= 1000000ul) ? (uint32_t)v : 4000u;
}

spc_status check_shape(int32_t B, int32_t gamma, int32_t V) {
  if (B < 1 || gamma < 1 || gamma > SPC_MAX_GAMMA || V < 2)
    return fail(SPC_E_SHAPE, "bad shape B=%d gamma=%d V=%d (need B>=1, 1<=gamma<=%d, V>=2)", B,
                gamma, V, SPC_MAX_GAMMA);
  return SPC_OK;
}

// The layout of one launch of a verify call of this shape.
spc::WsLayout launch_layout(int32_t B, int32_t gamma, int32_t V, int dtype) {
  return spc::ws_layout(seqs_per_launch(B, gamma), gamma, V, dtype, vec_path(dtype, V));
}

bool capturing(hipStream_t stream) {
  hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &st) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return st != hipStreamCaptureStatusNone;
}

// The internal workspace of the current device, at least `bytes` long.  A
// new buffer has its zero region cleared on `stream` before any kernel that
// uses it; that cannot be recorded into a graph, so a call being captured
// that would need a larger buffer fails instead (make one eager call of the
// largest shape first, or pass a caller workspace).
spc_status internal_workspace(size_t bytes, size_t zero_bytes, hipStream_t stream, char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SPC_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(g_ws_mu);
  DevWorkspace& w = g_ws[dev];
  if (w.bytes < bytes) {
    if (capturing(stream))
      return fail(SPC_E_WORKSPACE,
                  "the internal workspace must grow to %zu bytes, which a stream capture cannot "
                  "record: make an eager call of this shape first, or pass a workspace",
                  bytes);
    const size_t want = bytes + bytes / 4;  // headroom for nearby shapes
    void* ptr = nullptr;
    e = hipMalloc(&ptr, want);
    if (e != hipSuccess) return fail(SPC_E_HIP, "hipMalloc(%zu): %s", want, hipGetErrorString(e));
    // zero the counters, ordered before this call's kernels on the same stream
    e = hipMemsetAsync(ptr, 0, zero_bytes, stream);
    if (e != hipSuccess) {
      (void)hipFree(ptr);
      return fail(SPC_E_HIP, "hipMemsetAsync: %s", hipGetErrorString(e));
    }
    if (w.ptr) w.retired.push_back(w.ptr);
    w.ptr = ptr;
    w.bytes = want;
  }
  *out = static_cast<char*>(w.ptr);
  return SPC_OK;
}

// Static scratch of spc_verify_noalloc: each device that runs it holds its
// own copy until the process ends.  Host code never uses the array's name as
// an address: noalloc_scratch looks up the device address once per device.
constexpr size_t kNoAllocBytes = size_t(32) << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocBytes];

struct NoAllocDev {
  void* ptr = nullptr;  // the device address of `scratch` on this device
  bool cleared = false; // its counter region zeroed by a fill kernel
};
std::mutex g_na_mu;
std::map<int, NoAllocDev> g_na;

// Sequences per launch that the static scratch holds for this row shape
// (0: not even one).
int64_t noalloc_seqs(int64_t gamma, int64_t V, int dtype, bool vec) {
  const size_t one = spc::ws_layout(1, gamma, V, dtype, vec).total;
  if (one > kNoAllocBytes) return 0;
  int64_t lo = 1, hi = spc::kMaxRows;  // largest b with layout(b) <= the scratch
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) / 2;
    if (spc::ws_layout(mid, gamma, V, dtype, vec).total <= kNoAllocBytes) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// The static scratch of device `dev` (the current device).  The first call
// on a device looks up its address and clears its counter region with a
// fill kernel on `stream`; the kernels leave that region zero after every
// call, so later calls find it cleared.  Nothing here allocates.
spc_status noalloc_scratch(int dev, size_t zero_bytes, hipStream_t stream, char** out) {
  std::lock_guard<std::mutex> lk(g_na_mu);
  NoAllocDev& d = g_na[dev];
  if (!d.ptr) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(SPC_E_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    d.ptr = ptr;
  }
  if (!d.cleared) {
    const hipError_t e = spc::launch_fill_zero(d.ptr, zero_bytes, stream);
    if (e != hipSuccess) return fail(SPC_E_HIP, "clearing the scratch: %s", hipGetErrorString(e));
    d.cleared = true;
  }
  *out = static_cast<char*>(d.ptr);
  return SPC_OK;
}

template <class T>
T* offset(T* p, int64_t n) {
  return p ? p + n : p;
}

spc_status verify_impl(const void* q, const void* p, int32_t dtype, const int32_t* draft,
                       const float* uniforms, int32_t B, int32_t gamma, int32_t V, int32_t rule,
                       float alpha, float temperature, bool force_greedy, int32_t* out_accept,
                       int32_t* out_token, uint8_t* out_defer, const spc_verify_ex_args* ex,
                       hipStream_t stream, bool no_alloc = false) {
  g_err.clear();
  if (!q || !p || !draft || !out_accept || !out_token || !out_defer)
    return fail(SPC_E_NULL, "a required pointer is NULL");
  if (!force_greedy && !uniforms) return fail(SPC_E_NULL, "uniforms is NULL");
  spc_status st = check_shape(B, gamma, V);
  if (st != SPC_OK) return st;
  if (dtype != SPC_F32 && dtype != SPC_BF16) return fail(SPC_E_PARAM, "unknown dtype %d", dtype);
  const bool per_rule = ex && ex->rule_per_seq;
  const bool per_alpha = ex && ex->alpha_per_seq;
  const bool per_temp = ex && ex->temp_per_seq;
  if (!per_rule && (rule < SPC_RULE_CHOW || rule > SPC_RULE_OPTLOG))
    return fail(SPC_E_RULE, "unknown rule %d", rule);
  if (!per_alpha && !isfinite(alpha)) return fail(SPC_E_PARAM, "alpha is not finite");
  if (!per_rule && !per_alpha && rule == SPC_RULE_LOSSY && !(alpha < 1.0f))
    return fail(SPC_E_PARAM, "the lossy rule needs alpha < 1 (got %g)", (double)alpha);
  if (!force_greedy && !per_temp && !(isfinite(temperature) && temperature > 0.0f))
    return fail(SPC_E_PARAM, "temperature must be finite and > 0 (got %g)", (double)temperature);
  if (((uintptr_t)q | (uintptr_t)p) % 16 != 0)
    return fail(SPC_E_ALIGN, "logit base pointers must be 16-byte aligned");

  const bool vec = vec_path(dtype, V);
  const int64_t g1 = (int64_t)gamma + 1;
  int64_t b_launch = seqs_per_launch(B, gamma);
  if (no_alloc) {
    if (ex && ex->workspace)
      return fail(SPC_E_WORKSPACE, "spc_verify_noalloc takes no caller workspace");
    // as many sequences per launch as the static scratch holds (the layout
    // grows with the sequences of a launch)
    b_launch = std::min<int64_t>(b_launch, noalloc_seqs(gamma, V, dtype, vec));
    if (b_launch < 1)
      return fail(SPC_E_WORKSPACE,
                  "one sequence of gamma=%d V=%d needs %zu bytes of workspace, more than the "
                  "%zu-byte static scratch of spc_verify_noalloc",
                  gamma, V, spc::ws_layout(1, gamma, V, dtype, vec).total, kNoAllocBytes);
  }
  const spc::WsLayout L = spc::ws_layout(b_launch, gamma, V, dtype, vec);
  // argument checks end here: no HIP call precedes them
  if (ex && ex->workspace &&
      (ex->workspace_bytes < L.total || ((uintptr_t)ex->workspace % 256) != 0))
    return fail(SPC_E_WORKSPACE, "workspace of %zu bytes (need %zu, 256-byte aligned)",
                ex->workspace_bytes, L.total);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SPC_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  const int cus = cu_count(dev);
  if (cus <= 0) return fail(SPC_E_HIP, "cannot read the compute-unit count of device %d", dev);
  char* ws = nullptr;
  if (no_alloc) {
    const spc_status wst = noalloc_scratch(dev, L.zero_end, stream, &ws);
    if (wst != SPC_OK) return wst;
  } else if (ex && ex->workspace) {
    ws = static_cast<char*>(ex->workspace);
  } else {
    const spc_status wst = internal_workspace(L.total, L.zero_end, stream, &ws);
    if (wst != SPC_OK) return wst;
  }

  // The rules the batch may hold decide what each launch computes.
  constexpr uint32_t kAll = (1u << (SPC_RULE_OPTLOG + 1)) - 1u;
  constexpr uint32_t kTv = (1u << SPC_RULE_OPT) | (1u << SPC_RULE_OPTLOG);
  constexpr uint32_t kLog = (1u << SPC_RULE_BILD) | (1u << SPC_RULE_CHOWLOG) |
                            (1u << SPC_RULE_DIFFLOG) | (1u << SPC_RULE_OPTLOG);
  const uint32_t mask = ex ? ex->rules_present & kAll : 0u;
  const uint32_t rules = per_rule ? (mask ? mask : kAll) : (1u << rule);
  const bool may_sample = !force_greedy && (per_temp || temperature > 0.0f);
  // first moments of the log-loss rules (BiLD* at temperature 0 reads one
  // logit instead): x for BiLD*, H(q) for ChowLog, H(q) and H(p) otherwise
  const bool need_mom = (rules & kLog) && !(rules == (1u << SPC_RULE_BILD) && force_greedy);
  const int mom_set = !need_mom ? 0
                                : ((rules & (1u << SPC_RULE_BILD)) ? spc::kMomX : 0) |
                                      ((rules & (1u << SPC_RULE_CHOWLOG)) ? spc::kMomHQ : 0) |
                                      ((rules & ((1u << SPC_RULE_DIFFLOG) | (1u << SPC_RULE_OPTLOG)))
                                           ? spc::kMomHQ | spc::kMomHP
                                           : 0);
  // Rows of OPT / OPTLOG at T > 0 are decided after their TV pass, rows of
  // a token rule after their eta pass (the job pass, for the tiles their
  // statistics leave open), greedy rows after their argmax (the job pass);
  // every other row by its last statistics tile.
  constexpr uint32_t kTok = (1u << SPC_RULE_TOKEN_V1) | (1u << SPC_RULE_TOKEN_V2) |
                            (1u << SPC_RULE_TOKEN_V3);
  const bool may_greedy = force_greedy || per_temp;
  // Every sequence with a draw is drawn by the draw pass, the last kernel of
  // a launch (greedy ones write their token directly).
  const bool draw_pass = may_sample;
  const bool tv_rows = may_sample && (rules & kTv);
  // Small problems (rows that fit one workgroup's registers, at most two
  // rows per compute unit, no first moments) take the single-launch path.
  const bool small = !need_mom && V <= spc::small_row_elems(dtype, vec) &&
                     b_launch * g1 <= 2 * (int64_t)cus;
  const int64_t nt = stat_tiles(dtype, vec, V);
  const int64_t eb = dtype == SPC_BF16 ? 2 : 4;

  for (int64_t b0 = 0; b0 < B; b0 += b_launch) {
    const int64_t bl = std::min<int64_t>(b_launch, B - b0);
    const int64_t R = bl * g1;
    spc::Params P{};
    P.q = static_cast<const char*>(q) + b0 * g1 * V * eb;
    P.p = static_cast<const char*>(p) + b0 * g1 * V * eb;
    P.draft = draft + b0 * gamma;
    P.uniforms = offset(uniforms, b0 * g1);
    P.B = (int32_t)bl;
    P.gamma = gamma;
    P.V = V;
    P.nt = (int32_t)nt;
    P.rule = rule;
    P.alpha = alpha;
    P.temp = force_greedy ? 0.0f : temperature;
    P.force_greedy = force_greedy ? 1 : 0;
    P.rule_mask = per_rule ? mask : 0u;
    P.mom_set = mom_set;
    P.rule_ps = per_rule ? ex->rule_per_seq + b0 : nullptr;
    P.alpha_ps = per_alpha ? ex->alpha_per_seq + b0 : nullptr;
    P.temp_ps = (per_temp && !force_greedy) ? ex->temp_per_seq + b0 : nullptr;
    P.out_accept = out_accept + b0;
    P.out_token = out_token + b0;
    P.out_defer = out_defer + b0 * g1;
    P.out_stats = ex ? offset(ex->out_row_stats, b0 * g1 * 8) : nullptr;
    P.out_argmax = ex ? offset(ex->out_argmax, b0 * g1 * 2) : nullptr;
    P.out_norm = ex ? offset(ex->out_sample_norm, b0) : nullptr;
    // Where TV rows get their TV pass.  In a grid that is resident at once
    // (at most two workgroups per compute unit) each TV row takes it from
    // its own tiles' registers once the row is merged (tv_self).  Otherwise
    // a kernel of its own reads the TV rows again after the statistics
    // kernel (k_tvpass) when the rule is batch-wide, so that most rows may
    // need it; with per-sequence rules (a few TV rows among others) their
    // slices are job-pass items (tv_jobs).
    P.tv_self = (tv_rows && R * nt <= 2 * (int64_t)cus) ? 1 : 0;
    // batches of at least 64 statistics tiles per compute unit stream two
    // tiles per workgroup (without first moments): B = 32 at the Gemma
    // vocabulary (32 per CU) is faster with one, B = 128 and 256 with two
    P.pair = (!P.tv_self && mom_set == 0 && R * nt >= 64 * (int64_t)cus) ? 1 : 0;
    P.tv_jobs = (tv_rows && !P.tv_self && per_rule) ? 1 : 0;
    const bool tv_pass = tv_rows && !P.tv_self && !P.tv_jobs;
    // the job pass: argmax halves, eta slices, TV slices (tv_jobs), and the
    // TV tiles whose wait for their row's merge timed out (tv_self)
    const bool job_pass =
        may_greedy || (may_sample && (rules & kTok)) || P.tv_self || P.tv_jobs;
    P.wait_ticks = tv_wait_ticks();
    // jobs: argmax halves, TV tiles whose wait timed out or TV slices, the
    // slices of the tiles a token row lists for eta (a row has one kind)
    P.single_slots = 2 * R + bl + R * nt * spc::kSlices;
    P.nsub = (int32_t)(nt * spc::tile_subchunks(dtype, vec));
    // workgroups of the job pass: a wavefront per item of its largest
    // expected list (eta slices of every tile, argmax halves), at most two
    // workgroups per compute unit
    const int64_t np = nt * spc::kSlices;
    const int64_t items1 =
        np * (((rules & kTok) || P.tv_jobs) ? R : 0) + (may_greedy ? 2 * R : 0);
    constexpr int64_t kW = spc::kJobThreads / 64;
    const int job_groups = (int)std::max<int64_t>(
        1, std::min<int64_t>((items1 + kW - 1) / kW, 2 * (int64_t)cus));
    P.hdr = reinterpret_cast<uint32_t*>(ws + L.hdr);
    P.rowline = reinterpret_cast<uint32_t*>(ws + L.rowline);
    P.jobs = reinterpret_cast<uint64_t*>(ws + L.jobs);
    P.tiles = reinterpret_cast<spc::TilePart*>(ws + L.tiles);
    P.tvpart = reinterpret_cast<double*>(ws + L.tvpart);
    P.submass = reinterpret_cast<double*>(ws + L.submass);
    P.moms = reinterpret_cast<spc::TileMom*>(ws + L.moms);
    P.rowstat = reinterpret_cast<spc::RowStat*>(ws + L.rowstat);
    P.rowdec = reinterpret_cast<int32_t*>(ws + L.rowdec);
    P.etalist = reinterpret_cast<int32_t*>(ws + L.etalist);
    P.argres = reinterpret_cast<int32_t*>(ws + L.argres);
    P.etacnt = reinterpret_cast<int32_t*>(ws + L.etacnt);
    const bool first = b0 == 0;
    hipEvent_t ev0 = first && ex ? ex->ev_tiles_begin : nullptr;
    hipEvent_t ev1 = first && ex ? ex->ev_tiles_end : nullptr;
    if (small) {
      // one launch: a workgroup per row holding the row in registers
      P.nsub = spc::kSmallSub;
      e = spc::launch_small(P, dtype, vec, ev0, ev1, stream);
    } else {
      e = spc::launch_step(P, dtype, vec, draw_pass, tv_pass, job_pass, job_groups, ev0, ev1,
                           stream);
    }
    if (e != hipSuccess) return fail(SPC_E_HIP, "kernel launch: %s", hipGetErrorString(e));
  }
  return SPC_OK;
}

spc_status draft_impl(const void* logits, int32_t dtype, int32_t B, int32_t V, float temperature,
                      const float* temp_per_seq, const float* uniforms, int32_t* out_token,
                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
  g_err.clear();
  if (!logits || !out_token) return fail(SPC_E_NULL, "a required pointer is NULL");
  if (!temp_per_seq && !(isfinite(temperature) && temperature >= 0.0f))
    return fail(SPC_E_PARAM, "temperature must be finite and >= 0 (got %g)",
                (double)temperature);
  const bool greedy = !temp_per_seq && temperature == 0.0f;
  if (!greedy && !uniforms) return fail(SPC_E_NULL, "uniforms is NULL");
  if (B < 1 || V < 2) return fail(SPC_E_SHAPE, "bad shape B=%d V=%d (need B>=1, V>=2)", B, V);
  if (dtype != SPC_F32 && dtype != SPC_BF16) return fail(SPC_E_PARAM, "unknown dtype %d", dtype);
  if ((uintptr_t)logits % 16 != 0)
    return fail(SPC_E_ALIGN, "logit base pointer must be 16-byte aligned");
  const bool vec = vec_path(dtype, V);
  // rows per launch, as a verify step of gamma = 1 with as many sequences
  const int64_t b_launch = seqs_per_launch(B, 1);
  const spc::WsLayout L = spc::ws_layout(b_launch, 1, V, dtype, vec);
  // argument checks end here: no HIP call precedes them
  if (workspace && (workspace_bytes < L.total || ((uintptr_t)workspace % 256) != 0))
    return fail(SPC_E_WORKSPACE, "workspace of %zu bytes (need %zu, 256-byte aligned)",
                workspace_bytes, L.total);
  char* ws = static_cast<char*>(workspace);
  if (!ws) {
    const spc_status wst = internal_workspace(L.total, L.zero_end, stream, &ws);
    if (wst != SPC_OK) return wst;
  }
  const int64_t eb = dtype == SPC_BF16 ? 2 : 4;
  for (int64_t b0 = 0; b0 < B; b0 += b_launch) {
    const int64_t bl = std::min<int64_t>(b_launch, B - b0);
    spc::Params P{};
    P.q = static_cast<const char*>(logits) + b0 * V * eb;
    P.p = P.q;
    P.uniforms = offset(uniforms, b0);
    P.B = (int32_t)bl;
    P.gamma = 0;
    P.V = V;
    // Tiles twice as long as the statistics tiles once that still gives at
    // least 4 workgroups per CU; small batches take the statistics tile
    // length, for twice the workgroups (either way no more partials per row
    // than the workspace holds for this shape).
    const int64_t long_n = spc::draft_tile_elems(dtype, vec, true);
    const bool long_tiles = bl * ((V + long_n - 1) / long_n) >= 1024;
    const int64_t tile_n = long_tiles ? long_n : spc::draft_tile_elems(dtype, vec, false);
    P.nt = (int32_t)((V + tile_n - 1) / tile_n);
    P.rule = SPC_RULE_NEVER;
    P.temp = greedy ? 0.0f : temperature;
    P.force_greedy = greedy ? 1 : 0;
    P.temp_ps = offset(temp_per_seq, b0);
    P.out_token = out_token + b0;
    P.samp_cnt = reinterpret_cast<uint32_t*>(ws + L.rowline) + spc::kDraftArrive;
    P.tiles = reinterpret_cast<spc::TilePart*>(ws + L.tiles);
    const hipError_t e =
        spc::launch_draft(P, dtype, vec, greedy || temp_per_seq, long_tiles, stream);
    if (e != hipSuccess) return fail(SPC_E_HIP, "kernel launch: %s", hipGetErrorString(e));
  }
  return SPC_OK;
}

}  // namespace

extern "C" {

spc_status spc_verify(const void* q_logits, const void* p_logits, int32_t dtype,
                      const int32_t* draft_tokens, const float* uniforms, int32_t B,
                      int32_t gamma, int32_t V, int32_t rule, float alpha, float temperature,
                      int32_t* out_accept_len, int32_t* out_next_token,
                      uint8_t* out_defer_mask, hipStream_t stream) {
  return verify_impl(q_logits, p_logits, dtype, draft_tokens, uniforms, B, gamma, V, rule, alpha,
                     temperature, false, out_accept_len, out_next_token, out_defer_mask,
                     nullptr, stream);
}

spc_status spc_greedy_verify(const void* q_logits, const void* p_logits, int32_t dtype,
                             const int32_t* draft_tokens, int32_t B, int32_t gamma, int32_t V,
                             int32_t rule, float alpha, int32_t* out_accept_len,
                             int32_t* out_next_token, uint8_t* out_defer_mask,
                             hipStream_t stream) {
  return verify_impl(q_logits, p_logits, dtype, draft_tokens, nullptr, B, gamma, V, rule, alpha,
                     0.0f, true, out_accept_len, out_next_token, out_defer_mask, nullptr, stream);
}

spc_status spc_verify_ex(const void* q_logits, const void* p_logits, int32_t dtype,
                         const int32_t* draft_tokens, const float* uniforms, int32_t B,
                         int32_t gamma, int32_t V, int32_t rule, float alpha, float temperature,
                         int32_t* out_accept_len, int32_t* out_next_token,
                         uint8_t* out_defer_mask, const spc_verify_ex_args* ex,
                         hipStream_t stream) {
  // a scalar temperature of exactly 0 (no per-sequence array) is the
  // batch-wide greedy step of spc_greedy_verify
  const bool greedy = !(ex && ex->temp_per_seq) && temperature == 0.0f;
  return verify_impl(q_logits, p_logits, dtype, draft_tokens, uniforms, B, gamma, V, rule, alpha,
                     temperature, greedy, out_accept_len, out_next_token, out_defer_mask, ex,
                     stream);
}

spc_status spc_verify_noalloc(const void* q_logits, const void* p_logits, int32_t dtype,
                              const int32_t* draft_tokens, const float* uniforms, int32_t B,
                              int32_t gamma, int32_t V, int32_t rule, float alpha,
                              float temperature, int32_t* out_accept_len,
                              int32_t* out_next_token, uint8_t* out_defer_mask,
                              const spc_verify_ex_args* ex, hipStream_t stream) {
  const bool greedy = !(ex && ex->temp_per_seq) && temperature == 0.0f;
  return verify_impl(q_logits, p_logits, dtype, draft_tokens, uniforms, B, gamma, V, rule, alpha,
                     temperature, greedy, out_accept_len, out_next_token, out_defer_mask, ex,
                     stream, true);
}

size_t spc_noalloc_scratch_bytes(void) { return kNoAllocBytes; }

spc_status spc_draft_sample(const void* logits, int32_t dtype, int32_t B, int32_t V,
                            float temperature, const float* temp_per_seq,
                            const float* uniforms, int32_t* out_token, hipStream_t stream) {
  return draft_impl(logits, dtype, B, V, temperature, temp_per_seq, uniforms, out_token, nullptr,
                    0, stream);
}

spc_status spc_draft_sample_ws(const void* logits, int32_t dtype, int32_t B, int32_t V,
                               float temperature, const float* temp_per_seq,
                               const float* uniforms, int32_t* out_token, void* workspace,
                               size_t workspace_bytes, hipStream_t stream) {
  return draft_impl(logits, dtype, B, V, temperature, temp_per_seq, uniforms, out_token,
                    workspace, workspace_bytes, stream);
}

size_t spc_workspace_bytes(int32_t B, int32_t gamma, int32_t V, int32_t dtype) {
  if (check_shape(B, gamma, V) != SPC_OK || (dtype != SPC_F32 && dtype != SPC_BF16)) return 0;
  return launch_layout(B, gamma, V, dtype).total;
}

size_t spc_workspace_zero_bytes(int32_t B, int32_t gamma, int32_t V, int32_t dtype) {
  if (check_shape(B, gamma, V) != SPC_OK || (dtype != SPC_F32 && dtype != SPC_BF16)) return 0;
  return launch_layout(B, gamma, V, dtype).zero_end;
}

size_t spc_draft_workspace_bytes(int32_t B, int32_t V, int32_t dtype) {
  if (B < 1 || V < 2 || (dtype != SPC_F32 && dtype != SPC_BF16)) return 0;
  return spc::ws_layout(seqs_per_launch(B, 1), 1, V, dtype, vec_path(dtype, V)).total;
}

const char* spc_last_error(void) { return g_err.c_str(); }

void spc_release(void) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  int cur = 0;
  if (hipGetDevice(&cur) != hipSuccess) cur = 0;
  for (auto& kv : g_ws) {
    if (hipSetDevice(kv.first) != hipSuccess) continue;
    if (kv.second.ptr) (void)hipFree(kv.second.ptr);
    for (void* r : kv.second.retired) (void)hipFree(r);
  }
  g_ws.clear();
  (void)hipSetDevice(cur);
}

const char* spc_version(void) { return "libspeccascade 0.2 (gfx950)"; }

}  // extern "C"
