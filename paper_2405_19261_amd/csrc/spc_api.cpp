// spc_api.cpp -- the C interface of libspeccascade (declared in
// include/speccascade.h): argument checks, workspace, kernel dispatch.
#include <math.h>
#include <stdlib.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <string>

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

struct DevWorkspace {
  void* ptr = nullptr;
  size_t bytes = 0;
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

// Rows (gridDim.y of the statistics kernels) are capped by the launch limit.
constexpr int64_t kMaxRows = 65535;

// SPC_ONE_READ=1 in the environment selects the one-read statistics kernel
// for batches it can take (read on every call).  It is off by default: on
// MI355X it is slower than reading the second-pass rows again.
bool one_read_requested() {
  const char* v = getenv("SPC_ONE_READ");
  return v && v[0] && v[0] != '0';
}

bool vec_path(int dtype, int64_t V) {
  const int64_t eb = dtype == SPC_BF16 ? 2 : 4;
  return (V * eb) % 16 == 0;  // every row starts on a 16-byte boundary
}

}  // namespace

namespace spc {

WsLayout ws_layout(int64_t B, int64_t gamma, int64_t V, int dtype, bool vec) {
  // The completion counters sit at a fixed offset sized for the largest batch
  // the interface accepts, so a workspace reused across shapes never has one
  // call's data overlap another call's counters; they stay zero between calls.
  const int64_t R = B * (gamma + 1);
  const int64_t nt = (V + stat_tile_elems(dtype, vec) - 1) / stat_tile_elems(dtype, vec);
  WsLayout L;
  L.samp_cnt = 0;
  size_t o = align_up(4 * (size_t)(kMaxRows + 1), 256);
  // the drafter kernel's per-row counters, one per 128-byte line
  L.draft_cnt = o;
  o = align_up(o + 4 * (size_t)kDraftCntStride * (kMaxRows / 2 + 1), 256);
  // the one-read statistics kernel's per-row counters, one per 128-byte line
  L.row_cnt = o;
  o = align_up(o + 4 * (size_t)kRowCntStride * kResRows, 256);
  L.zero_end = o;
  L.tiles = o; o = align_up(o + sizeof(TilePart) * R * nt, 256);
  L.tvpart = o; o = align_up(o + sizeof(double) * R * nt, 256);
  const int64_t nc = (V + samp_chunk_elems(dtype, vec) - 1) / samp_chunk_elems(dtype, vec);
  L.masses = o; o = align_up(o + sizeof(double) * B * nc, 256);
  L.moms = o; o = align_up(o + sizeof(TileMom) * R * nt, 256);
  L.total = o;
  return L;
}

}  // namespace spc

namespace {

spc_status check_shape(int32_t B, int32_t gamma, int32_t V) {
  if (B < 1 || gamma < 1 || gamma > SPC_MAX_GAMMA || V < 2)
    return fail(SPC_E_SHAPE, "bad shape B=%d gamma=%d V=%d (need B>=1, 1<=gamma<=%d, V>=2)", B,
                gamma, V, SPC_MAX_GAMMA);
  const int64_t R = (int64_t)B * (gamma + 1);
  if (R > kMaxRows)
    return fail(SPC_E_SHAPE, "B*(gamma+1)=%lld exceeds %lld rows", (long long)R,
                (long long)kMaxRows);
  return SPC_OK;
}

// The internal workspace of the current device, grown to L.total if needed
// (its counters zeroed on `stream` before any kernel that uses them).
spc_status internal_workspace(const spc::WsLayout& L, hipStream_t stream, char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SPC_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(g_ws_mu);
  DevWorkspace& w = g_ws[dev];
  if (w.bytes < L.total) {
    // growing: the old buffer may still be in use by work on `stream`
    if (w.ptr) {
      e = hipStreamSynchronize(stream);
      if (e == hipSuccess) e = hipFree(w.ptr);
      w.ptr = nullptr;
      w.bytes = 0;
      if (e != hipSuccess) return fail(SPC_E_HIP, "workspace release: %s", hipGetErrorString(e));
    }
    const size_t want = L.total + L.total / 4;  // headroom for nearby shapes
    e = hipMalloc(&w.ptr, want);
    if (e != hipSuccess) {
      w.ptr = nullptr;
      return fail(SPC_E_HIP, "hipMalloc(%zu): %s", want, hipGetErrorString(e));
    }
    // zero counters, ordered before this call's kernels on the same stream;
    // the kernels leave them zero
    e = hipMemsetAsync(w.ptr, 0, L.zero_end, stream);
    if (e != hipSuccess) {
      (void)hipFree(w.ptr);
      w.ptr = nullptr;
      return fail(SPC_E_HIP, "hipMemsetAsync: %s", hipGetErrorString(e));
    }
    w.bytes = want;
  }
  *out = static_cast<char*>(w.ptr);
  return SPC_OK;
}

spc_status verify_impl(const void* q, const void* p, int32_t dtype, const int32_t* draft,
                       const float* uniforms, int32_t B, int32_t gamma, int32_t V, int32_t rule,
                       float alpha, float temperature, bool force_greedy, int32_t* out_accept,
                       int32_t* out_token, uint8_t* out_defer, const spc_verify_ex_args* ex,
                       hipStream_t stream) {
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
  if (!force_greedy && !per_temp && !(isfinite(temperature) && temperature >= 1e-20f))
    return fail(SPC_E_PARAM, "temperature must be finite and >= 1e-20 (got %g)",
                (double)temperature);
  if (((uintptr_t)q | (uintptr_t)p) % 16 != 0)
    return fail(SPC_E_ALIGN, "logit base pointers must be 16-byte aligned");

  const bool vec = vec_path(dtype, V);
  const spc::WsLayout L = spc::ws_layout(B, gamma, V, dtype, vec);
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
  if (ex && ex->workspace) {
    ws = static_cast<char*>(ex->workspace);
  } else {
    const spc_status wst = internal_workspace(L, stream, &ws);
    if (wst != SPC_OK) return wst;
  }

  spc::Params P{};
  P.q = q;
  P.p = p;
  P.draft = draft;
  P.uniforms = uniforms;
  P.B = B;
  P.gamma = gamma;
  P.V = V;
  P.nt = (int32_t)((V + spc::stat_tile_elems(dtype, vec) - 1) / spc::stat_tile_elems(dtype, vec));
  P.nc = (int32_t)((V + spc::samp_chunk_elems(dtype, vec) - 1) / spc::samp_chunk_elems(dtype, vec));
  P.K = spc::samp_groups(P.nc, B, cus);
  P.rule = rule;
  P.alpha = alpha;
  P.temp = force_greedy ? 0.0f : temperature;
  P.force_greedy = force_greedy ? 1 : 0;
  P.rule_ps = per_rule ? ex->rule_per_seq : nullptr;
  P.alpha_ps = per_alpha ? ex->alpha_per_seq : nullptr;
  P.temp_ps = (per_temp && !force_greedy) ? ex->temp_per_seq : nullptr;
  P.out_accept = out_accept;
  P.out_token = out_token;
  P.out_defer = out_defer;
  P.out_stats = ex ? ex->out_row_stats : nullptr;
  P.out_argmax = ex ? ex->out_argmax : nullptr;
  P.out_norm = ex ? ex->out_sample_norm : nullptr;
  P.samp_cnt = reinterpret_cast<uint32_t*>(ws + L.samp_cnt);
  P.row_cnt = reinterpret_cast<uint32_t*>(ws + L.row_cnt);
  P.tiles = reinterpret_cast<spc::TilePart*>(ws + L.tiles);
  P.tvpart = reinterpret_cast<double*>(ws + L.tvpart);
  P.masses = reinterpret_cast<double*>(ws + L.masses);
  P.moms = reinterpret_cast<spc::TileMom*>(ws + L.moms);

  // sequences at temperature > 0 may exist unless the whole batch is greedy;
  // OPT at temperature > 0 needs the TV pass
  const bool need_sample = !force_greedy && (per_temp || temperature > 0.0f);
  // The rules the batch may hold decide the passes.  OPT, OPTLOG (D_TV) and
  // the token rules (eta) need the second pass over their rows at
  // temperature > 0; rows that need first moments (log-loss rules, BiLD* at
  // temperature > 0) and rows that do not each get their statistics kernel.
  constexpr uint32_t kAll = (1u << (SPC_RULE_OPTLOG + 1)) - 1u;
  constexpr uint32_t kTv = (1u << SPC_RULE_OPT) | (1u << SPC_RULE_OPTLOG) |
                           (1u << SPC_RULE_TOKEN_V1) | (1u << SPC_RULE_TOKEN_V2) |
                           (1u << SPC_RULE_TOKEN_V3);
  constexpr uint32_t kLog = (1u << SPC_RULE_BILD) | (1u << SPC_RULE_CHOWLOG) |
                            (1u << SPC_RULE_DIFFLOG) | (1u << SPC_RULE_OPTLOG);
  const uint32_t mask = ex ? ex->rules_present & kAll : 0u;
  const uint32_t rules = per_rule ? (mask ? mask : kAll) : (1u << rule);
  P.rule_mask = per_rule ? mask : 0u;
  constexpr uint32_t kEta = (1u << SPC_RULE_TOKEN_V1) | (1u << SPC_RULE_TOKEN_V2) |
                            (1u << SPC_RULE_TOKEN_V3);
  const int tv_kinds = !need_sample ? 0
                                    : ((rules & (kTv & ~kEta)) ? spc::kPassTv : 0) |
                                          ((rules & kEta) ? spc::kPassEta : 0);
  const bool need_argmax = force_greedy || per_temp;
  // BiLD* at temperature 0 reads one logit instead of moments
  const bool bild_t0 = (rules & (1u << SPC_RULE_BILD)) && (force_greedy || per_temp);
  const bool need_mom = (rules & kLog) && !(rules == (1u << SPC_RULE_BILD) && force_greedy);
  const bool need_plain = (rules & ~kLog) || per_temp || bild_t0;
  P.mom_split = (need_mom && need_plain) ? 1 : 0;
  // moments by rule: BiLD* reads x, ChowLog H(q), DiffLog and OPTLog H(q) - H(p)
  P.mom_set = ((rules & (1u << SPC_RULE_BILD)) ? spc::kMomX : 0) |
              ((rules & (1u << SPC_RULE_CHOWLOG)) ? spc::kMomHQ : 0) |
              ((rules & ((1u << SPC_RULE_DIFFLOG) | (1u << SPC_RULE_OPTLOG)))
                   ? spc::kMomHQ | spc::kMomHP
                   : 0);
  // The second pass reads its rows again, unless the one-read kernel is
  // requested and fits: a resident grid holding at least one whole row of
  // tiles per round.
  int res_grid = 0;
  const int64_t R = (int64_t)B * (gamma + 1);
  if (tv_kinds && !need_mom && R <= spc::kResRows && one_read_requested()) {
    const int nb = spc::res_blocks_per_cu(dtype, vec, need_argmax);
    const int64_t rows_per_round = (int64_t)nb * cus / P.nt;
    if (rows_per_round >= 1) res_grid = (int)(std::min<int64_t>(rows_per_round, R) * P.nt);
  }
  e = spc::launch_verify(P, dtype, vec, tv_kinds, need_sample, need_argmax, need_plain, need_mom,
                         res_grid, ex ? ex->ev_hot_begin : nullptr,
                         ex ? ex->ev_hot_end : nullptr, stream);
  if (e != hipSuccess) return fail(SPC_E_HIP, "kernel launch: %s", hipGetErrorString(e));
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

spc_status spc_draft_sample(const void* logits, int32_t dtype, int32_t B, int32_t V,
                            float temperature, const float* temp_per_seq,
                            const float* uniforms, int32_t* out_token, hipStream_t stream) {
  g_err.clear();
  if (!logits || !out_token) return fail(SPC_E_NULL, "a required pointer is NULL");
  if (!temp_per_seq && !(isfinite(temperature) && temperature >= 0.0f))
    return fail(SPC_E_PARAM, "temperature must be finite and >= 0 (got %g)",
                (double)temperature);
  const bool greedy = !temp_per_seq && temperature == 0.0f;
  if (!greedy && !uniforms) return fail(SPC_E_NULL, "uniforms is NULL");
  if (B < 1 || V < 2 || (int64_t)B > kMaxRows / 2)
    return fail(SPC_E_SHAPE, "bad shape B=%d V=%d (need 1<=B<=%lld, V>=2)", B, V,
                (long long)(kMaxRows / 2));
  if (dtype != SPC_F32 && dtype != SPC_BF16) return fail(SPC_E_PARAM, "unknown dtype %d", dtype);
  if ((uintptr_t)logits % 16 != 0)
    return fail(SPC_E_ALIGN, "logit base pointer must be 16-byte aligned");
  const bool vec = vec_path(dtype, V);
  const spc::WsLayout L = spc::ws_layout(B, 0, V, dtype, vec);
  // argument checks end here: no HIP call precedes them
  char* ws = nullptr;
  const spc_status wst = internal_workspace(L, stream, &ws);
  if (wst != SPC_OK) return wst;
  spc::Params P{};
  P.q = logits;
  P.p = logits;
  P.uniforms = uniforms;
  P.B = B;
  P.gamma = 0;
  P.V = V;
  // Tiles twice as long as the statistics tiles once that still gives at
  // least 4 workgroups per CU; small batches take the statistics tile
  // length, for twice the workgroups (either way no more partials per row
  // than the workspace holds for this shape).
  const int64_t long_n = spc::draft_tile_elems(dtype, vec, true);
  const bool long_tiles = (int64_t)B * ((V + long_n - 1) / long_n) >= 1024;
  const int64_t tile_n = long_tiles ? long_n : spc::draft_tile_elems(dtype, vec, false);
  P.nt = (int32_t)((V + tile_n - 1) / tile_n);
  P.rule = SPC_RULE_NEVER;
  P.temp = greedy ? 0.0f : temperature;
  P.force_greedy = greedy ? 1 : 0;
  P.temp_ps = temp_per_seq;
  P.out_token = out_token;
  P.samp_cnt = reinterpret_cast<uint32_t*>(ws + L.draft_cnt);
  P.tiles = reinterpret_cast<spc::TilePart*>(ws + L.tiles);
  const hipError_t e =
      spc::launch_draft(P, dtype, vec, greedy || temp_per_seq, long_tiles, stream);
  if (e != hipSuccess) return fail(SPC_E_HIP, "kernel launch: %s", hipGetErrorString(e));
  return SPC_OK;
}

size_t spc_workspace_bytes(int32_t B, int32_t gamma, int32_t V, int32_t dtype) {
  if (check_shape(B, gamma, V) != SPC_OK || (dtype != SPC_F32 && dtype != SPC_BF16)) return 0;
  return spc::ws_layout(B, gamma, V, dtype, vec_path(dtype, V)).total;
}

size_t spc_workspace_zero_bytes(int32_t B, int32_t gamma, int32_t V, int32_t dtype) {
  if (check_shape(B, gamma, V) != SPC_OK || (dtype != SPC_F32 && dtype != SPC_BF16)) return 0;
  return spc::ws_layout(B, gamma, V, dtype, vec_path(dtype, V)).zero_end;
}

const char* spc_last_error(void) { return g_err.c_str(); }

void spc_release(void) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  int cur = 0;
  if (hipGetDevice(&cur) != hipSuccess) cur = 0;
  for (auto& kv : g_ws) {
    if (kv.second.ptr && hipSetDevice(kv.first) == hipSuccess) (void)hipFree(kv.second.ptr);
  }
  g_ws.clear();
  (void)hipSetDevice(cur);
}

const char* spc_version(void) { return "libspeccascade 0.1 (gfx950)"; }

}  // extern "C"
