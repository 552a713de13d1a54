// C ABI entry points: argument validation, lane-tree preprocessing and
// launches on the caller's stream.  Every check runs before anything is
// enqueued; nothing here allocates, prints or throws.
#include <math.h>
#include <stdint.h>

#include "../../include/asynclane.h"
#include "launch.h"

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

int hip_status(hipError_t e) { return e == hipSuccess ? AL_OK : AL_ERR_HIP; }

// Ancestor-or-self sets of the lane tree: bit j of vis[i] is set when lane j
// is lane i or one of its ancestors (parent[i] < i, so one forward pass).
int lane_visibility(const int32_t* parent, int L, unsigned long long* vis) {
  for (int i = 0; i < L; ++i) {
    const int pi = parent[i];
    if (pi < -1 || pi >= i) return AL_ERR_TREE;
    vis[i] = (1ull << i) | (pi >= 0 ? vis[pi] : 0ull);
  }
  return AL_OK;
}

}  // namespace

extern "C" {

const char* al_status_string(int status) {
  switch (status) {
    case AL_OK: return "ok";
    case AL_ERR_NULL: return "required pointer is null";
    case AL_ERR_SHAPE: return "size or scalar out of the supported range";
    case AL_ERR_TREE: return "lane tree invalid: parent[i] must be in [-1, i)";
    case AL_ERR_WORKSPACE: return "workspace too small";
    case AL_ERR_ALIGN: return "device pointer not 16-byte aligned";
    case AL_ERR_UNSUPPORTED: return "unsupported configuration";
    case AL_ERR_HIP: return "HIP launch error";
    default: return "unknown status";
  }
}

static bool attn_shape_ok(int L, int B, int P, int Hq, int Hkv, int D, int n_refresh) {
  // L = 0 is a refresh-only call (compact cache refresh).
  if (L < 0 || L > AL_MAX_LANES || (L == 0 && n_refresh == 0)) return false;
  if (L > 0 && (B < 16 || B > 1024 || B % 16 != 0)) return false;
  if (P < 0 || n_refresh < 0 || n_refresh > P) return false;
  if (Hkv < 1 || Hq < Hkv || Hq % Hkv != 0 || Hq / Hkv > 16) return false;
  if (D != 64 && D != 128) return false;
  if ((long long)L * B * Hq * D >= (1ll << 31) || (long long)P * Hkv * D >= (1ll << 31)) return false;
  return true;
}

size_t lane_attn_workspace_size(int L, int B, int P, int Hq, int Hkv, int D, int n_refresh) {
  if (!attn_shape_ok(L, B, P, Hq, Hkv, D, n_refresh)) return 0;
  return al::attn_plan(L, B, P, Hq, Hkv, D, n_refresh).total;
}

int lane_attn_forward(const al_bf16* q, const al_bf16* k_lane, const al_bf16* v_lane,
                      al_bf16* k_prefix, al_bf16* v_prefix, const int32_t* parent, int L, int B,
                      int P, int Hq, int Hkv, int D, float scale, const int32_t* refresh_idx,
                      int n_refresh, const al_bf16* q_ref, const al_bf16* k_ref,
                      const al_bf16* v_ref, al_bf16* o_ref, float* lse_ref, al_bf16* o, float* lse,
                      void* workspace, size_t workspace_bytes, void* stream) {
  if (L > 0 && (!q || !k_lane || !v_lane || !parent || !o)) return AL_ERR_NULL;
  if (P > 0 && (!k_prefix || !v_prefix)) return AL_ERR_NULL;
  if (n_refresh > 0 && (!refresh_idx || !q_ref || !k_ref || !v_ref || !o_ref)) return AL_ERR_NULL;
  if (!attn_shape_ok(L, B, P, Hq, Hkv, D, n_refresh)) return AL_ERR_SHAPE;
  if (isnan(scale) || isinf(scale)) return AL_ERR_SHAPE;
  if ((L > 0 && (!aligned16(q) || !aligned16(k_lane) || !aligned16(v_lane) || !aligned16(o) ||
                 (lse && !aligned4(lse)))) ||
      (P > 0 && (!aligned16(k_prefix) || !aligned16(v_prefix))))
    return AL_ERR_ALIGN;
  if (n_refresh > 0 && (!aligned16(q_ref) || !aligned16(k_ref) || !aligned16(v_ref) ||
                        !aligned16(o_ref) || !aligned4(refresh_idx) || (lse_ref && !aligned4(lse_ref))))
    return AL_ERR_ALIGN;
  unsigned long long vis[AL_MAX_LANES];
  const int tree = lane_visibility(parent, L, vis);
  if (tree != AL_OK) return tree;
  const al::AttnPlan plan = al::attn_plan(L, B, P, Hq, Hkv, D, n_refresh);
  if (plan.total > 0) {
    if (!workspace) return AL_ERR_NULL;
    if (workspace_bytes < plan.total) return AL_ERR_WORKSPACE;
    if (!aligned16(workspace)) return AL_ERR_ALIGN;
  }
  const float sc = scale > 0.f ? scale : 1.0f / sqrtf((float)D);
  return hip_status(al::launch_lane_attention(
      q, k_lane, v_lane, k_prefix, v_prefix, vis, L, B, P, Hq, Hkv, D, sc, refresh_idx, n_refresh,
      q_ref, k_ref, v_ref, o_ref, lse_ref, o, lse, workspace, static_cast<hipStream_t>(stream)));
}

static bool lm_shape_ok(int N, int d, int V) {
  return N >= 0 && d >= 8 && d <= 65536 && d % 8 == 0 && V >= 1 && V <= (1 << 30);
}

size_t lmhead_confidence_workspace_size(int N, int d, int V) {
  if (!lm_shape_ok(N, d, V)) return 0;
  return al::lmhead_workspace_bytes(N, d, V);
}

// Checks shared by lmhead_confidence and lmhead_confidence_noalloc.  Returns
// AL_OK with *skip = true for N == 0 (nothing to enqueue).
static int lmhead_check(const al_bf16* hidden, int n_rows, const int32_t* row_idx, int N,
                        const al_bf16* W, int d, int V, const uint8_t* suppress_eos, int eos_id,
                        float* conf, int32_t* argmax, float* lse, bool* skip) {
  *skip = false;
  if (!lm_shape_ok(N, d, V) || n_rows < 0 || N > n_rows) return AL_ERR_SHAPE;
  if ((long long)n_rows * d >= (1ll << 31)) return AL_ERR_SHAPE;  // 32-bit row offsets
  if (eos_id < -1 || eos_id >= V) return AL_ERR_SHAPE;
  // A suppressed row of a one-token vocabulary whose only id is EOS would
  // have no candidate token at all.
  if (V == 1 && eos_id == 0 && suppress_eos) return AL_ERR_SHAPE;
  if (N == 0) {
    *skip = true;
    return AL_OK;
  }
  if (!hidden || !W || !conf || !argmax) return AL_ERR_NULL;
  if (!aligned16(hidden) || !aligned16(W) || !aligned4(conf) || !aligned4(argmax) ||
      (row_idx && !aligned4(row_idx)) || (lse && !aligned4(lse)))
    return AL_ERR_ALIGN;
  return AL_OK;
}

int lmhead_confidence(const al_bf16* hidden, int n_rows, const int32_t* row_idx, int N,
                      const al_bf16* W, int d, int V, const uint8_t* suppress_eos, int eos_id,
                      float* conf, int32_t* argmax, float* lse, void* workspace,
                      size_t workspace_bytes, void* stream) {
  bool skip = false;
  const int st = lmhead_check(hidden, n_rows, row_idx, N, W, d, V, suppress_eos, eos_id, conf,
                              argmax, lse, &skip);
  if (st != AL_OK || skip) return st;
  const size_t need = al::lmhead_workspace_bytes(N, d, V);
  if (!workspace) return AL_ERR_NULL;
  if (workspace_bytes < need) return AL_ERR_WORKSPACE;
  if (!aligned16(workspace)) return AL_ERR_ALIGN;
  return hip_status(al::launch_lmhead(hidden, row_idx, N, W, d, V, suppress_eos, eos_id, conf,
                                      argmax, lse, workspace, static_cast<hipStream_t>(stream)));
}

size_t lmhead_packed_weight_size(int d, int V) {
  if (!lm_shape_ok(1, d, V)) return 0;
  return al::lmhead_packed_bytes(d, V);
}

int lmhead_pack_weight(const al_bf16* W, int d, int V, al_bf16* W_packed, size_t packed_bytes,
                       void* stream) {
  if (!lm_shape_ok(1, d, V)) return AL_ERR_SHAPE;
  if (!W || !W_packed) return AL_ERR_NULL;
  if (!aligned16(W) || !aligned16(W_packed)) return AL_ERR_ALIGN;
  if (packed_bytes < al::lmhead_packed_bytes(d, V)) return AL_ERR_WORKSPACE;
  return hip_status(al::launch_lmhead_pack(W, d, V, W_packed, static_cast<hipStream_t>(stream)));
}

int lmhead_confidence_packed(const al_bf16* hidden, int n_rows, const int32_t* row_idx, int N,
                             const al_bf16* W_packed, int d, int V, const uint8_t* suppress_eos,
                             int eos_id, float* conf, int32_t* argmax, float* lse,
                             void* workspace, size_t workspace_bytes, void* stream) {
  bool skip = false;
  const int st = lmhead_check(hidden, n_rows, row_idx, N, W_packed, d, V, suppress_eos, eos_id,
                              conf, argmax, lse, &skip);
  if (st != AL_OK || skip) return st;
  const size_t need = al::lmhead_workspace_bytes(N, d, V);
  if (!workspace) return AL_ERR_NULL;
  if (workspace_bytes < need) return AL_ERR_WORKSPACE;
  if (!aligned16(workspace)) return AL_ERR_ALIGN;
  return hip_status(al::launch_lmhead(hidden, row_idx, N, W_packed, d, V, suppress_eos, eos_id,
                                      conf, argmax, lse, workspace,
                                      static_cast<hipStream_t>(stream), true));
}

int lmhead_confidence_noalloc(const al_bf16* hidden, int n_rows, const int32_t* row_idx, int N,
                              const al_bf16* W, int d, int V, const uint8_t* suppress_eos,
                              int eos_id, float* conf, int32_t* argmax, float* lse,
                              void* stream) {
  bool skip = false;
  const int st = lmhead_check(hidden, n_rows, row_idx, N, W, d, V, suppress_eos, eos_id, conf,
                              argmax, lse, &skip);
  if (st != AL_OK || skip) return st;
  if (al::lmhead_workspace_bytes(N, d, V) > al::lmhead_scratch_bytes()) return AL_ERR_WORKSPACE;
  void* scratch_dev = nullptr;  // device address of the library's partials array
  if (al::lmhead_scratch(&scratch_dev) != hipSuccess) return AL_ERR_HIP;
  return hip_status(al::launch_lmhead(hidden, row_idx, N, W, d, V, suppress_eos, eos_id, conf,
                                      argmax, lse, scratch_dev, static_cast<hipStream_t>(stream)));
}

int select_unmask(const float* conf, const int32_t* argmax, const int32_t* row_pos, int N,
                  int32_t* tokens, uint8_t* is_masked, int L, int B, const uint8_t* role,
                  const int32_t* b_len, const int32_t* t_lane, int mode, float tau, int fallback_k,
                  const int32_t* k_lane, const int32_t* delim_ids, int n_delim,
                  const int32_t* digit_ids, int n_digit, const int32_t* open_ids, int n_open,
                  const int32_t* close_ids, int n_close, int eos_id,
                  float rho_min, int t_min, float tau_future, uint8_t* unmask_flag,
                  int32_t* unmasked_pos,
                  int32_t* still_masked_pos, int32_t* counts, int32_t* lane_stats,
                  uint8_t* delim_flag, void* stream) {
  if (L < 1 || L > AL_MAX_LANES || B < 1 || (long long)L * B > al::kSelMaxPositions)
    return AL_ERR_SHAPE;
  if (N < 0 || N > L * B) return AL_ERR_SHAPE;
  if (mode != AL_MODE_THRESHOLD && mode != AL_MODE_TOPK) return AL_ERR_SHAPE;
  if (isnan(tau) || isnan(rho_min) || isnan(tau_future) || fallback_k < 0 || n_delim < 0 || n_delim > AL_MAX_DELIMS)
    return AL_ERR_SHAPE;
  if (!tokens || !is_masked || !role || !counts || !lane_stats) return AL_ERR_NULL;
  if (n_delim > 0 && !delim_ids) return AL_ERR_NULL;
  if (n_digit < 0 || n_digit > AL_MAX_BOUNDARY_IDS || n_open < 0 || n_open > AL_MAX_BOUNDARY_IDS ||
      n_close < 0 || n_close > AL_MAX_BOUNDARY_IDS)
    return AL_ERR_SHAPE;
  if ((n_digit > 0 && !digit_ids) || (n_open > 0 && !open_ids) || (n_close > 0 && !close_ids))
    return AL_ERR_NULL;
  if (mode == AL_MODE_TOPK && !k_lane) return AL_ERR_NULL;
  if (N > 0 && (!conf || !argmax || !row_pos || !unmask_flag || !unmasked_pos || !still_masked_pos))
    return AL_ERR_NULL;
  if (!aligned4(tokens) || !aligned4(counts) || !aligned4(lane_stats) ||
      (N > 0 && (!aligned4(conf) || !aligned4(argmax) || !aligned4(row_pos) ||
                 !aligned4(unmasked_pos) || !aligned4(still_masked_pos))))
    return AL_ERR_ALIGN;
  al::SelHost h{};
  h.L = L;
  h.B = B;
  h.N = N;
  h.mode = mode;
  h.tau = tau;
  h.tau_future = tau_future;
  h.fallback_k = fallback_k;
  h.eos_id = eos_id;
  h.rho_min = rho_min;
  h.t_min = t_min;
  h.n_delim = n_delim;
  for (int j = 0; j < n_delim; ++j) h.delim[j] = delim_ids[j];
  h.n_digit = n_digit;
  h.n_open = n_open;
  h.n_close = n_close;
  for (int j = 0; j < n_digit; ++j) h.digit[j] = digit_ids[j];
  for (int j = 0; j < n_open; ++j) h.open[j] = open_ids[j];
  for (int j = 0; j < n_close; ++j) h.close[j] = close_ids[j];
  for (int i = 0; i < L; ++i) {
    if (role[i] != AL_ROLE_GEN && role[i] != AL_ROLE_REF) return AL_ERR_SHAPE;
    h.role[i] = role[i];
    h.b_len[i] = b_len ? b_len[i] : B;
    if (h.b_len[i] < 0 || h.b_len[i] > B) return AL_ERR_SHAPE;
    h.t_lane[i] = t_lane ? t_lane[i] : 0;
    h.k_lane[i] = (mode == AL_MODE_TOPK) ? k_lane[i] : 0;
    if (h.k_lane[i] < 0) return AL_ERR_SHAPE;
  }
  return hip_status(al::launch_select(h, conf, argmax, row_pos, tokens, is_masked, unmask_flag,
                                      unmasked_pos, still_masked_pos, counts, lane_stats,
                                      delim_flag, static_cast<hipStream_t>(stream)));
}

int al_refresh_window(int P, int L_gen, const int32_t* lane_start, const int32_t* valid_len,
                      int n_lanes, int margin) {
  if (P < 0 || L_gen < 0 || n_lanes < 0 || margin < 0) return AL_ERR_SHAPE;
  if (n_lanes > 0 && (!lane_start || !valid_len)) return AL_ERR_NULL;
  long long l_eff = 0;
  for (int i = 0; i < n_lanes; ++i) {
    if (lane_start[i] < 0 || valid_len[i] < 0) return AL_ERR_SHAPE;
    const long long f = (long long)lane_start[i] + valid_len[i];
    if (f > l_eff) l_eff = f;
  }
  const long long full = (long long)P + L_gen;
  const long long win = (long long)P + l_eff + margin;
  const long long r = win < full ? win : full;
  return r > INT32_MAX ? AL_ERR_SHAPE : (int)r;
}

}  // extern "C"
