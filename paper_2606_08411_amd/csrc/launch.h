// Internal launchers behind the C ABI (argument validation happens in abi.cpp).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace al {

// ---- lane attention
struct AttnPlan {
  bool wsplit_lane, wsplit_ref;  // keys split over the wavefronts of a workgroup
  int n_split_lane, n_split_ref;  // else: key splits over workgroups
  size_t ws_lane, ws_ref, total;
};
AttnPlan attn_plan(int L, int B, int P, int Hq, int Hkv, int D, int n_refresh);

hipError_t launch_lane_attention(const uint16_t* q, const uint16_t* k_lane, const uint16_t* v_lane,
                                 uint16_t* k_pre, uint16_t* v_pre, const unsigned long long* vis,
                                 int L, int B, int P, int Hq, int Hkv, int D, float scale,
                                 const int32_t* refresh_idx, int n_refresh, const uint16_t* q_ref,
                                 const uint16_t* k_ref, const uint16_t* v_ref, uint16_t* o_ref,
                                 float* lse_ref, uint16_t* o, float* lse, void* ws,
                                 hipStream_t stream);

// ---- LM head
size_t lmhead_workspace_bytes(int N, int d, int V);
// Device address (current device) of the fixed partials array used by
// lmhead_confidence_noalloc; looked up once per device.
hipError_t lmhead_scratch(void** out);
size_t lmhead_scratch_bytes();
// packed: W is in the layout lmhead_pack_weight writes.
hipError_t launch_lmhead(const uint16_t* hidden, const int32_t* row_idx, int N, const uint16_t* W,
                         int d, int V, const uint8_t* sup, int eos_id, float* conf,
                         int32_t* argmax, float* lse, void* ws, hipStream_t stream,
                         bool packed = false);
size_t lmhead_packed_bytes(int d, int V);
hipError_t launch_lmhead_pack(const uint16_t* W, int d, int V, uint16_t* Wp, hipStream_t stream);

// ---- selection
constexpr int kSelMaxPositions = 8192;
constexpr int kSelMaxLanes = 64;
constexpr int kSelMaxDelims = 16;
constexpr int kSelMaxBoundaryIds = 32;
struct SelHost {
  int L, B, N, mode, fallback_k, eos_id, t_min, n_delim;
  float tau, rho_min, tau_future;
  int32_t delim[kSelMaxDelims];
  // ValidBoundary id sets (empty = always valid).
  int n_digit, n_open, n_close;
  int32_t digit[kSelMaxBoundaryIds], open[kSelMaxBoundaryIds], close[kSelMaxBoundaryIds];
  uint8_t role[kSelMaxLanes];
  int32_t b_len[kSelMaxLanes];
  int32_t t_lane[kSelMaxLanes];
  int32_t k_lane[kSelMaxLanes];
};
hipError_t launch_select(const SelHost& h, const float* conf, const int32_t* argmax,
                         const int32_t* row_pos, int32_t* tokens, uint8_t* is_masked,
                         uint8_t* unmask_flag, int32_t* unmasked_pos, int32_t* still_pos,
                         int32_t* counts, int32_t* lane_stats, uint8_t* delim_flag,
                         hipStream_t stream);

}  // namespace al
