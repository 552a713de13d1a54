// Fused LM head + confidence for gfx950.
//
// For each scored hidden row n the kernel forms z[v] = <H[row_idx[n]], W[v]>
// on bf16 MFMA with fp32 accumulation and reduces every vocabulary tile to a
// running (max m, sum s = sum exp(z - m), first argmax) triple in registers,
// so the logits never reach memory (paper Section 3.2: confidence-based
// transfer uses the max-probability token of each masked position; refine
// lanes suppress EOS).
//
// Work split.  A workgroup (4 wavefronts) owns 128 vocabulary rows (32 per
// wavefront) and one tile of up to 128 hidden rows ("columns").  W is
// streamed from HBM exactly once, straight into registers (each W element is
// used by one wavefront only); the hidden-row chunk is staged once per
// workgroup in LDS and shared by the four wavefronts.  The vocabulary tiles
// of one column tile are merged in a fixed order by the last workgroup to
// arrive (two levels of arrival counters), so one launch produces the final
// conf / argmax / lse and the result is bitwise reproducible.
#include <math.h>

#include "common.h"
#include "launch.h"

namespace al {

constexpr int LM_WAVES = 4;
constexpr int LM_THREADS = LM_WAVES * kWave;
constexpr int LM_VT = 32 * LM_WAVES;        // vocabulary rows per workgroup
constexpr int LM_KC = 64;                   // K (hidden) elements per chunk
constexpr int LM_LDS_STRIDE = LM_KC + 8;    // bf16 per staged hidden row (+16 B pad)
constexpr int LM_MIN_GROUP = 16;            // vocab tiles merged by one level-1 merger
constexpr size_t LM_CNT_BYTES = 65536;      // arrival-counter area at the workspace start
constexpr float LM_LOG2E = 1.4426950408889634f;

struct LmPartial {
  float m;
  float s;
  int idx;
  int pad;
};

struct LmParams {
  const uint16_t* hidden;
  const int32_t* row_idx;
  const uint16_t* W;
  const uint8_t* sup;
  float* conf;
  int32_t* argmax;
  float* lse;
  LmPartial* part;    // [n_nt][n_vt][NT]
  LmPartial* gpart;   // [n_nt][n_groups][NT]
  unsigned* cnt1;     // [n_nt][n_groups]
  unsigned* cnt2;     // [n_nt]
  int N, d, V, eos_id;
  int n_vt, n_nt, n_groups, group, tiles_total, tiles_per_xcd;
};

// Merge (m2, s2, i2) into (m, s, i): max, rescaled sum, lowest index on ties.
// Commutative, so both halves of a lane pair obtain identical bits.
__device__ __forceinline__ void merge_state(float& m, float& s, int& idx, float m2, float s2,
                                            int idx2) {
  if (m2 == -INFINITY) return;
  if (m == -INFINITY) {
    m = m2;
    s = s2;
    idx = idx2;
    return;
  }
  const float M = fmaxf(m, m2);
  s = s * exp2_fast((m - M) * LM_LOG2E) + s2 * exp2_fast((m2 - M) * LM_LOG2E);
  if (m2 > m || (m2 == m && idx2 < idx)) idx = idx2;
  m = M;
}

template <int NB>
__global__ __launch_bounds__(LM_THREADS) __attribute__((amdgpu_waves_per_eu(3, 4)))
void lmhead_conf_kernel(LmParams p) {
  constexpr int NT = 32 * NB;
  __shared__ __attribute__((aligned(16))) uint16_t hs[2][NT * LM_LDS_STRIDE];
  __shared__ float red_m[LM_WAVES][NT];
  __shared__ float red_s[LM_WAVES][NT];
  __shared__ int red_i[LM_WAVES][NT];
  __shared__ unsigned s_ticket;

  // XCD-aware tile order: blocks are dealt round-robin to the 8 XCDs, so
  // give each XCD a contiguous run of tiles (the column tiles of one vocab
  // tile then share that XCD's L2 while their W rows are hot).
  const int b = blockIdx.x;
  const int t = (b & 7) * p.tiles_per_xcd + (b >> 3);
  if (t >= p.tiles_total) return;
  const int vt = t / p.n_nt;
  const int nt = t - vt * p.n_nt;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int r32 = lane & 31;
  const int hh = lane >> 5;
  const int d = p.d;
  const int v0 = vt * LM_VT + w * 32;
  const int n0 = nt * NT;

  const uint16_t* wrow = p.W + (size_t)min(v0 + r32, p.V - 1) * d;

  // Hidden-row staging: NT rows x 8 segments of 8 bf16 per chunk; thread
  // tid moves segments tid + 256*i.
  const uint16_t* hsrc[NB];
  int hdst[NB];
  int hk[NB];
  bool hok[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int seg = tid + LM_THREADS * i;
    const int row = seg >> 3;
    const int kseg = seg & 7;
    const int n = n0 + row;
    hok[i] = n < p.N;
    const int r = hok[i] ? (p.row_idx ? p.row_idx[n] : n) : 0;
    hsrc[i] = p.hidden + (size_t)r * d + kseg * 8;
    hk[i] = kseg * 8;
    hdst[i] = row * LM_LDS_STRIDE + kseg * 8;
  }

  bf16x8 wc[4], wn[4], hr[NB];
  auto load_w = [&](bf16x8* dst, int kc) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int k = kc + s * 16 + hh * 8;
      dst[s] = (k < d) ? load_bf16x8(wrow + k) : zero_bf16x8();
    }
  };
  auto load_h = [&](int kc) {
#pragma unroll
    for (int i = 0; i < NB; ++i)
      hr[i] = (hok[i] && kc + hk[i] < d) ? load_bf16x8(hsrc[i] + kc) : zero_bf16x8();
  };
  auto store_h = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NB; ++i)
      *reinterpret_cast<bf16x8*>(&hs[buf][hdst[i]]) = hr[i];
  };

  f32x16 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[nb][r] = 0.f;

  const int nch = (d + LM_KC - 1) / LM_KC;
  load_h(0);
  load_w(wc, 0);
  store_h(0);
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    const int buf = c & 1;
    const bool more = c + 1 < nch;
    if (more) {
      load_h((c + 1) * LM_KC);
      load_w(wn, (c + 1) * LM_KC);
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const bf16x8 bv = *reinterpret_cast<const bf16x8*>(
            &hs[buf][(nb * 32 + r32) * LM_LDS_STRIDE + s * 16 + hh * 8]);
        acc[nb] = mfma32x32x16(wc[s], bv, acc[nb]);
      }
    }
    if (more) store_h(buf ^ 1);
    __syncthreads();
#pragma unroll
    for (int s = 0; s < 4; ++s) wc[s] = wn[s];
  }

  // Epilogue: each lane holds 16 vocab rows of column n0 + nb*32 + r32.
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int n = n0 + nb * 32 + r32;
    const bool sup_row = (n < p.N) && p.sup && p.sup[n];
    float m = -INFINITY;
    int idx = 0x7fffffff;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int v = v0 + 8 * (r >> 2) + 4 * hh + (r & 3);
      const bool ok = v < p.V && !(sup_row && v == p.eos_id);
      if (ok && acc[nb][r] > m) {
        m = acc[nb][r];
        idx = v;
      }
    }
    float s = 0.f;
    if (m != -INFINITY) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = v0 + 8 * (r >> 2) + 4 * hh + (r & 3);
        const bool ok = v < p.V && !(sup_row && v == p.eos_id);
        if (ok) s += exp2_fast((acc[nb][r] - m) * LM_LOG2E);
      }
    }
    merge_state(m, s, idx, xor32(m), xor32(s), xor32(idx));
    if (hh == 0) {
      red_m[w][nb * 32 + r32] = m;
      red_s[w][nb * 32 + r32] = s;
      red_i[w][nb * 32 + r32] = idx;
    }
  }
  __syncthreads();
  if (tid < NT) {
    float m = red_m[0][tid], s = red_s[0][tid];
    int idx = red_i[0][tid];
#pragma unroll
    for (int ww = 1; ww < LM_WAVES; ++ww) merge_state(m, s, idx, red_m[ww][tid], red_s[ww][tid], red_i[ww][tid]);
    LmPartial q;
    q.m = m;
    q.s = s;
    q.idx = idx;
    q.pad = 0;
    p.part[((size_t)nt * p.n_vt + vt) * NT + tid] = q;
  }

  // ---- level 1: the last vocab tile of a group to arrive merges the group.
  const int g = vt / p.group;
  const int g_lo = g * p.group;
  const int g_hi = min(g_lo + p.group, p.n_vt);
  __threadfence();
  __syncthreads();
  if (tid == 0) s_ticket = atomicAdd(&p.cnt1[nt * p.n_groups + g], 1u);
  __syncthreads();
  if (s_ticket != (unsigned)(g_hi - g_lo - 1)) return;
  __threadfence();
  if (tid < NT) {
    float m = -INFINITY, s = 0.f;
    int idx = 0x7fffffff;
    for (int v = g_lo; v < g_hi; ++v) {
      const LmPartial q = p.part[((size_t)nt * p.n_vt + v) * NT + tid];
      merge_state(m, s, idx, q.m, q.s, q.idx);
    }
    LmPartial q;
    q.m = m;
    q.s = s;
    q.idx = idx;
    q.pad = 0;
    p.gpart[((size_t)nt * p.n_groups + g) * NT + tid] = q;
  }
  if (tid == 0) atomicExch(&p.cnt1[nt * p.n_groups + g], 0u);

  // ---- level 2: the last group merger of this column tile finishes it.
  __threadfence();
  __syncthreads();
  if (tid == 0) s_ticket = atomicAdd(&p.cnt2[nt], 1u);
  __syncthreads();
  if (s_ticket != (unsigned)(p.n_groups - 1)) return;
  __threadfence();
  if (tid < NT) {
    const int n = n0 + tid;
    if (n < p.N) {
      float m = -INFINITY, s = 0.f;
      int idx = 0x7fffffff;
      for (int gg = 0; gg < p.n_groups; ++gg) {
        const LmPartial q = p.gpart[((size_t)nt * p.n_groups + gg) * NT + tid];
        merge_state(m, s, idx, q.m, q.s, q.idx);
      }
      p.conf[n] = 1.0f / s;
      p.argmax[n] = idx;
      if (p.lse) p.lse[n] = m + logf(s);
    }
  }
  if (tid == 0) atomicExch(&p.cnt2[nt], 0u);
}

// ------------------------------------------------------------------ host
static int lm_nb(int N) { return N >= 128 ? 4 : (N + 31) / 32; }

// Workspace: [0, 64 KiB) holds only the arrival counters (cnt1 then cnt2),
// whatever the shape, so counters left at zero by any completed call are
// still zero for the next call even when the shape changes.  Partials
// follow.  The level-1 group grows when the counters would not fit.
struct LmLayout {
  int nb, nt_cols, n_nt, n_vt, n_groups, group;
  size_t off_cnt2, off_part, off_gpart, total;
};

static LmLayout lm_layout(int N, int V) {
  LmLayout L{};
  L.nb = N > 0 ? lm_nb(N) : 1;
  L.nt_cols = 32 * L.nb;
  L.n_nt = N > 0 ? (N + L.nt_cols - 1) / L.nt_cols : 0;
  L.n_vt = (V + LM_VT - 1) / LM_VT;
  const size_t max_cnt = LM_CNT_BYTES / sizeof(unsigned);
  L.group = LM_MIN_GROUP;
  for (;;) {
    L.n_groups = (L.n_vt + L.group - 1) / L.group;
    if ((size_t)L.n_nt * (L.n_groups + 1) <= max_cnt || L.group >= L.n_vt) break;
    L.group *= 2;
  }
  L.off_cnt2 = sizeof(unsigned) * (size_t)L.n_nt * L.n_groups;
  L.off_part = LM_CNT_BYTES;
  L.off_gpart = L.off_part + sizeof(LmPartial) * (size_t)L.n_nt * L.n_vt * L.nt_cols;
  L.total = L.off_gpart + sizeof(LmPartial) * (size_t)L.n_nt * L.n_groups * L.nt_cols;
  return L;
}

size_t lmhead_workspace_bytes(int N, int d, int V) {
  (void)d;
  if (N <= 0 || V <= 0) return 0;
  return lm_layout(N, V).total;
}

bool lmhead_counters_fit(int N, int V) {
  const LmLayout L = lm_layout(N, V);
  return (size_t)L.n_nt * (L.n_groups + 1) * sizeof(unsigned) <= LM_CNT_BYTES;
}

hipError_t launch_lmhead(const uint16_t* hidden, const int32_t* row_idx, int N,
                         const uint16_t* W, int d, int V, const uint8_t* sup, int eos_id,
                         float* conf, int32_t* argmax, float* lse, void* ws,
                         hipStream_t stream) {
  if (N <= 0) return hipSuccess;
  const LmLayout L = lm_layout(N, V);
  LmParams p{};
  p.hidden = hidden;
  p.row_idx = row_idx;
  p.W = W;
  p.sup = sup;
  p.conf = conf;
  p.argmax = argmax;
  p.lse = lse;
  char* base = static_cast<char*>(ws);
  p.cnt1 = reinterpret_cast<unsigned*>(base);
  p.cnt2 = reinterpret_cast<unsigned*>(base + L.off_cnt2);
  p.part = reinterpret_cast<LmPartial*>(base + L.off_part);
  p.gpart = reinterpret_cast<LmPartial*>(base + L.off_gpart);
  p.N = N;
  p.d = d;
  p.V = V;
  p.eos_id = eos_id;
  p.n_vt = L.n_vt;
  p.n_nt = L.n_nt;
  p.n_groups = L.n_groups;
  p.group = L.group;
  p.tiles_total = L.n_vt * L.n_nt;
  p.tiles_per_xcd = (p.tiles_total + 7) / 8;
  const dim3 grid(8 * p.tiles_per_xcd), block(LM_THREADS);
  switch (L.nb) {
    case 1: hipLaunchKernelGGL(lmhead_conf_kernel<1>, grid, block, 0, stream, p); break;
    case 2: hipLaunchKernelGGL(lmhead_conf_kernel<2>, grid, block, 0, stream, p); break;
    case 3: hipLaunchKernelGGL(lmhead_conf_kernel<3>, grid, block, 0, stream, p); break;
    default: hipLaunchKernelGGL(lmhead_conf_kernel<4>, grid, block, 0, stream, p); break;
  }
  return hipGetLastError();
}

}  // namespace al
