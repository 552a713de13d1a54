// Fused LM head + confidence for gfx950.
//
// For each scored hidden row n the kernels form z[v] = <H[row_idx[n]], W[v]>
// on bf16 MFMA with fp32 accumulation and reduce every vocabulary tile to a
// (max m, sum s = sum exp(z - m), first argmax) triple in registers, so the
// logits never reach memory (paper Section 3.2: confidence-based transfer
// uses the max-probability token of each masked position; refine lanes
// suppress EOS).
//
// The step streams the whole weight W ([V][d] bf16, ~1 GB at V=126464,
// d=4096) once for a few hundred hidden rows, so lmhead_partial_kernel is
// shaped for HBM streaming rather than for MFMA reuse (measured on MI355X):
// * each wavefront owns 16 vocabulary rows (the A operand of the 16x16x32
//   bf16 MFMA); per chunk it loads 256 contiguous bytes of each row
//   (4 instructions x 4 lanes x 16 B, issued back to back) straight into
//   registers, two chunks ahead of the MFMAs -- each W element is used by
//   one wavefront only;
// * the chunk of the scored hidden rows (B operand, <= 128 rows) is staged
//   once per workgroup in LDS and shared by its wavefronts; the LDS buffer
//   is small enough for several workgroups per CU, which keeps enough W
//   loads in flight;
// * workgroups are dealt to the 8 XCDs in contiguous runs of vocab tiles;
// * the epilogue writes one partial (m, s, argmax) per column and vocab
//   tile; lmhead_merge_kernel combines them in a fixed order, so results
//   are bitwise reproducible.  (A single-kernel merge by the last workgroup
//   to arrive needs agent-scope fences, which on gfx950 write back and
//   invalidate the L2 in every workgroup; the separate launch is cheaper.)
#include <math.h>

#include "common.h"
#include "launch.h"

namespace al {

constexpr int LM_MAX_FRAG = 8;   // <= 128 scored rows per column tile
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
  LmPartial* part;  // [n_nt][nt_cols][n_vt]: a row's partials are contiguous
  int N, d, V, eos_id;
  int n_vt, n_nt, nt_cols, tiles_total, tiles_per_xcd;
};

// Merge (m2, s2, i2) into (m, s, i): max, rescaled sum, lowest index on ties.
// Commutative, so lanes that exchange states obtain identical bits.
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

// WAVES wavefronts x 16 vocab rows per workgroup.  W is streamed in chunks
// of KC hidden elements (each lane loads KC/4 contiguous elements of its row
// per chunk, PF chunks ahead of the MFMAs, so the MFMA work overlaps the
// stream).  The hidden chunk is staged once per workgroup in LDS.
// OCC: wavefronts per SIMD the register allocation must allow.
template <int NFRAG, bool RAGGED, int WAVES, int KC, int PF, int OCC>
__global__ __launch_bounds__(WAVES * 64) __attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void lmhead_partial_kernel(LmParams p) {
  constexpr int THREADS = WAVES * 64;
  constexpr int VT = 16 * WAVES;                 // vocab rows per workgroup
  constexpr int STEPS = KC / 32;                 // MFMA k-steps per chunk
  constexpr int KCH = KC;                        // hidden elements staged at once
  constexpr int NT = 16 * NFRAG;                 // scored rows (columns) per tile
  constexpr int KSEG = KCH / 8;                  // 16-byte segments per staged row
  // bf16 per staged row: +32 B of padding makes the B-operand reads below
  // conflict-free (measured on gfx950; +16 B costs 2x in bank conflicts).
  constexpr int STRIDE = KCH + 16;
  constexpr int SEGS = NT * KSEG;
  constexpr int HREG = (SEGS + THREADS - 1) / THREADS;
  // Rows past NT are written (by the last staging pass) but never read:
  // every thread stores, so the staging code has no divergent branch.
  constexpr int ROWS_STAGED = HREG * THREADS / KSEG;
  __shared__ __attribute__((aligned(16))) uint16_t hs[ROWS_STAGED * STRIDE];
  // After the K loop the staging buffer holds the per-wavefront (m, s, idx).
  static_assert(sizeof(hs) >= 3 * sizeof(float) * WAVES * NT, "reduction scratch");
  float (*red_m)[NT] = reinterpret_cast<float (*)[NT]>(&hs[0]);
  float (*red_s)[NT] = red_m + WAVES;
  int (*red_i)[NT] = reinterpret_cast<int (*)[NT]>(red_s + WAVES);

  const int b = blockIdx.x;
  const int t = (b & 7) * p.tiles_per_xcd + (b >> 3);
  if (t >= p.tiles_total) return;
  const int vt = t / p.n_nt;
  const int nt = t - vt * p.n_nt;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int r16 = lane & 15;
  const int g4 = lane >> 4;
  const int d = p.d;
  const int v0 = vt * VT + w * 16;
  const int n0 = nt * p.nt_cols;
  const int ncols = min(NT, p.N - n0);

  // Loads are unconditional and in bounds (clamped addresses); values are
  // not post-processed after loading.  A W segment past d meets hidden
  // values zeroed at the LDS store; rows past V are dropped in the epilogue.
  const uint16_t* wrow = p.W + (size_t)min(v0 + r16, p.V - 1) * d;
  const uint16_t* wlane = wrow + g4 * 8;
  // Hidden staging: thread tid moves segments tid + THREADS*i of the
  // NT x KSEG staged block (row-major); 32-bit row offsets (n_rows * d <
  // 2^31 is checked by the caller).
  unsigned hoff[HREG];
  int hcol[HREG];
  int hdst[HREG];
  unsigned hvalid = 0;
#pragma unroll
  for (int i = 0; i < HREG; ++i) {
    const int seg = tid + THREADS * i;
    const int row = seg / KSEG;
    const int k = (seg - row * KSEG) * 8;
    const bool ok = row < ncols;
    const int n = n0 + (ok ? row : 0);
    hoff[i] = (unsigned)(p.row_idx ? p.row_idx[n] : n) * (unsigned)d + (unsigned)k;
    hcol[i] = k;
    hdst[i] = row * STRIDE + k;
    hvalid |= (ok ? 1u : 0u) << i;
  }

  f32x4 acc[NFRAG];
#pragma unroll
  for (int f = 0; f < NFRAG; ++f)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[f][r] = 0.f;

  bf16x8 wr[PF + 1][STEPS], hr[HREG];
  // Step s of a chunk covers K elements kc + s*32 .. +32; lane group g4
  // takes kc + s*32 + g4*8 .. +8 on both operands, so each W load
  // instruction reads 64 contiguous bytes of every row of the wavefront.
  auto load_w = [&](bf16x8* wv, int kc) {
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      if (RAGGED) {
        const int k = kc + s * 32 + g4 * 8;
        wv[s] = load_bf16x8(wrow + (k < d ? k : 0));
      } else {
        wv[s] = load_bf16x8(wlane + kc + s * 32);
      }
    }
  };
  // Hidden segment i of the block starting at kh covers element
  // hcol[i] + kh of its row; past d it reads the row start instead and is
  // zeroed at the LDS store.
  auto load_h = [&](int kh) {
#pragma unroll
    for (int i = 0; i < HREG; ++i) {
      if (RAGGED)
        hr[i] = load_bf16x8(p.hidden + (hcol[i] + kh < d ? hoff[i] + kh : hoff[i] - hcol[i]));
      else
        hr[i] = load_bf16x8(p.hidden + (hoff[i] + kh));
    }
  };
  // Zeroing past d and for unused columns happens at the LDS store, where
  // the data is awaited anyway (a select right after a load would stall).
  auto store_h = [&](int kh) {
#pragma unroll
    for (int i = 0; i < HREG; ++i) {
      const bool kin = !RAGGED || hcol[i] + kh < d;
      *reinterpret_cast<bf16x8*>(&hs[hdst[i]]) = (kin && ((hvalid >> i) & 1u)) ? hr[i] : zero_bf16x8();
    }
  };
  // MFMA step s covers, for lane group g4, the K elements
  // kc + s*32 + g4*8 + e (e = 0..7) on both operands.
  auto mma = [&](const bf16x8* wv) {
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
#pragma unroll
      for (int f = 0; f < NFRAG; ++f) {
        const bf16x8 bv = *reinterpret_cast<const bf16x8*>(
            &hs[(f * 16 + r16) * STRIDE + s * 32 + g4 * 8]);
        acc[f] = mfma16x16x32(wv[s], bv, acc[f]);
      }
    }
  };

  // Chunk c uses register buffer c % (PF+1); W(c+PF) is prefetched while
  // chunk c is multiplied.  The next hidden chunk's loads are issued before
  // that prefetch (the load counter is in-order and the LDS store waits for
  // them).  The steady-state loop has every prefetch in range and no
  // branches; the last chunks are peeled.
  const int nch = (d + KC - 1) / KC;
  load_h(0);
#pragma unroll
  for (int j = 0; j < PF; ++j)
    if (j < nch) load_w(wr[j], j * KC);
  store_h(0);
  __syncthreads();
  auto chunk_full = [&](int c, const bf16x8* cur, bf16x8* pre) {
    load_h((c + 1) * KC);
    load_w(pre, (c + PF) * KC);
    __builtin_amdgcn_sched_barrier(0);
    mma(cur);
    __syncthreads();  // every wavefront is done with this hidden chunk
    store_h((c + 1) * KC);
    __syncthreads();
  };
  auto chunk_tail = [&](int c, const bf16x8* cur, bf16x8* pre) {
    const bool has_next = c + 1 < nch;
    if (has_next) load_h((c + 1) * KC);
    if (c + PF < nch) load_w(pre, (c + PF) * KC);
    mma(cur);
    if (has_next) {
      __syncthreads();
      store_h((c + 1) * KC);
      __syncthreads();
    }
  };
  int c = 0;
  for (; c + 2 * PF < nch; c += PF + 1) {
#pragma unroll
    for (int j = 0; j <= PF; ++j) chunk_full(c + j, wr[j], wr[(j + PF) % (PF + 1)]);
  }
#pragma unroll
  for (int j = 0; j < 2 * PF + 1; ++j)
    if (c + j < nch) chunk_tail(c + j, wr[j % (PF + 1)], wr[(j + PF) % (PF + 1)]);
  __syncthreads();

  // Epilogue: lane (r16, g4) holds vocab rows v0 + 4*g4 + r (r = 0..3) of
  // column n0 + f*16 + r16.
#pragma unroll
  for (int f = 0; f < NFRAG; ++f) {
    const int n = n0 + f * 16 + r16;
    const bool sup_row = (n < p.N) && p.sup && p.sup[n];
    float m = -INFINITY;
    int idx = 0x7fffffff;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int v = v0 + 4 * g4 + r;
      const bool ok = v < p.V && !(sup_row && v == p.eos_id);
      if (ok && acc[f][r] > m) {
        m = acc[f][r];
        idx = v;
      }
    }
    float s = 0.f;
    if (m != -INFINITY) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int v = v0 + 4 * g4 + r;
        const bool ok = v < p.V && !(sup_row && v == p.eos_id);
        if (ok) s += exp2_fast((acc[f][r] - m) * LM_LOG2E);
      }
    }
    merge_state(m, s, idx, __shfl_xor(m, 16, kWave), __shfl_xor(s, 16, kWave),
                __shfl_xor(idx, 16, kWave));
    merge_state(m, s, idx, __shfl_xor(m, 32, kWave), __shfl_xor(s, 32, kWave),
                __shfl_xor(idx, 32, kWave));
    if (g4 == 0) {
      red_m[w][f * 16 + r16] = m;
      red_s[w][f * 16 + r16] = s;
      red_i[w][f * 16 + r16] = idx;
    }
  }
  __syncthreads();
  for (int col = tid; col < NT; col += THREADS) {
    float m = red_m[0][col], s = red_s[0][col];
    int idx = red_i[0][col];
    for (int ww = 1; ww < WAVES; ++ww) merge_state(m, s, idx, red_m[ww][col], red_s[ww][col], red_i[ww][col]);
    LmPartial q;
    q.m = m;
    q.s = s;
    q.idx = idx;
    q.pad = 0;
    p.part[((size_t)nt * p.nt_cols + col) * p.n_vt + vt] = q;
  }
}

// One 256-thread workgroup per scored row.  Thread t merges vocab-tile
// partials t, t+256, ... in ascending order (loads issued four at a time so
// they overlap), then a fixed xor butterfly combines the lanes of each
// wavefront and wavefront 0 combines the four wavefront results in order.
constexpr int LM_MERGE_THREADS = 256;
__global__ __launch_bounds__(LM_MERGE_THREADS) void lmhead_merge_kernel(
    const LmPartial* part, int N, int n_vt, int nt_cols, float* conf, int32_t* argmax, float* lse) {
  __shared__ float sm[LM_MERGE_THREADS / kWave], ss[LM_MERGE_THREADS / kWave];
  __shared__ int si[LM_MERGE_THREADS / kWave];
  const int n = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int nt = n / nt_cols;
  const int col = n - nt * nt_cols;
  const LmPartial* base = part + ((size_t)nt * nt_cols + col) * n_vt;
  float m = -INFINITY, s = 0.f;
  int idx = 0x7fffffff;
  for (int v0 = tid; v0 < n_vt; v0 += 4 * LM_MERGE_THREADS) {
    LmPartial q[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int v = v0 + j * LM_MERGE_THREADS;
      q[j] = base[min(v, n_vt - 1)];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (v0 + j * LM_MERGE_THREADS < n_vt) merge_state(m, s, idx, q[j].m, q[j].s, q[j].idx);
  }
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1)
    merge_state(m, s, idx, __shfl_xor(m, o, kWave), __shfl_xor(s, o, kWave), __shfl_xor(idx, o, kWave));
  if (lane == 0) {
    sm[w] = m;
    ss[w] = s;
    si[w] = idx;
  }
  __syncthreads();
  if (tid == 0) {
    for (int ww = 1; ww < LM_MERGE_THREADS / kWave; ++ww) merge_state(m, s, idx, sm[ww], ss[ww], si[ww]);
    conf[n] = 1.0f / s;
    argmax[n] = idx;
    if (lse) lse[n] = m + logf(s);
  }
}

// ------------------------------------------------------------------ host
constexpr int LM_WAVES = 8;
constexpr int LM_KC = 128;
// Prefetch depth: two W chunks in flight where registers allow (up to 96
// scored columns), one beyond that (no spills at 128 columns).
constexpr int lm_pf(int nfrag) { return nfrag <= 6 ? 2 : 1; }
constexpr int LM_OCC = 4;
constexpr int LM_VT = 16 * LM_WAVES;

// Column tiling: n_nt tiles of nfrag 16-column fragments (<= 128 columns).
struct LmLayout {
  int nfrag, nt_cols, n_nt, n_vt;
  size_t total;
};

static LmLayout lm_layout(int N, int V) {
  LmLayout L{};
  const int frags = N > 0 ? (N + 15) / 16 : 1;
  L.n_nt = N > 0 ? (frags + LM_MAX_FRAG - 1) / LM_MAX_FRAG : 0;
  L.nfrag = N > 0 ? (frags + L.n_nt - 1) / L.n_nt : 1;
  L.nt_cols = 16 * L.nfrag;
  L.n_vt = (V + LM_VT - 1) / LM_VT;
  L.total = sizeof(LmPartial) * (size_t)L.n_nt * L.n_vt * L.nt_cols;
  return L;
}

size_t lmhead_workspace_bytes(int N, int d, int V) {
  (void)d;
  if (N <= 0 || V <= 0) return 0;
  return lm_layout(N, V).total;
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
  p.part = static_cast<LmPartial*>(ws);
  p.N = N;
  p.d = d;
  p.V = V;
  p.eos_id = eos_id;
  p.n_vt = L.n_vt;
  p.n_nt = L.n_nt;
  p.nt_cols = L.nt_cols;
  p.tiles_total = L.n_vt * L.n_nt;
  p.tiles_per_xcd = (p.tiles_total + 7) / 8;
  const dim3 grid(8 * p.tiles_per_xcd), block(LM_WAVES * 64);
  const bool ragged = d % LM_KC != 0;
#define AL_LM_CASE(F)                                                                         \
  case F:                                                                                     \
    if (ragged)                                                                               \
      hipLaunchKernelGGL((lmhead_partial_kernel<F, true, LM_WAVES, LM_KC, lm_pf(F), LM_OCC>), grid, block, 0,  \
                         stream, p);                                                          \
    else                                                                                      \
      hipLaunchKernelGGL((lmhead_partial_kernel<F, false, LM_WAVES, LM_KC, lm_pf(F), LM_OCC>), grid, block, 0, \
                         stream, p);                                                          \
    break;
  switch (L.nfrag) {
    AL_LM_CASE(1)
    AL_LM_CASE(2)
    AL_LM_CASE(3)
    AL_LM_CASE(4)
    AL_LM_CASE(5)
    AL_LM_CASE(6)
    AL_LM_CASE(7)
    default:
      AL_LM_CASE(8)
  }
#undef AL_LM_CASE
  hipLaunchKernelGGL(lmhead_merge_kernel, dim3(N), dim3(LM_MERGE_THREADS), 0, stream, p.part, N,
                     L.n_vt, L.nt_cols, conf, argmax, lse);
  return hipGetLastError();
}

}  // namespace al
