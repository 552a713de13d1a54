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
// d=4096) for a few tens to a few hundred hidden rows, so
// lmhead_partial_kernel is shaped for HBM streaming first and MFMA reuse
// second (measured on MI355X):
// * each wavefront owns 32 or 64 vocabulary rows (A operands of the 32x32x16
//   bf16 MFMA) and loads them straight into registers, one to three chunks
//   ahead; each W element is used by one wavefront only;
// * the scored hidden rows (B operand, <= 224 rows per column tile; more
//   rows take several tiles of 224, or of 128 on the packed weight, each
//   streaming W again) are staged per block of K once per workgroup in LDS
//   and shared by its 8 wavefronts;
// * workgroups are dealt to the 8 XCDs in contiguous runs of vocab tiles;
//   on W as given the 512-row workgroups walk K in a rotated order per
//   group of tiles (the packed copy, read chunk-major, needs none);
// * the epilogue writes one partial (m, s, argmax) per column and vocab
//   tile; lmhead_merge_kernel combines them in a fixed order, so results
//   are bitwise reproducible.  (A single-kernel merge by the last workgroup
//   to arrive needs agent-scope fences, which on gfx950 write back and
//   invalidate the L2 in every workgroup; the separate launch is cheaper.)
#include <math.h>

#include <atomic>
#include <mutex>

#include "../../include/asynclane.h"
#include "common.h"
#include "launch.h"

namespace al {

constexpr int LM_MAX_NF = 7;
constexpr int gcd_c(int a, int b) { return b == 0 ? a : gcd_c(b, a % b); }
constexpr int lcm_c(int a, int b) { return a / gcd_c(a, b) * b; }     // <= 224 scored rows per column tile
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
  // Plain W: vocab tile vt covers rows [vt*V/n_vt, (vt+1)*V/n_vt) (<= 32*RT*WAVES
  // rows).  Packed W: it covers the 32-row units [vt*n_hg/n_vt, (vt+1)*n_hg/n_vt).
  int n_vt, n_nt, nt_cols, tiles_total, tiles_per_xcd;
  int n_hg;  // packed W: 32-row units, ceil(V / 32)
};

// Packed W layout (lmhead_pack_weight).  W is cut into 32-row units u =
// v / 32 and 64-element K chunks c = k / 64.  Inside a (c, u) block the
// elements sit exactly as one wavefront's A-operand loads take them: 4
// MFMA k-steps s of 64 lanes x 8 elements, lane l = 32 h + r holding row
// 32u + r, K elements 64c + 16s + 8h .. +8.  Blocks are ordered K-chunk
// major, (c * n_hg + u): while the workgroups stream their tiles in step,
// the chip reads one contiguous window of ~V * 128 bytes per chunk, like a
// linear read, instead of 128-byte pieces of every row.  Rows past V and
// K past d are zero.
__device__ __host__ __forceinline__ size_t packed_offset(int c, int u, int s, int l, int n_hg) {
  return ((((size_t)c * n_hg + u) * 4 + s) * 64 + l) * 8;
}

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

// WAVES wavefronts x 32*RT vocab rows per workgroup (VT = 32*RT*WAVES), NF
// 32-column fragments (NT = 32*NF scored rows) per tile, 32x32x16 bf16 MFMA.
// * RT = 2 (N <= 96): each wavefront owns two 32-row A tiles and uses every
//   B fragment it reads from LDS for both, and a workgroup covers 512 vocab
//   rows, so the hidden-chunk traffic per W byte halves.  Staging the hidden
//   chunks was the main cost over a plain W stream (MI355X, LLaDA shape:
//   186 µs with 32-row wavefronts, 177 µs with 64-row ones, 170 µs with no
//   staging at all).
// * W streams straight into registers, KC elements per chunk, PF chunks
//   ahead (lane half h of row r takes K elements kc + 16s + 8h .. +8; over
//   a chunk each row is read as one 2*KC-byte run).  Each W element is used
//   by one wavefront only.
// * The hidden rows are staged in blocks of SC chunks (NT x KC*SC),
//   double-buffered in LDS with one barrier per block and shared by the
//   workgroup's wavefronts.  The next block's loads go into registers one
//   block ahead, issued before the W prefetch, so the wait for them (the
//   load counter is in order) never waits for W loads still needed later.
// * 32-row A tiles halve the B-operand LDS reads per FLOP of 16x16x32
//   steps, and 256*RT vocab rows per workgroup keep the hidden-chunk
//   traffic at NT/(256*RT) of the W traffic.
// * Two wavefronts per SIMD: the accumulators take 16*NF*RT registers.
// PACKED: W in the packed layout above (KC = 64, no K rotation: the
// K-chunk-major order already spreads the reads evenly).
// WNT: W is loaded non-temporally.  Used for the packed layout with one
// column tile: every W element is then read exactly once per call, and
// every load instruction takes 1 KB of consecutive bytes (whole cache
// lines), so caching W only evicts other data.  MI355X, per call, one box,
// two runs each: LLaDA shape 187-192 -> 172-174 us, Dream shape 265 ->
// 259-261 us, Long shape unchanged; the bench step 0.201-0.203 -> 0.189-0.190
// ms.  On W as given (128-byte row pieces gathered over four load
// instructions) the same hint is much slower (LLaDA shape 218 -> 323 us):
// a line evicted after its first 32-byte piece is fetched again for the
// next, so that layout keeps ordinary loads, and so do several column
// tiles, which re-read W from L2.
template <int NF, bool RAGGED, int WAVES, int KC, int PF, int RT, int SC, bool ROT, bool PACKED,
          bool WNT>
__global__ __launch_bounds__(WAVES * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void lmhead_partial_kernel(LmParams p) {
  static_assert(!PACKED || (KC == 64 && !ROT), "packed W: 64-element chunks, natural K order");
  constexpr int THREADS = WAVES * 64;
  constexpr int VT = 32 * RT * WAVES;            // vocab rows per workgroup
  constexpr int STEPS = KC / 16;                 // MFMA k-steps per chunk
  constexpr int NT = 32 * NF;                    // scored rows (columns) per tile
  constexpr int KH = KC * SC;                    // K elements per staged hidden block
  constexpr int KSEG = KH / 8;                   // 16-byte segments per staged row
  // +16 B per staged row: the 32 rows read by one half-wavefront start
  // 4 banks apart, so the B-operand reads are conflict-free.
  constexpr int STRIDE = KH + 8;
  constexpr int SEGS = NT * KSEG;
  constexpr int HREG = (SEGS + THREADS - 1) / THREADS;
  constexpr int BUF = NT * STRIDE;
  __shared__ __attribute__((aligned(16))) uint16_t hs[2 * BUF];
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
  const int r32 = lane & 31;
  const int h = lane >> 5;
  const int d = p.d;
  int vb, ve, ub = 0, ue = 0;
  if (PACKED) {
    ub = (int)((long long)vt * p.n_hg / p.n_vt);
    ue = (int)((long long)(vt + 1) * p.n_hg / p.n_vt);
    vb = ub * 32;
    ve = min(p.V, ue * 32);
  } else {
    vb = (int)((long long)vt * p.V / p.n_vt);
    ve = (int)((long long)(vt + 1) * p.V / p.n_vt);
  }
  const int v0 = vb + w * 32 * RT;
  const int n0 = nt * p.nt_cols;
  const int ncols = min(NT, p.N - n0);

  // Rows past the tile read its last row (cache hits; dropped in the
  // epilogue).  Packed: wrow[q] is this lane's element of unit u, chunk 0,
  // step 0; chunk c, step s adds c * n_hg * 2048 + s * 512.
  const uint16_t* wrow[RT];
#pragma unroll
  for (int q = 0; q < RT; ++q) {
    if (PACKED)
      wrow[q] = p.W + packed_offset(0, min(ub + w * RT + q, ue - 1), 0, lane, p.n_hg);
    else
      wrow[q] = p.W + (size_t)min(v0 + 32 * q + r32, ve - 1) * d;
  }
  const size_t wchunk = (size_t)p.n_hg * 2048;   // packed: elements per K chunk
  // Hidden staging: segment i of this thread is row hrow0 + i * RSTEP of
  // the column tile, at K offset hk of the staged block.  Only rows < ncols
  // are loaded and stored each block; rows ncols..NT-1 (read by the MFMAs
  // of the last fragment) are zeroed once in both buffers, and segments
  // past NT rows do nothing.
  static_assert(THREADS % KSEG == 0, "every segment of a thread has the same K offset");
  constexpr int RSTEP = THREADS / KSEG;          // staged rows per segment round
  const int hk = (tid % KSEG) * 8;               // this thread's K offset in a block
  const int hrow0 = tid / KSEG;                  // segment i is row hrow0 + i * RSTEP
  unsigned hoff[HREG];
  unsigned hvalid = 0;
#pragma unroll
  for (int i = 0; i < HREG; ++i) {
    const int row = hrow0 + i * RSTEP;
    const bool ok = row < ncols;
    const int n = n0 + (ok ? row : 0);
    hoff[i] = (unsigned)(p.row_idx ? p.row_idx[n] : n) * (unsigned)d + (unsigned)hk;
    hvalid |= (ok ? 1u : 0u) << i;
    if (!ok && row < NT) {
      *reinterpret_cast<bf16x8*>(&hs[row * STRIDE + hk]) = zero_bf16x8();
      *reinterpret_cast<bf16x8*>(&hs[BUF + row * STRIDE + hk]) = zero_bf16x8();
    }
  }

  // EOS-suppression flags of this lane's columns, read before the K loop:
  // a global load issued in the epilogue waits behind the W stream (per
  // workgroup, LLaDA shape: epilogue 3.8-4.5 us against 6.1-7.8 us, from
  // s_memrealtime stamps).
  unsigned supmask = 0;
  if (p.sup) {
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const int n = n0 + f * 32 + r32;
      if (n < p.N && p.sup[n]) supmask |= 1u << f;
    }
  }

  f32x16 acc[RT][NF];
#pragma unroll
  for (int q = 0; q < RT; ++q)
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[q][f][r] = 0.f;

  constexpr int RING = PF + 1;   // W register slots (chunks)
  bf16x8 wr[RING][RT * STEPS], hr[HREG];
  auto ld = [](const uint16_t* a) {
    if (WNT) return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(reinterpret_cast<const i32x4*>(a)));
    return load_bf16x8(a);
  };
  auto load_w1 = [&](int q, int kc, int s) {
    if (PACKED) return ld(wrow[q] + (size_t)(kc >> 6) * wchunk + s * 512);
    const int k = kc + s * 16 + h * 8;
    if (RAGGED) return ld(wrow[q] + (k < d ? k : 0));
    return ld(wrow[q] + k);
  };
  auto load_w = [&](bf16x8* wv, int kc) {
#pragma unroll
    for (int q = 0; q < RT; ++q)
#pragma unroll
      for (int s = 0; s < STEPS; ++s) wv[q * STEPS + s] = load_w1(q, kc, s);
  };
  auto load_h = [&](bf16x8* hv, int kh) {
#pragma unroll
    for (int i = 0; i < HREG; ++i) {
      if (!((hvalid >> i) & 1u)) continue;
      if (RAGGED)
        hv[i] = load_bf16x8(p.hidden + (hk + kh < d ? hoff[i] + kh : hoff[i] - hk));
      else
        hv[i] = load_bf16x8(p.hidden + (hoff[i] + kh));
    }
  };
  auto store_h = [&](const bf16x8* hv, uint16_t* buf, int kh) {
#pragma unroll
    for (int i = 0; i < HREG; ++i) {
      if (!((hvalid >> i) & 1u)) continue;
      const bool kin = !RAGGED || hk + kh < d;
      *reinterpret_cast<bf16x8*>(&buf[(hrow0 + i * RSTEP) * STRIDE + hk]) = kin ? hv[i] : zero_bf16x8();
    }
  };
  auto mma = [&](const bf16x8* wv, const uint16_t* buf) {
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        const bf16x8 bv = *reinterpret_cast<const bf16x8*>(&buf[(f * 32 + r32) * STRIDE + s * 16 + h * 8]);
#pragma unroll
        for (int q = 0; q < RT; ++q) acc[q][f] = mfma32x32x16(wv[q * STEPS + s], bv, acc[q][f]);
      }
    }
  };

  // Chunk c (KC columns of K): W in register slot c % RING.  The hidden
  // rows are staged SC chunks at a time: block s (chunks s*SC ..) sits in
  // LDS buffer s % 2 while the registers hr bring block s + 1; at the end
  // of block s that block is stored (the only barrier follows) and hr is
  // refilled with block s + 2.  Two-chunk blocks cost less than one
  // staging step per chunk (MI355X, per call: LLaDA 203 -> 201 us, Dream
  // 275 -> 269 us, Long 293 -> 286 us, Wide 754 -> 731 us).
  //
  // With ROT the workgroup walks the K blocks in a rotated order (position
  // sb covers block (sb + rot) % nsc).  Without it, the 512-row workgroups,
  // which run in step, all read one column offset of W at a time; how those
  // requests spread over the HBM channels then depends on where W happens
  // to sit physically.  Six copies of the LLaDA-shape W in one process
  // took 190-241 us per call unrotated, 186-187 us rotated.  The 256-row
  // workgroups are not sensitive to it, and lose 2.6% rotated (Dream).
  // Groups of 8 consecutive tiles (one XCD's neighbours) share a rotation,
  // so a hidden block read by one of them is still in L2 for the others:
  // per-tile rotations re-fetched it (HBM/MALL fetch 1.125 GB per call
  // against 1.061 GB, the same time).  Every position runs all SC chunks
  // of its block, so the chunk count is nsc * SC (a partial last block's
  // extra chunk reads zeros from the staged hidden rows).
  const int nsc = (d + KH - 1) / KH;
  const int nch = ROT ? nsc * SC : (d + KC - 1) / KC;
  const int rot = ROT ? (int)(((long long)(t >> 3) * 13) % nsc) : 0;
  auto kblk = [&](int sb) {
    const int q = sb + rot;
    return (q < nsc ? q : q - nsc) * KH;
  };
  auto kchunk = [&](int cc) { return kblk(cc / SC) + (cc % SC) * KC; };
  load_h(hr, kblk(0));
#pragma unroll
  for (int j = 0; j < PF; ++j)
    if (j < nch) load_w(wr[j], kchunk(j));
  store_h(hr, hs, kblk(0));
  if (nsc > 1) load_h(hr, kblk(1));
  __syncthreads();
  // jl = c % SC and hb = (c / SC) % 2 are static in the unrolled loops
  // (they start at multiples of U).
  auto chunk = [&](int c, int jl, int hb, const bf16x8* cur, bf16x8* pre, bool full) {
    if (full || c + PF < nch) load_w(pre, kchunk(c + PF));
    __builtin_amdgcn_sched_barrier(0);
    mma(cur, hs + hb * BUF + jl * KC);
    if (jl == SC - 1) {
      const int sb = c / SC;
      if (full || sb + 1 < nsc) store_h(hr, hs + (hb ^ 1) * BUF, kblk(sb + 1));
      __syncthreads();
      if (full || sb + 2 < nsc) load_h(hr, kblk(sb + 2));
    }
  };
  // Steady state: unrolled over lcm(RING, 2 * SC) chunks so every register
  // index and buffer offset is static; all loads in range there.
  constexpr int U = lcm_c(RING, 2 * SC);
  constexpr int AHEAD = PF + 1 > 2 * SC ? PF + 1 : 2 * SC;
  int c = 0;
  for (; c + U - 1 + AHEAD < nch; c += U) {
#pragma unroll
    for (int j = 0; j < U; ++j)
      chunk(c + j, j % SC, (j / SC) & 1, wr[j % RING], wr[(j + PF) % RING], true);
  }
#pragma unroll
  for (int j = 0; j < U - 1 + AHEAD; ++j)
    if (c + j < nch)
      chunk(c + j, j % SC, (j / SC) & 1, wr[j % RING], wr[(j + PF) % RING], false);

  // Epilogue: lane (r32, h) holds vocab rows v0 + 32q + 8*(r/4) + 4h + r%4
  // (q < RT, r = 0..15) of column n0 + 32f + r32.  Rows are visited in
  // ascending order, so the first maximum is the lowest index.
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const bool sup_row = (supmask >> f) & 1u;
    // Branch-free: excluded rows become -inf, whose exponential is 0.
    float z[RT][16];
    float m = -INFINITY;
    int idx = 0x7fffffff;
#pragma unroll
    for (int q = 0; q < RT; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = v0 + 32 * q + 8 * (r >> 2) + 4 * h + (r & 3);
        const bool ok = v < ve && !(sup_row && v == p.eos_id);
        z[q][r] = ok ? acc[q][f][r] : -INFINITY;
        const bool gt = z[q][r] > m;
        m = gt ? z[q][r] : m;
        idx = gt ? v : idx;
      }
    const float m0 = (m == -INFINITY) ? 0.f : m;
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < RT; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) s += exp2_fast((z[q][r] - m0) * LM_LOG2E);
    merge_state(m, s, idx, __shfl_xor(m, 32, kWave), __shfl_xor(s, 32, kWave),
                __shfl_xor(idx, 32, kWave));
    if (h == 0) {
      red_m[w][f * 32 + r32] = m;
      red_s[w][f * 32 + r32] = s;
      red_i[w][f * 32 + r32] = idx;
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
// Row tiles per wavefront and W chunks in flight per fragment count (no
// register spills at two wavefronts per SIMD): up to 96 columns two 32-row
// tiles with one chunk in flight (two spill; LLaDA shape 201 us against
// 205 us); 128 columns one tile and three chunks (Dream shape 273 us
// against 277 us); above, one tile and two chunks.  Chunks of 64 K
// elements (128-byte W runs per row).  Hidden rows are staged four chunks
// at a time up to 128 columns (over six W placements: LLaDA shape 186.5 us
// against 187.8 us with two, 101 KB of LDS, 243 registers; Dream shape
// 260.3 us against 264.4 us, 135 KB, 224 registers), two above.
// Rejected for up to 96 columns: 32-element chunks three or four ahead
// (207 / 199.5 us: shorter runs per row), one 32-row tile with
// 128-element chunks one or two ahead (196-210 us).
constexpr int lm_rt(int nf) { return nf <= 3 ? 2 : 1; }
constexpr int lm_pf(int nf) { return nf <= 3 ? 1 : (nf == 4 ? 3 : 2); }
constexpr int lm_sc(int nf) { return nf <= 4 ? 4 : 2; }
constexpr int LM_KC = 64;
// More than 224 columns take several column tiles, each streaming W
// again (mostly from L2: the column tiles of a vocab tile run on
// neighbouring workgroups).  On the packed weight, 128-column tiles with
// two 32-row tiles per wavefront replace 224-column tiles with one there:
// every B fragment read from LDS feeds two MFMAs, and a workgroup's
// hidden block serves 512 vocab rows instead of 256 (these shapes are not
// HBM-bound).  Wide shape, N = 614 (one box, two runs each): 710 us
// against 776 us per call; at 128 and 205 columns (one column tile) the
// same change is slower (Dream +8%, Long +2.5%), and on the plain weight
// too (801 against 735 us: that variant spills).
constexpr int LM_MULTI_NF = 4;
constexpr int LM_MULTI_PF = 1;
constexpr int LM_MULTI_SC = 2;

// Column tiling: n_nt tiles of nf 32-column fragments (<= 224 columns),
// rt 32-row vocabulary tiles per wavefront.
struct LmLayout {
  int nf, rt, nt_cols, n_nt, n_vt;
  size_t total;
};

// Compute units of the current device (cached per device).
static int lm_cu_count() {
  static int cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] <= 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

// Packed W is tiled in whole 32-row units (a tile holds up to RT * 8 of
// them), plain W in rows; both balance the tiles over the CUs the same way.
static LmLayout lm_layout(int N, int V, bool packed) {
  LmLayout L{};
  const int frags = N > 0 ? (N + 31) / 32 : 1;
  const bool multi = packed && frags > LM_MAX_NF;
  const int per_tile = multi ? LM_MULTI_NF : LM_MAX_NF;
  L.n_nt = N > 0 ? (frags + per_tile - 1) / per_tile : 0;
  L.nf = N > 0 ? (frags + L.n_nt - 1) / L.n_nt : 1;
  L.rt = multi ? 2 : lm_rt(L.nf);
  L.nt_cols = 32 * L.nf;
  // One workgroup per CU runs at a time.  When the vocabulary needs more
  // than one round of full tiles, the tile count is rounded up to a
  // multiple of the CU count and the rows are spread evenly, so the last
  // round is not partly empty (V = 152064 on W as given: 594 full tiles
  // would take 3 rounds at 77% use; 768 tiles of 198 rows take 3 even
  // rounds).  A packed tile holds whole 32-row units, one per wavefront
  // row tile; where the even spread would leave more than 1/8 of those
  // slots repeating a tile's last unit (MFMA work without new W), the full
  // tiles are kept: V = 152064 at 128 columns takes 594 tiles of 8 units
  // instead of 768 of 6.19 (per call, one box, three runs each: 262-272
  // us against 279-287 us).
  const int vt_rows = 32 * L.rt * LM_WAVES;
  const int base = packed ? ((V + 31) / 32 + vt_rows / 32 - 1) / (vt_rows / 32)
                          : (V + vt_rows - 1) / vt_rows;
  const int units = lm_cu_count();
  L.n_vt = base <= units ? base : units * ((base + units - 1) / units);
  if (packed && L.n_vt > base) {
    const long long n_hg = (V + 31) / 32, slots = (long long)L.n_vt * (vt_rows / 32);
    if (8 * n_hg < 7 * slots) L.n_vt = base;
  }
  L.total = sizeof(LmPartial) * (size_t)L.n_nt * L.n_vt * L.nt_cols;
  return L;
}

// Partials of lmhead_confidence_noalloc.  In host code `scratch` names a
// host-side stand-in, not device memory: kernels get the device address
// that hipGetSymbolAddress returns for the current device (each GPU holds
// its own copy of the array).
static __device__ __align__(256) unsigned char scratch[AL_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
static std::atomic<void*> g_scratch_addr[kMaxDevices];
static std::mutex g_scratch_mu;

size_t lmhead_scratch_bytes() { return sizeof(scratch); }

hipError_t lmhead_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    p = g_scratch_addr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return e;
      if (!p) return hipErrorInvalidSymbol;
      g_scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return hipSuccess;
}

// Either layout's partials fit (one size query serves both entry points).
size_t lmhead_workspace_bytes(int N, int d, int V) {
  (void)d;
  if (N <= 0 || V <= 0) return 0;
  const size_t a = lm_layout(N, V, false).total, b = lm_layout(N, V, true).total;
  return a > b ? a : b;
}

size_t lmhead_packed_bytes(int d, int V) {
  return (size_t)((d + 63) / 64) * 64 * (size_t)((V + 31) / 32) * 32 * sizeof(uint16_t);
}

// One 16-byte segment per thread and step: segment o of the packed buffer
// is lane l = o % 64, step s = (o / 64) % 4 of block (c, u) = o / 256.
__global__ __launch_bounds__(256) void lmhead_pack_kernel(const uint16_t* W, int d, int V,
                                                          int n_hg, long long n_seg, uint16_t* Wp) {
  for (long long o = (long long)blockIdx.x * 256 + threadIdx.x; o < n_seg;
       o += (long long)gridDim.x * 256) {
    const int l = (int)(o & 63);
    const int st = (int)((o >> 6) & 3);
    const long long blk = o >> 8;
    const int u = (int)(blk % n_hg);
    const int c = (int)(blk / n_hg);
    const int v = u * 32 + (l & 31);
    const int k = c * 64 + st * 16 + (l >> 5) * 8;
    i32x4 val = {0, 0, 0, 0};
    if (v < V && k < d) val = *reinterpret_cast<const i32x4*>(W + (size_t)v * d + k);
    reinterpret_cast<i32x4*>(Wp)[o] = val;
  }
}

hipError_t launch_lmhead_pack(const uint16_t* W, int d, int V, uint16_t* Wp, hipStream_t stream) {
  const int n_hg = (V + 31) / 32;
  const long long n_seg = (long long)((d + 63) / 64) * n_hg * 256;
  hipLaunchKernelGGL(lmhead_pack_kernel, dim3(8192), dim3(256), 0, stream, W, d, V, n_hg, n_seg, Wp);
  return hipGetLastError();
}

hipError_t launch_lmhead(const uint16_t* hidden, const int32_t* row_idx, int N,
                         const uint16_t* W, int d, int V, const uint8_t* sup, int eos_id,
                         float* conf, int32_t* argmax, float* lse, void* ws,
                         hipStream_t stream, bool packed) {
  if (N <= 0) return hipSuccess;
  const LmLayout L = lm_layout(N, V, packed);
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
  p.n_hg = (V + 31) / 32;
  const dim3 grid(8 * p.tiles_per_xcd), block(LM_WAVES * 64);
  // The plain kernel assumes d % (KC * SC) == 0; other d take the RAGGED variant.
#define AL_LM_LAUNCH1(F, RG, PK, NT)                                                          \
  hipLaunchKernelGGL((lmhead_partial_kernel<F, RG, LM_WAVES, LM_KC, lm_pf(F), lm_rt(F), lm_sc(F), \
                                            !(PK) && lm_rt(F) == 2, PK, NT>),                 \
                     grid, block, 0, stream, p)
#define AL_LM_LAUNCH(F, RG, PK) AL_LM_LAUNCH1(F, RG, PK, PK)
#define AL_LM_CASE(F)                                                                         \
  case F:                                                                                     \
    if (d % (LM_KC * lm_sc(F)) != 0) {                                                        \
      if (packed) AL_LM_LAUNCH(F, true, true); else AL_LM_LAUNCH(F, true, false);             \
    } else {                                                                                  \
      if (packed) AL_LM_LAUNCH(F, false, true); else AL_LM_LAUNCH(F, false, false);           \
    }                                                                                         \
    break;
#define AL_LM_MULTI(RG, PK)                                                                   \
  hipLaunchKernelGGL((lmhead_partial_kernel<LM_MULTI_NF, RG, LM_WAVES, LM_KC, LM_MULTI_PF, 2,  \
                                            LM_MULTI_SC, false, PK, false>),                  \
                     grid, block, 0, stream, p)
  if (L.nf == LM_MULTI_NF && L.rt == 2) {  // only the packed layout tiles this way
    if (d % (LM_KC * LM_MULTI_SC) != 0)
      AL_LM_MULTI(true, true);
    else
      AL_LM_MULTI(false, true);
  } else switch (L.nf) {
    AL_LM_CASE(1)
    AL_LM_CASE(2)
    AL_LM_CASE(3)
    AL_LM_CASE(4)
    AL_LM_CASE(5)
    AL_LM_CASE(6)
    default:
      AL_LM_CASE(7)
  }
#undef AL_LM_CASE
#undef AL_LM_MULTI
#undef AL_LM_LAUNCH
#undef AL_LM_LAUNCH1
  hipLaunchKernelGGL(lmhead_merge_kernel, dim3(N), dim3(LM_MERGE_THREADS), 0, stream, p.part, N,
                     L.n_vt, L.nt_cols, conf, argmax, lse);
  return hipGetLastError();
}

}  // namespace al
