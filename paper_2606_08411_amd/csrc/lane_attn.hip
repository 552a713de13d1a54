// Shared-prefix lane-batched bidirectional attention for gfx950.
//
// Paper Section 3.2 ("Lane-local denoising") and Section 3.4 ("Shared-prefix
// lane batching", "Compact cache refresh and reuse"): every active lane of a
// prefix-sharing group is evaluated in one batched call; lane i's B query
// rows see the shared cached prefix, the blocks of its ancestors in the lane
// tree and, bidirectionally, its own block.
//
// Kernel layout.  A workgroup of 8 wavefronts serves one K/V head and eight
// query tiles (32 query rows of one lane and one query head each; for
// grouped-query attention the Hq/Hkv heads of a lane are adjacent tiles).
// Key tiles of 64 rows are staged once per workgroup in LDS, K and V both
// row-major as loaded, and consumed by every wavefront whose lane sees them,
// so a prefix tile read from HBM serves all lanes of the workgroup.  Both
// products run transposed on the 32x32x16 bf16 MFMA:
//     S^T = K Q^T      (lane l owns query row l%32, half of the keys)
//     O^T = V^T P^T    (lane l owns query row l%32, a quarter of D)
// so the running max / sum of the online softmax and the rescale of O stay
// inside a lane pair (l, l^32) and need no cross-lane broadcast.  The V^T
// operand comes from LDS transpose reads (ds_read_b64_tr_b16), which hand
// each lane 4 consecutive keys of one column.  Inside each 16-key MFMA step
// lane half h takes keys 4h..4h+3 and 8+4h..8+4h+3 on both operands, the
// keys the S^T accumulator gives it (a contraction is invariant under a
// common permutation of its summed index).
//
// Short grids (few heads x few lanes) either split each query tile's keys
// over the wavefronts of one workgroup (lane_attn_wsplit_kernel, merged in
// LDS) or, when that grid would not fit the chip at once, split the key
// tiles over blockIdx.z, whose unnormalised partials attn_merge_kernel
// combines.  The partial outputs are kept in bf16 (the softmax statistics
// in fp32): one rounding of a value that the output rounds to bf16 again,
// for half the partial traffic (Long shape, 4 splits: 49-51 -> 46.4 us per
// call, MI355X; outputs move by at most one bf16 step).
#include <math.h>

#include "common.h"
#include "launch.h"

namespace al {

constexpr int AT_WAVES = 8;
constexpr int AT_THREADS = AT_WAVES * kWave;
constexpr int AT_KT = 64;  // keys per staged tile
constexpr int AT_MAX_LANES = 64;
constexpr float AT_LN2 = 0.6931471805599453f;
// Deferred rescaling of the online softmax: a row's reference max moves
// only when a tile's scores exceed it by more than this many powers of two
// (P then stays <= 2^8, well inside bf16 and fp32 range), so O is rescaled
// in few tiles instead of in nearly every one.  O / l and m + log2 l are the
// same whichever reference is used, up to rounding.
constexpr float AT_RESCALE_LOG2 = 8.0f;

struct AttnParams {
  const uint16_t* q;       // [n_rows][Hq][D]
  const uint16_t* k_lane;  // [n_key_lanes*B_keys][Hkv][D] (lane mode)
  const uint16_t* v_lane;
  const uint16_t* k_pre;   // [P][Hkv][D]
  const uint16_t* v_pre;
  uint16_t* o;             // [n_rows][Hq][D]
  float* lse;              // [n_rows][Hq] or null
  uint16_t* part_o;        // [n_split][n_rows][Hq][D] bf16, unnormalised, when n_split > 1
  float* part_ml;          // [n_split][n_rows][Hq][2]
  int n_rows, rows_per_lane, tiles_per_lane, q_tiles_kv;
  int P, Hq, Hkv, g;
  int B_keys, n_key_lanes, lane_key_tiles, n_pre_tiles, total_key_tiles, n_split;
  float scale_log2;
  unsigned long long vis[AT_MAX_LANES];  // bit j: lane block j visible to lane i
};

// Two wavefronts per SIMD (<= 256 registers each, no spills at D = 128),
// one workgroup per CU: the next tile's loads go to registers while the
// current tile is multiplied, and the two wavefronts of a SIMD interleave
// their MFMA and VALU phases.  At one wavefront per SIMD (312 registers)
// the phases serialize: 530 us vs 270 us on the Wide lane pass (MI355X).
// Eight query tiles per workgroup instead of four (two 4-wavefront
// workgroups per CU) halve the K/V staging per MFMA: Wide lane + refresh
// passes 293-297 us against 308-310 us per call, Long 53 us either way
// (one box, two runs each; identical outputs).
constexpr int AT_OCC = 2;

template <int D>
__global__ __launch_bounds__(AT_THREADS) __attribute__((amdgpu_waves_per_eu(AT_OCC, AT_OCC)))
void lane_attn_kernel(AttnParams p) {
  constexpr int KS = D / 16;       // MFMA k-steps of S^T = K Q^T
  constexpr int DT = D / 32;       // 32-row tiles of O^T
  constexpr int KSTR = D + 8;      // bf16 per K row in LDS (+16 B: spreads banks)
  constexpr int VROW = D + 32;     // bf16 per V row in LDS (rows 64 B apart in bank order)
  constexpr int DSEG = D / 8;      // 16-byte segments per K/V row
  __shared__ __attribute__((aligned(16))) uint16_t k_s[AT_KT * KSTR];
  __shared__ __attribute__((aligned(16))) uint16_t v_s[AT_KT * VROW];

  const int hk = blockIdx.y;
  const int split = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar registers and branches
  const int r32 = lane & 31;
  const int hh = lane >> 5;
  const int lgrp = lane >> 4;  // 16-lane group of the transpose reads
  const int lg = lane & 15;
  const int per_lane = p.tiles_per_lane * p.g;

  // This wavefront's query tile.
  const int qt = blockIdx.x * AT_WAVES + w;
  const bool active = qt < p.q_tiles_kv;
  int lane_i = 0, c = 0, hg = 0;
  if (active) {
    lane_i = qt / per_lane;
    const int rem = qt - lane_i * per_lane;
    c = rem / p.g;
    hg = rem - c * p.g;
  }
  const int hq = hk * p.g + hg;
  const int row0 = lane_i * p.rows_per_lane + c * 32;
  int nrows = 0;
  if (active) nrows = min(min(32, p.rows_per_lane - c * 32), p.n_rows - row0);
  const unsigned long long my_vis = (active && p.n_key_lanes) ? p.vis[lane_i] : 0ull;
  unsigned long long wg_vis = 0ull;
  bool wg_active = false;
  for (int ww = 0; ww < AT_WAVES; ++ww) {
    const int qt2 = blockIdx.x * AT_WAVES + ww;
    if (qt2 < p.q_tiles_kv) {
      wg_active = true;
      if (p.n_key_lanes) wg_vis |= p.vis[qt2 / per_lane];
    }
  }
  if (!wg_active) return;  // uniform for the workgroup

  // Q fragments (B operand of S^T = K Q^T), kept in registers.
  bf16x8 qf[KS];
  {
    const bool ok = r32 < nrows;
    const uint16_t* qrow = p.q + ((size_t)(row0 + (ok ? r32 : 0)) * p.Hq + hq) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = ok ? load_bf16x8(qrow + ks * 16 + hh * 8) : zero_bf16x8();
  }

  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[dt][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  // Key tiles of this split: prefix tiles, then lane-block tiles.  Tiles no
  // wavefront of the workgroup sees are skipped (uniformly).
  const int kt0 = (int)((long long)split * p.total_key_tiles / p.n_split);
  const int kt1 = (int)((long long)(split + 1) * p.total_key_tiles / p.n_split);
  struct Tile {
    const uint16_t* k;  // first key row of the tile, K/V head hk applied
    const uint16_t* v;
    int nvalid;         // valid keys (1..64); 0 = no tile
    bool vis;           // this wavefront attends to it
  };
  auto tile_at = [&](int kt) -> Tile {
    Tile tl{nullptr, nullptr, 0, false};
    for (; kt < kt1; ++kt) {
      if (kt < p.n_pre_tiles) {
        const int r0 = kt * AT_KT;
        tl.k = p.k_pre + ((size_t)r0 * p.Hkv + hk) * D;
        tl.v = p.v_pre + ((size_t)r0 * p.Hkv + hk) * D;
        tl.nvalid = min(AT_KT, p.P - r0);
        tl.vis = active;
        return tl;
      }
      const int lt = kt - p.n_pre_tiles;
      const int j = lt / p.lane_key_tiles;
      const int sub = lt - j * p.lane_key_tiles;
      if (!((wg_vis >> j) & 1ull)) continue;
      const int r0 = j * p.B_keys + sub * AT_KT;
      tl.k = p.k_lane + ((size_t)r0 * p.Hkv + hk) * D;
      tl.v = p.v_lane + ((size_t)r0 * p.Hkv + hk) * D;
      tl.nvalid = min(AT_KT, p.B_keys - sub * AT_KT);
      tl.vis = active && ((my_vis >> j) & 1ull);
      return tl;
    }
    return tl;
  };
  auto next_kt = [&](int kt) {  // index after the tile found from kt
    for (; kt < kt1; ++kt) {
      if (kt < p.n_pre_tiles) return kt + 1;
      const int j = (kt - p.n_pre_tiles) / p.lane_key_tiles;
      if ((wg_vis >> j) & 1ull) return kt + 1;
    }
    return kt1;
  };

  // Register staging of one tile: K and V as KREG 16-byte row segments
  // each; both are stored row-major (V is transposed by the reads).
  constexpr int KREG = (AT_KT * DSEG) / AT_THREADS;
  static_assert(KREG * AT_THREADS == AT_KT * DSEG, "whole tiles per thread");
  bf16x8 kr[KREG], vr[KREG];
  auto load_tile = [&](const Tile& tl) {
#pragma unroll
    for (int i = 0; i < KREG; ++i) {
      const int seg = tid + AT_THREADS * i;
      const int krow = seg / DSEG;
      const int ds = seg - krow * DSEG;
      kr[i] = load_bf16x8(tl.k + (size_t)min(krow, tl.nvalid - 1) * p.Hkv * D + ds * 8);
    }
#pragma unroll
    for (int i = 0; i < KREG; ++i) {
      const int seg = tid + AT_THREADS * i;
      const int krow = seg / DSEG;
      const int ds = seg - krow * DSEG;
      vr[i] = load_bf16x8(tl.v + (size_t)min(krow, tl.nvalid - 1) * p.Hkv * D + ds * 8);
    }
  };
  // Rows past nvalid are zeroed here (not right after the loads, which
  // would stall on them); their scores are masked to -inf anyway.
  auto store_tile = [&](int nvalid) {
#pragma unroll
    for (int i = 0; i < KREG; ++i) {
      const int seg = tid + AT_THREADS * i;
      const int krow = seg / DSEG;
      const int ds = seg - krow * DSEG;
      const bool ok = nvalid == AT_KT || krow < nvalid;
      *reinterpret_cast<bf16x8*>(&k_s[krow * KSTR + ds * 8]) = ok ? kr[i] : zero_bf16x8();
      *reinterpret_cast<bf16x8*>(&v_s[krow * VROW + ds * 8]) = ok ? vr[i] : zero_bf16x8();
    }
  };

  // One staged tile: S^T = K Q^T, the online softmax update in log2 units,
  // then O^T += V^T P^T.  Only ragged tiles (nvalid < 64) mask; a 32-key
  // half with no valid key is skipped in both products.
  //
  // Wavefront priority: low for the two MFMA blocks, high for the softmax
  // and for the tile staging between tiles, so the SIMD's arbiter favours
  // the wavefront whose vector work the next MFMAs wait for while the other
  // wavefront's MFMAs run (graph replay, one box, two runs each: Wide lane
  // + refresh 253-254 us against 259-260 us, Long 50-51 us against 52-53;
  // no gain on the wavefront-split kernel's shapes).
  auto tile_compute = [&](int nvalid) {
    const int nsub = (nvalid + 31) >> 5;  // 32-key halves holding valid keys
    const f32x16 zero16 = {};
    f32x16 sacc[2];
    auto kfrag = [&](int kb, int ks) {
      return *reinterpret_cast<const bf16x8*>(&k_s[(kb * 32 + r32) * KSTR + ks * 16 + hh * 8]);
    };
    __builtin_amdgcn_s_setprio(0);
    if (nsub == 2) {
      // Both 32-key halves: the two accumulation chains interleave, so
      // consecutive MFMAs are independent.
      sacc[0] = zero16;
      sacc[1] = zero16;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 a0 = kfrag(0, ks), a1 = kfrag(1, ks);
        sacc[0] = mfma32x32x16(a0, qf[ks], sacc[0]);
        sacc[1] = mfma32x32x16(a1, qf[ks], sacc[1]);
      }
    } else {
      sacc[0] = zero16;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) sacc[0] = mfma32x32x16(kfrag(0, ks), qf[ks], sacc[0]);
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[1][r] = -INFINITY;
    }
    if (nvalid < AT_KT) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kb * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
          sacc[kb][r] = (key < nvalid) ? sacc[kb][r] : -INFINITY;
        }
    }
    __builtin_amdgcn_s_setprio(1);
    // The max is taken on the raw scores (the scale is positive, so
    // max-then-scale is exact); each exponent is then one FMA.
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][r]);
    mx = pair_max32(mx);
    const float m_tile = mx * p.scale_log2;
    const float m_new = m_tile > m_run + AT_RESCALE_LOG2 ? m_tile : m_run;
    const float alpha = exp2_fast(m_run - m_new);
    // P in bf16 (round-to-nearest-even, two values per conversion), packed
    // per 16-key MFMA step; the row sum adds the rounded values (bf16 dot
    // products with 1), so O / l is a convex combination of V rows.
    float rs = 0.f;
    bf16x8 pk[4];
    const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int ks2 = 0; ks2 < 4; ++ks2)
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const int r = 8 * (ks2 & 1) + e;
        bf16x2 pr;
        pr[0] = (__bf16)exp2_fast(fmaf(sacc[ks2 >> 1][r], p.scale_log2, -m_new));
        pr[1] = (__bf16)exp2_fast(fmaf(sacc[ks2 >> 1][r + 1], p.scale_log2, -m_new));
        pk[ks2][e] = pr[0];
        pk[ks2][e + 1] = pr[1];
        rs = __builtin_amdgcn_fdot2_f32_bf16(pr, one2, rs, false);
      }
    rs = pair_sum32(rs);
    l_run = l_run * alpha + rs;
    m_run = m_new;
    // Rescale O only when some row's reference max moved (otherwise alpha
    // is exactly 1 and the product would change nothing).
    if (__builtin_amdgcn_read_exec() & __ballot(alpha != 1.0f)) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
    }
    __builtin_amdgcn_s_setprio(0);
    // O^T += V^T P^T, one 16-key MFMA step at a time.  The V^T fragment
    // of lane (d, h) is keys 16 ks2 + 4h + {0..3, 8..11} at column d: two
    // transpose reads of 4 x 16 blocks of the row-major V tile.
#pragma unroll
    for (int ks2 = 0; ks2 < 4; ++ks2) {
      if ((ks2 >> 1) < nsub) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const uint16_t* va = &v_s[(16 * ks2 + 4 * hh + (lg >> 2)) * VROW + dt * 32 + 16 * (lgrp & 1) + 4 * (lg & 3)];
          const bf16x8 a = cat_bf16x4(lds_read_tr16(va), lds_read_tr16(va + 8 * VROW));
          oacc[dt] = mfma32x32x16(a, pk[ks2], oacc[dt]);
        }
      }
    }
    __builtin_amdgcn_s_setprio(1);
  };

  int kt = kt0;
  Tile cur = tile_at(kt);
  kt = next_kt(kt);
  {
    // The first tile's loads are issued unconditionally (a split with no
    // tile reads row 0 of Q instead, which always exists), so that straight
    // after them one wait covers exactly the Q fragments.  Without it the
    // compiler cannot tell at the loop header whether the Q loads are done
    // and waits for every outstanding load before the first MFMA of each
    // tile, which also waited for the next tile's prefetch.
    Tile first = cur;
    if (!first.nvalid) {
      first.k = first.v = p.q;
      first.nvalid = 1;
    }
    load_tile(first);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * KREG));
  }
  while (cur.nvalid) {
    __syncthreads();  // the previous tile is no longer read
    if (cur.nvalid == AT_KT)
      store_tile(AT_KT);
    else
      store_tile(cur.nvalid);
    __syncthreads();
    // Prefetch the next visible tile while this one is multiplied.
    const Tile nxt = tile_at(kt);
    kt = next_kt(kt);
    if (nxt.nvalid) load_tile(nxt);
    if (cur.vis) {
      tile_compute(cur.nvalid);
    }
    cur = nxt;
  }

  if (!active || r32 >= nrows) return;
  const size_t orow = (size_t)(row0 + r32) * p.Hq + hq;
  if (p.n_split == 1) {
    const float inv_l = 1.0f / l_run;
    uint16_t* op = p.o + orow * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        bf16x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(oacc[dt][rg * 4 + e] * inv_l);
        *reinterpret_cast<bf16x4*>(op + dt * 32 + 8 * rg + 4 * hh) = v4;
      }
    if (p.lse && hh == 0) p.lse[orow] = (m_run + log2f(l_run)) * AT_LN2;
  } else {
    uint16_t* po = p.part_o + ((size_t)split * p.n_rows * p.Hq + orow) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        bf16x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (__bf16)oacc[dt][rg * 4 + e];
        *reinterpret_cast<bf16x4*>(po + dt * 32 + 8 * rg + 4 * hh) = v4;
      }
    if (hh == 0) {
      float* pm = p.part_ml + ((size_t)split * p.n_rows * p.Hq + orow) * 2;
      pm[0] = m_run;
      pm[1] = l_run;
    }
  }
}

// Keys of one query tile split over the wavefronts of one workgroup.
//
// On short grids (a few lanes x a few heads) the kernel above leaves most
// SIMDs idle unless it splits the key range over workgroups, and then its
// partials cross a kernel boundary to attn_merge_kernel (written back
// from L2 at the end of the kernel, read again by the merge).  Here a
// workgroup of KW wavefronts serves one query tile (32 rows of one lane,
// one query head).  Wavefront w takes the lane's visible 32-key units w,
// w + KW, w + 2 KW, ... (prefix units first, then the visible lane blocks
// in ascending order), stages each in an LDS region of its own and keeps
// its own online-softmax state; nothing is shared between wavefronts until
// the end, so the loop has no workgroup barrier.  The KW states are then
// combined in LDS in ascending w (the same arithmetic as attn_merge_kernel)
// and the output is written once, in bf16.  Every lane's workgroups re-read
// the prefix units; workgroup ids run head-fastest, so with Hq a multiple
// of 8 all query tiles of a head land on one XCD (ids are dealt to the 8
// XCDs round-robin) and those re-reads hit that XCD's L2.
template <int D, int KW>
__global__ __launch_bounds__(KW * kWave) __attribute__((amdgpu_waves_per_eu(KW / 4, KW / 4)))
void lane_attn_wsplit_kernel(AttnParams p) {
  constexpr int KT = 32;                    // keys per unit
  constexpr int KS = D / 16;
  constexpr int DT = D / 32;
  constexpr int KSTR = D + 8;
  constexpr int VROW = D + 32;
  constexpr int DSEG = D / 8;
  constexpr int KREG = KT * DSEG / kWave;   // 16-byte K (and V) segments per lane
  constexpr int WBUF = KT * (KSTR + VROW);  // bf16 per wavefront region
  constexpr int OSTR = D + 4;               // fp32 per row of the merge area
  static_assert(KREG * kWave == KT * DSEG, "whole tiles per lane");
  static_assert((KW * 32 * OSTR + KW * 32 * 2) * 4 <= KW * WBUF * 2, "merge area inside the tile regions");
  __shared__ __attribute__((aligned(16))) uint16_t lds[KW * WBUF];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r32 = lane & 31;
  const int hh = lane >> 5;
  const int lgrp = lane >> 4;
  const int lg = lane & 15;
  uint16_t* k_s = lds + w * WBUF;
  uint16_t* v_s = k_s + KT * KSTR;

  const int hq = blockIdx.x % p.Hq;
  const int qt = blockIdx.x / p.Hq;
  const int lane_i = qt / p.tiles_per_lane;
  const int c = qt - lane_i * p.tiles_per_lane;
  const int hk = hq / p.g;
  const int row0 = lane_i * p.rows_per_lane + c * 32;
  const int nrows = min(min(32, p.rows_per_lane - c * 32), p.n_rows - row0);
  const unsigned long long vis = p.n_key_lanes ? p.vis[lane_i] : 0ull;
  const int n_pre = (p.P + KT - 1) / KT;
  const int lane_units = (p.B_keys + KT - 1) / KT;
  const int n_units = n_pre + __popcll(vis) * lane_units;

  // The query tile is the same for every wavefront: wavefront w < KS loads
  // its k-step w once and the fragments are shared through LDS (8x fewer Q
  // loads per workgroup; graph replay, one box: LLaDA 9.7 against 11.1 us,
  // Dream 14.9 against 16.6 us).
  bf16x8 qf[KS];
  __shared__ __attribute__((aligned(16))) bf16x8 q_sh[KS * kWave];
  bf16x8 qslice = zero_bf16x8();
  {
    const bool ok = r32 < nrows;
    const uint16_t* qrow = p.q + ((size_t)(row0 + (ok ? r32 : 0)) * p.Hq + hq) * D;
    if (w < KS) qslice = ok ? load_bf16x8(qrow + w * 16 + hh * 8) : zero_bf16x8();
  }
  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[dt][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  struct Unit {
    const uint16_t* k;
    const uint16_t* v;
    int nvalid;  // 0 = past the last unit
  };
  auto unit_at = [&](int u) -> Unit {
    Unit t{nullptr, nullptr, 0};
    if (u >= n_units) return t;
    int r0;
    if (u < n_pre) {
      r0 = u * KT;
      t.k = p.k_pre + ((size_t)r0 * p.Hkv + hk) * D;
      t.v = p.v_pre + ((size_t)r0 * p.Hkv + hk) * D;
      t.nvalid = min(KT, p.P - r0);
      return t;
    }
    const int lu = u - n_pre;
    int jj = lu / lane_units;
    const int sub = lu - jj * lane_units;
    unsigned long long m = vis;
    for (; jj > 0; --jj) m &= m - 1;  // drop the jj lowest visible lanes
    r0 = __builtin_ctzll(m) * p.B_keys + sub * KT;
    t.k = p.k_lane + ((size_t)r0 * p.Hkv + hk) * D;
    t.v = p.v_lane + ((size_t)r0 * p.Hkv + hk) * D;
    t.nvalid = min(KT, p.B_keys - sub * KT);
    return t;
  };

  bf16x8 kr[KREG], vr[KREG];
  auto load_unit = [&](const Unit& t) {
#pragma unroll
    for (int i = 0; i < KREG; ++i) {
      const int seg = lane + kWave * i;
      const int krow = seg / DSEG;
      const int ds = seg - krow * DSEG;
      kr[i] = load_bf16x8(t.k + (size_t)min(krow, t.nvalid - 1) * p.Hkv * D + ds * 8);
    }
#pragma unroll
    for (int i = 0; i < KREG; ++i) {
      const int seg = lane + kWave * i;
      const int krow = seg / DSEG;
      const int ds = seg - krow * DSEG;
      vr[i] = load_bf16x8(t.v + (size_t)min(krow, t.nvalid - 1) * p.Hkv * D + ds * 8);
    }
  };
  auto store_unit = [&](int nvalid) {
#pragma unroll
    for (int i = 0; i < KREG; ++i) {
      const int seg = lane + kWave * i;
      const int krow = seg / DSEG;
      const int ds = seg - krow * DSEG;
      const bool ok = nvalid == KT || krow < nvalid;
      *reinterpret_cast<bf16x8*>(&k_s[krow * KSTR + ds * 8]) = ok ? kr[i] : zero_bf16x8();
      *reinterpret_cast<bf16x8*>(&v_s[krow * VROW + ds * 8]) = ok ? vr[i] : zero_bf16x8();
    }
  };
  // S^T = K Q^T in two interleaved chains (even / odd k-steps), the online
  // softmax update in log2 units, then O^T += V^T P^T -- the arithmetic of
  // lane_attn_kernel's tile step on one 32-key half.
  auto unit_compute = [&](int nvalid) {
    f32x16 s0 = {}, s1 = {};
#pragma unroll
    for (int ks = 0; ks < KS; ks += 2) {
      s0 = mfma32x32x16(*reinterpret_cast<const bf16x8*>(&k_s[r32 * KSTR + ks * 16 + hh * 8]), qf[ks], s0);
      s1 = mfma32x32x16(*reinterpret_cast<const bf16x8*>(&k_s[r32 * KSTR + (ks + 1) * 16 + hh * 8]), qf[ks + 1], s1);
    }
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = s0[r] + s1[r];
    if (nvalid < KT) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 8 * (r >> 2) + 4 * hh + (r & 3);
        s[r] = (key < nvalid) ? s[r] : -INFINITY;
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[r]);
    mx = pair_max32(mx);
    const float m_tile = mx * p.scale_log2;
    const float m_new = m_tile > m_run + AT_RESCALE_LOG2 ? m_tile : m_run;
    const float alpha = exp2_fast(m_run - m_new);
    float rs = 0.f;
    bf16x8 pk[2];
    const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int ks2 = 0; ks2 < 2; ++ks2)
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const int r = 8 * ks2 + e;
        bf16x2 pr;
        pr[0] = (__bf16)exp2_fast(fmaf(s[r], p.scale_log2, -m_new));
        pr[1] = (__bf16)exp2_fast(fmaf(s[r + 1], p.scale_log2, -m_new));
        pk[ks2][e] = pr[0];
        pk[ks2][e + 1] = pr[1];
        rs = __builtin_amdgcn_fdot2_f32_bf16(pr, one2, rs, false);
      }
    rs = pair_sum32(rs);
    l_run = l_run * alpha + rs;
    m_run = m_new;
    if (__builtin_amdgcn_read_exec() & __ballot(alpha != 1.0f)) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
    }
#pragma unroll
    for (int ks2 = 0; ks2 < 2; ++ks2)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const uint16_t* va = &v_s[(16 * ks2 + 4 * hh + (lg >> 2)) * VROW + dt * 32 + 16 * (lgrp & 1) + 4 * (lg & 3)];
        const bf16x8 a = cat_bf16x4(lds_read_tr16(va), lds_read_tr16(va + 8 * VROW));
        oacc[dt] = mfma32x32x16(a, pk[ks2], oacc[dt]);
      }
  };

  int u = w;
  Unit cur = unit_at(u);
  {
    // Unconditional first loads and an exact wait for this wavefront's Q
    // slice, as in lane_attn_kernel (a wavefront without a unit reads Q row
    // 0); then the slices are exchanged through LDS.
    Unit first = cur;
    if (!first.nvalid) {
      first.k = first.v = p.q;
      first.nvalid = 1;
    }
    load_unit(first);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * KREG));
    if (w < KS) q_sh[w * kWave + lane] = qslice;
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = q_sh[ks * kWave + lane];
  }
  while (cur.nvalid) {
    // The region is this wavefront's own: its LDS operations complete in
    // issue order, so wavefront-scope fences (compiler ordering only)
    // separate the previous unit's reads, this unit's stores and its reads.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    store_unit(cur.nvalid);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    u += KW;
    const Unit nxt = unit_at(u);
    if (nxt.nvalid) load_unit(nxt);
    unit_compute(cur.nvalid);
    cur = nxt;
  }

  // Combine the KW states: each wavefront writes (m, l, O) to LDS, then
  // D / 8 threads per row merge 8 columns each in ascending w.
  __syncthreads();  // every wavefront is done with its tile region
  float* o_s = reinterpret_cast<float*>(lds);
  float* ml_s = o_s + KW * 32 * OSTR;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg)
      *reinterpret_cast<float4*>(&o_s[(w * 32 + r32) * OSTR + dt * 32 + 8 * rg + 4 * hh]) =
          make_float4(oacc[dt][rg * 4 + 0], oacc[dt][rg * 4 + 1], oacc[dt][rg * 4 + 2], oacc[dt][rg * 4 + 3]);
  if (hh == 0) {
    ml_s[(w * 32 + r32) * 2 + 0] = m_run;
    ml_s[(w * 32 + r32) * 2 + 1] = l_run;
  }
  __syncthreads();
  constexpr int TPR = D / 8;            // threads per row
  constexpr int RPP = KW * kWave / TPR;  // rows per pass
  const int d0 = (tid % TPR) * 8;
  for (int row = tid / TPR; row < nrows; row += RPP) {
    float mw[KW], M = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < KW; ++ww) {
      mw[ww] = ml_s[(ww * 32 + row) * 2];
      M = fmaxf(M, mw[ww]);
    }
    float Lsum = 0.f, acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
    for (int ww = 0; ww < KW; ++ww) {
      const float wgt = (mw[ww] == -INFINITY) ? 0.f : exp2_fast(mw[ww] - M);
      Lsum += ml_s[(ww * 32 + row) * 2 + 1] * wgt;
      const float4 a = *reinterpret_cast<const float4*>(&o_s[(ww * 32 + row) * OSTR + d0]);
      const float4 b = *reinterpret_cast<const float4*>(&o_s[(ww * 32 + row) * OSTR + d0 + 4]);
      acc[0] += a.x * wgt;
      acc[1] += a.y * wgt;
      acc[2] += a.z * wgt;
      acc[3] += a.w * wgt;
      acc[4] += b.x * wgt;
      acc[5] += b.y * wgt;
      acc[6] += b.z * wgt;
      acc[7] += b.w * wgt;
    }
    const float inv = 1.0f / Lsum;
    bf16x8 out;
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = (__bf16)(acc[e] * inv);
    const size_t orow = (size_t)(row0 + row) * p.Hq + hq;
    *reinterpret_cast<bf16x8*>(p.o + orow * D + d0) = out;
    if (p.lse && d0 == 0) p.lse[orow] = (M + log2f(Lsum)) * AT_LN2;
  }
}

// Combine the NS key splits of each (row, head): D / 8 lanes per (row,
// head), each taking 8 elements (16-byte loads and stores).  NS is a
// template argument so every split's loads issue at once (one memory round
// trip); the splits are summed in ascending order.
template <int D>
constexpr int merge_rows_per_block() { return 256 / (D / 8); }
template <int D, int NS>
__global__ __launch_bounds__(256) void attn_merge_kernel(const uint16_t* part_o, const float* part_ml,
                                                         int n_rowheads, uint16_t* o, float* lse) {
  constexpr int LPR = D / 8;  // lanes per (row, head)
  const int rh = blockIdx.x * merge_rows_per_block<D>() + threadIdx.x / LPR;
  const int sl = threadIdx.x % LPR;
  if (rh >= n_rowheads) return;
  float m[NS], l[NS], po[NS][8];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const float2 ml = *reinterpret_cast<const float2*>(part_ml + ((size_t)s * n_rowheads + rh) * 2);
    m[s] = ml.x;
    l[s] = ml.y;
    const bf16x8 v = load_bf16x8(part_o + ((size_t)s * n_rowheads + rh) * D + sl * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) po[s][e] = (float)v[e];
  }
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < NS; ++s) M = fmaxf(M, m[s]);
  float L = 0.f;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const float wgt = (m[s] == -INFINITY) ? 0.f : exp2_fast(m[s] - M);
    L += l[s] * wgt;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += po[s][e] * wgt;
  }
  const float inv = 1.0f / L;
  bf16x8 out;
#pragma unroll
  for (int e = 0; e < 8; ++e) out[e] = (__bf16)(acc[e] * inv);
  *reinterpret_cast<bf16x8*>(o + (size_t)rh * D + sl * 8) = out;
  if (lse && sl == 0) lse[rh] = (M + log2f(L)) * AT_LN2;
}

// Compact-refresh row rewrite: prefix[idx[r]] = ref[r] for K and V.
__global__ __launch_bounds__(256) void prefix_scatter_kernel(const int32_t* idx, int n_ref,
                                                             int row_segs, const uint16_t* k_ref,
                                                             const uint16_t* v_ref, uint16_t* k_pre,
                                                             uint16_t* v_pre) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long total = (long long)n_ref * row_segs;
  if (i >= total) return;
  const int r = (int)(i / row_segs);
  const int sgi = (int)(i - (long long)r * row_segs);
  const size_t dst = (size_t)idx[r] * row_segs + sgi;
  const size_t src = (size_t)r * row_segs + sgi;
  reinterpret_cast<i32x4*>(k_pre)[dst] = reinterpret_cast<const i32x4*>(k_ref)[src];
  reinterpret_cast<i32x4*>(v_pre)[dst] = reinterpret_cast<const i32x4*>(v_ref)[src];
}

// ------------------------------------------------------------------ host
static int choose_split(int base_wgs, int total_key_tiles) {
  // Short grids on the 8-tile kernel leave CUs idle: split the key tiles
  // until about 256 workgroups exist (one per CU at two wavefronts per
  // SIMD), keeping at least 3 key tiles per split, since each split adds
  // partials to merge.  Measured with the merge on 4-wavefront workgroups
  // (MI355X, best in [1, 16]):
  // Long 4 splits, 62.8 us (128 us unsplit); Wide 1, 277 us (the LLaDA and
  // Dream step shapes, 4 and 8 splits here, now take the wavefront-split
  // kernel).
  int s = 1;
  while (s < 16 && base_wgs * s < 256 && total_key_tiles >= 3 * (2 * s)) s *= 2;
  return s;
}

struct PassShape {
  int n_rows, rows_per_lane, tiles_per_lane, q_tiles_kv, base_wgs, n_pre_tiles, total_key_tiles;
};

static PassShape pass_shape(int n_rows, int rows_per_lane, int n_lanes, int g, int Hkv, int P,
                            int B_keys, int n_key_lanes) {
  PassShape s{};
  s.n_rows = n_rows;
  s.rows_per_lane = rows_per_lane;
  s.tiles_per_lane = (rows_per_lane + 31) / 32;
  s.q_tiles_kv = n_lanes * s.tiles_per_lane * g;
  s.base_wgs = ((s.q_tiles_kv + AT_WAVES - 1) / AT_WAVES) * Hkv;
  s.n_pre_tiles = (P + AT_KT - 1) / AT_KT;
  const int lane_key_tiles = B_keys ? (B_keys + AT_KT - 1) / AT_KT : 0;
  s.total_key_tiles = s.n_pre_tiles + n_key_lanes * lane_key_tiles;
  return s;
}

// The wavefront-split kernel when its grid fits the chip in one round (one
// workgroup per CU: 256 on MI355X) and no wavefront takes more than 8 key
// units; otherwise the 8-query-tile kernel, whose shared K/V staging wins
// on large grids and long key ranges.  Measured per call after a
// cache-evicting copy (MI355X): LLaDA step shape 16.6 us against 19.7 us,
// Dream 20.9 against 30.0; Long 56.6 against 57.0 (512 workgroups: stays),
// Wide 342 against 222, Wide's refresh rows 87 against 67.
constexpr int kWsplitWaves = 8;
static bool use_wsplit(const PassShape& s, int Hkv, int max_units) {
  return s.q_tiles_kv * Hkv <= 256 && max_units <= 8 * kWsplitWaves;
}

AttnPlan attn_plan(int L, int B, int P, int Hq, int Hkv, int D, int n_refresh) {
  AttnPlan pl{};
  const int g = Hq / Hkv;
  const int pre_units = (P + 31) / 32;
  const PassShape a = pass_shape(L * B, B, L, g, Hkv, P, B, L);
  pl.wsplit_lane = L > 0 && use_wsplit(a, Hkv, pre_units + L * ((B + 31) / 32));
  pl.n_split_lane = (L > 0 && !pl.wsplit_lane) ? choose_split(a.base_wgs, a.total_key_tiles) : 1;
  pl.ws_lane = pl.n_split_lane > 1 ? (size_t)pl.n_split_lane * L * B * Hq * (D * sizeof(uint16_t) + 2 * sizeof(float)) : 0;
  pl.wsplit_ref = false;
  pl.n_split_ref = 1;
  pl.ws_ref = 0;
  if (n_refresh > 0) {
    const int nl = (n_refresh + 31) / 32;
    const PassShape r = pass_shape(n_refresh, 32, nl, g, Hkv, P, 0, 0);
    pl.wsplit_ref = use_wsplit(r, Hkv, pre_units);
    pl.n_split_ref = pl.wsplit_ref ? 1 : choose_split(r.base_wgs, r.total_key_tiles);
    pl.ws_ref = pl.n_split_ref > 1 ? (size_t)pl.n_split_ref * n_refresh * Hq * (D * sizeof(uint16_t) + 2 * sizeof(float)) : 0;
  }
  pl.total = pl.ws_lane > pl.ws_ref ? pl.ws_lane : pl.ws_ref;
  return pl;
}

template <int D>
static hipError_t run_pass(const AttnParams& base, const PassShape& s, int n_split, void* ws,
                           hipStream_t stream) {
  AttnParams p = base;
  p.n_rows = s.n_rows;
  p.rows_per_lane = s.rows_per_lane;
  p.tiles_per_lane = s.tiles_per_lane;
  p.q_tiles_kv = s.q_tiles_kv;
  p.n_pre_tiles = s.n_pre_tiles;
  p.total_key_tiles = s.total_key_tiles;
  p.n_split = n_split;
  if (n_split > 1) {
    p.part_o = static_cast<uint16_t*>(ws);
    p.part_ml = reinterpret_cast<float*>(p.part_o + (size_t)n_split * s.n_rows * p.Hq * D);
  }
  const dim3 grid((s.q_tiles_kv + AT_WAVES - 1) / AT_WAVES, p.Hkv, n_split);
  hipLaunchKernelGGL(lane_attn_kernel<D>, grid, dim3(AT_THREADS), 0, stream, p);
  if (n_split > 1) {
    const int nrh = s.n_rows * p.Hq;
    const dim3 mgrid((nrh + merge_rows_per_block<D>() - 1) / merge_rows_per_block<D>()), mblock(256);
    switch (n_split) {  // choose_split returns a power of two <= 16
      case 2:
        hipLaunchKernelGGL((attn_merge_kernel<D, 2>), mgrid, mblock, 0, stream, p.part_o, p.part_ml, nrh, p.o, p.lse);
        break;
      case 4:
        hipLaunchKernelGGL((attn_merge_kernel<D, 4>), mgrid, mblock, 0, stream, p.part_o, p.part_ml, nrh, p.o, p.lse);
        break;
      case 8:
        hipLaunchKernelGGL((attn_merge_kernel<D, 8>), mgrid, mblock, 0, stream, p.part_o, p.part_ml, nrh, p.o, p.lse);
        break;
      case 16:
        hipLaunchKernelGGL((attn_merge_kernel<D, 16>), mgrid, mblock, 0, stream, p.part_o, p.part_ml, nrh, p.o, p.lse);
        break;
      default:
        return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

template <int D, int KW>
static hipError_t run_pass_wsplit(const AttnParams& base, const PassShape& s, hipStream_t stream) {
  AttnParams p = base;
  p.n_rows = s.n_rows;
  p.rows_per_lane = s.rows_per_lane;
  p.tiles_per_lane = s.tiles_per_lane;
  p.q_tiles_kv = s.q_tiles_kv;
  p.n_pre_tiles = s.n_pre_tiles;
  p.total_key_tiles = s.total_key_tiles;
  p.n_split = 1;
  const unsigned n_wg = (unsigned)(s.q_tiles_kv * p.Hkv);  // one per (query tile, query head)
  hipLaunchKernelGGL((lane_attn_wsplit_kernel<D, KW>), dim3(n_wg), dim3(KW * kWave), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_lane_attention(const uint16_t* q, const uint16_t* k_lane, const uint16_t* v_lane,
                                 uint16_t* k_pre, uint16_t* v_pre, const unsigned long long* vis,
                                 int L, int B, int P, int Hq, int Hkv, int D, float scale,
                                 const int32_t* refresh_idx, int n_refresh, const uint16_t* q_ref,
                                 const uint16_t* k_ref, const uint16_t* v_ref, uint16_t* o_ref,
                                 float* lse_ref, uint16_t* o, float* lse, void* ws,
                                 hipStream_t stream) {
  const int g = Hq / Hkv;
  const AttnPlan pl = attn_plan(L, B, P, Hq, Hkv, D, n_refresh);
  if (n_refresh > 0) {
    const int row_segs = Hkv * D / 8;
    const long long total = (long long)n_refresh * row_segs;
    hipLaunchKernelGGL(prefix_scatter_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
                       stream, refresh_idx, n_refresh, row_segs, k_ref, v_ref, k_pre, v_pre);
  }
  AttnParams p{};
  p.Hq = Hq;
  p.Hkv = Hkv;
  p.g = g;
  p.P = P;
  p.k_pre = k_pre;
  p.v_pre = v_pre;
  p.scale_log2 = scale * 1.4426950408889634f;

  // Lane pass.
  p.q = q;
  p.k_lane = k_lane;
  p.v_lane = v_lane;
  p.o = o;
  p.lse = lse;
  p.B_keys = B;
  p.n_key_lanes = L;
  p.lane_key_tiles = (B + AT_KT - 1) / AT_KT;
  for (int i = 0; i < L; ++i) p.vis[i] = vis[i];
  hipError_t e = hipSuccess;
  if (L > 0) {  // L = 0: refresh-only call
    const PassShape a = pass_shape(L * B, B, L, g, Hkv, P, B, L);
    if (pl.wsplit_lane)
      e = (D == 64) ? run_pass_wsplit<64, kWsplitWaves>(p, a, stream)
                    : run_pass_wsplit<128, kWsplitWaves>(p, a, stream);
    else
      e = (D == 64) ? run_pass<64>(p, a, pl.n_split_lane, ws, stream)
                    : run_pass<128>(p, a, pl.n_split_lane, ws, stream);
  }
  if (e != hipSuccess || n_refresh <= 0) return e;

  // Refresh pass: refreshed rows over the updated prefix only.
  AttnParams r = p;
  r.q = q_ref;
  r.k_lane = nullptr;
  r.v_lane = nullptr;
  r.o = o_ref;
  r.lse = lse_ref;
  r.B_keys = 0;
  r.n_key_lanes = 0;
  r.lane_key_tiles = 1;
  for (int i = 0; i < AT_MAX_LANES; ++i) r.vis[i] = 0ull;
  const int nl = (n_refresh + 31) / 32;
  const PassShape b = pass_shape(n_refresh, 32, nl, g, Hkv, P, 0, 0);
  if (pl.wsplit_ref)
    return (D == 64) ? run_pass_wsplit<64, kWsplitWaves>(r, b, stream)
                     : run_pass_wsplit<128, kWsplitWaves>(r, b, stream);
  return (D == 64) ? run_pass<64>(r, b, pl.n_split_ref, ws, stream)
                   : run_pass<128>(r, b, pl.n_split_ref, ws, stream);
}

}  // namespace al
