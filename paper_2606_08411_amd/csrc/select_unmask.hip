// Per-lane transfer selection, lookahead drafts, write-back, ordered
// compaction and lane boundary statistics for gfx950 -- one workgroup of 16
// wavefronts.
//
// Paper Section 3.2: each lane applies the block-wise sampler's confidence
// rule inside its valid update region [0, b_len); transferred positions take
// their argmax token and are written back; masked positions of a generate
// lane's lookahead window [b_len, B) whose confidence reaches tau_future
// and whose prediction is not EOS are written back as drafts ("Advancement
// control", eq. lane_input); the lane's split point (eq. split_point), fill
// ratio and step condition (eq. fork_condition) and valid prefix length
// ("Advancement control") are read on the updated state.
//
// The whole step touches a few KB, so it is latency-bound: one workgroup
// reads every input once into LDS (one memory latency instead of one per
// phase or per loop iteration), ranks top-k candidates by comparison
// counting (ties: lower position first), compacts the unmasked /
// still-masked row lists in order with wavefront ballots, and reads each
// lane's statistics off wavefront ballots.
#include "common.h"
#include "launch.h"

namespace al {

constexpr int SEL_THREADS = 1024;
constexpr int SEL_WAVES = SEL_THREADS / kWave;

struct SelParams {
  SelHost h;
  const float* conf;
  const int32_t* argmax;
  const int32_t* row_pos;
  int32_t* tokens;
  uint8_t* is_masked;
  uint8_t* unmask_flag;
  int32_t* unmasked_pos;
  int32_t* still_pos;
  int32_t* counts;
  int32_t* lane_stats;
  uint8_t* delim_flag;
};

// Per-row selection bits in LDS.
constexpr uint8_t SEL_TRANSFER = 1;   // chosen by the transfer rule
constexpr uint8_t SEL_CANDIDATE = 2;  // masked, inside [0, b_len)
constexpr uint8_t SEL_DRAFT = 4;      // lookahead draft

__global__ __launch_bounds__(SEL_THREADS) void select_unmask_kernel(SelParams p) {
  __shared__ int s_tok[kSelMaxPositions];
  __shared__ uint8_t s_msk[kSelMaxPositions];
  __shared__ uint8_t s_sel[kSelMaxPositions];  // SEL_* bits
  __shared__ int s_pos[kSelMaxPositions];      // row_pos
  __shared__ __attribute__((aligned(16))) float s_conf[kSelMaxPositions];
  __shared__ int s_arg[kSelMaxPositions];
  __shared__ int s_lo[kSelMaxLanes], s_hi[kSelMaxLanes], s_cnt[kSelMaxLanes], s_nsel[kSelMaxLanes];
  __shared__ int s_blen[kSelMaxLanes], s_k[kSelMaxLanes], s_role[kSelMaxLanes], s_ndraft[kSelMaxLanes];
  __shared__ int s_tlane[kSelMaxLanes];
  // Delimiter, digit, open- and close-bracket ids.
  constexpr int ID_DIGIT = kSelMaxDelims, ID_OPEN = ID_DIGIT + kSelMaxBoundaryIds;
  constexpr int ID_CLOSE = ID_OPEN + kSelMaxBoundaryIds, ID_ALL = ID_CLOSE + kSelMaxBoundaryIds;
  __shared__ int32_t s_ids[ID_ALL];
  constexpr int SEL_PASSES = kSelMaxPositions / SEL_THREADS;
  __shared__ int s_wu[SEL_PASSES][SEL_WAVES], s_ws[SEL_PASSES][SEL_WAVES];

  const SelHost& h = p.h;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  // Every scalar argument is fetched here in one batch: left to the
  // compiler, each would be loaded at its first use, a separate round trip
  // to the argument buffer inside later phases.
  const int L = h.L, B = h.B, N = h.N, mode = h.mode, fallback_k = h.fallback_k;
  const int eos_id = h.eos_id, t_min = h.t_min, n_delim = h.n_delim;
  const int n_digit = h.n_digit, n_open = h.n_open, n_close = h.n_close;
  const float tau = h.tau, rho_min = h.rho_min, tau_future = h.tau_future;
  int delim[kSelMaxDelims];  // the delimiter ids (scalar registers); entries past n_delim unused
#pragma unroll
  for (int j = 0; j < kSelMaxDelims; ++j) delim[j] = h.delim[j];
  int32_t* const tokens = p.tokens;
  uint8_t* const is_masked = p.is_masked;
  const int32_t* const row_pos = p.row_pos;
  const float* const conf = p.conf;
  const int32_t* const argmax = p.argmax;
  uint8_t* const unmask_flag = p.unmask_flag;
  int32_t* const unmasked_pos = p.unmasked_pos;
  int32_t* const still_pos = p.still_pos;
  int32_t* const counts = p.counts;
  int32_t* const lane_stats = p.lane_stats;
  uint8_t* const delim_flag = p.delim_flag;
  asm volatile("" ::"s"(L), "s"(B), "s"(N), "s"(mode), "s"(fallback_k), "s"(eos_id), "s"(t_min),
               "s"(n_delim), "s"(n_digit), "s"(n_open), "s"(n_close), "s"(tau), "s"(rho_min),
               "s"(tau_future), "s"(tokens), "s"(is_masked), "s"(row_pos), "s"(conf), "s"(argmax));
  asm volatile("" ::"s"(unmask_flag), "s"(unmasked_pos), "s"(still_pos), "s"(counts),
               "s"(lane_stats), "s"(delim_flag));
  const int LB = L * B;

  // Every input of the first SEL_THREADS positions / rows, the per-lane
  // limits and the id sets (kernel arguments) is loaded before anything is
  // used, without branches (indices clamped into range; with N = 0 the row
  // arrays may be absent and the token buffer, which is never empty, stands
  // in), so the whole first pass costs one memory round trip; larger inputs
  // continue below.
  {
    const bool pi = tid < LB, ri = tid < N;
    const int ip = min(tid, LB - 1);
    const int ir = min(tid, max(N - 1, 0));
    const int il = min(tid, kSelMaxLanes - 1);
    const int32_t* rp_src = N ? row_pos : tokens;
    const float* cf_src = N ? conf : reinterpret_cast<const float*>(tokens);
    const int32_t* ag_src = N ? argmax : tokens;
    const int tk = tokens[ip];
    const uint8_t mk = is_masked[ip];
    const int ps = rp_src[ir];
    const float cf = cf_src[ir];
    const int ag = ag_src[ir];
    const int bl = h.b_len[il];
    const int kl = h.k_lane[il];
    const int rl = h.role[il];
    const int tl = h.t_lane[il];
    const int32_t* idp = tid < ID_DIGIT  ? h.delim + tid
                         : tid < ID_OPEN  ? h.digit + (tid - ID_DIGIT)
                         : tid < ID_CLOSE ? h.open + (tid - ID_OPEN)
                         : tid < ID_ALL   ? h.close + (tid - ID_CLOSE)
                                          : h.delim;
    const int id = *idp;
    if (pi) {
      s_tok[tid] = tk;
      s_msk[tid] = mk;
    }
    if (ri) {
      s_pos[tid] = ps;
      s_conf[tid] = cf;
      s_arg[tid] = ag;
    }
    if (tid < kSelMaxLanes) {
      const bool li = tid < L;
      s_lo[tid] = 0;
      s_hi[tid] = 0;
      s_cnt[tid] = 0;
      s_nsel[tid] = 0;
      s_ndraft[tid] = 0;
      s_blen[tid] = li ? bl : 0;
      s_k[tid] = li ? kl : 0;
      s_role[tid] = li ? rl : 1;
      s_tlane[tid] = li ? tl : 0;
    }
    if (tid < ID_ALL) s_ids[tid] = id;
  }
  for (int i = tid + SEL_THREADS; i < LB; i += SEL_THREADS) {
    s_tok[i] = tokens[i];
    s_msk[i] = is_masked[i];
  }
  for (int n = tid + SEL_THREADS; n < N; n += SEL_THREADS) {
    s_pos[n] = row_pos[n];
    s_conf[n] = conf[n];
    s_arg[n] = argmax[n];
  }
  // Every load has landed by now in the wavefronts that store them; the
  // explicit wait also retires the loads of wavefronts that had nothing to
  // store, which the compiler would otherwise keep pending and wait for at
  // a later reuse of their registers -- after the write-back's stores,
  // which the same counter then includes.
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  __syncthreads();

  // Candidates, lane row ranges (row_pos is ascending, so each lane's rows
  // are contiguous) and threshold passes.  The reads of a row are issued
  // together: its position, its neighbours' positions, then the lane's
  // limits and the row's state.
  for (int n = tid; n < N; n += SEL_THREADS) {
    const int pos = s_pos[n];
    const int prev = s_pos[max(n - 1, 0)];
    const int next = s_pos[min(n + 1, N - 1)];
    const float c = s_conf[n];
    const int ag = s_arg[n];
    const int ln = pos / B;
    const int i = pos - ln * B;
    const bool msk = s_msk[pos] != 0;
    const int blen = s_blen[ln];
    const bool gen = s_role[ln] == 0;
    if (n == 0 || prev / B != ln) s_lo[ln] = n;
    if (n == N - 1 || next / B != ln) s_hi[ln] = n + 1;
    const bool cand = i < blen && msk;
    uint8_t f = cand ? SEL_CANDIDATE : 0;
    if (mode == 0 && cand && c >= tau) {
      f |= SEL_TRANSFER;
      atomicAdd(&s_cnt[ln], 1);
    }
    // Lookahead window of a generate lane (tau_future > 1 never passes).
    if (gen && i >= blen && msk && c >= tau_future && ag != eos_id) f |= SEL_DRAFT;
    s_sel[n] = f;
    if (!cand) s_conf[n] = __builtin_nanf("");  // compares false in the ranking below
  }
  __syncthreads();

  // Top-k (TOPK mode) or fallback (THRESHOLD mode, lanes with no pass),
  // write-back and the compaction counts, in one pass over the rows.
  //
  // A candidate is chosen when fewer than k candidates of its lane come
  // first (higher confidence, or equal confidence and lower position).
  // row_pos is strictly ascending, so on equal confidence exactly the
  // lane's earlier rows come first; non-candidates hold NaN, which compares
  // false.  tpr threads share a row (as many as fit when N is small): each
  // reads every tpr-th 16-byte block of the lane's rows (blocks aligned, so
  // entries outside [lo, hi) are masked) and the counts are summed over the
  // group with butterfly shuffles, every lane of the wavefront taking part.
  //
  // The group's first thread (the leader) then writes the row back:
  // transfers (flag 1) and drafts (flag 2) take their argmax token; it
  // records the final flags and contributes the row to its wavefront's
  // ballots of transferred / still-masked rows (a still-masked row's mask
  // bit is not changed by the write-back, so both are known here).
  const int tpr = N <= 64 ? 16 : N <= 128 ? 8 : N <= 256 ? 4 : N <= 512 ? 2 : 1;
  const int rpp = SEL_THREADS / tpr;  // rows per pass (at most SEL_PASSES passes)
  const int sub = tid & (tpr - 1);
  for (int n0 = 0, ps = 0; n0 < N; n0 += rpp, ++ps) {
    const int n = n0 + tid / tpr;
    const bool valid = n < N;
    const int nn = valid ? n : 0;
    const uint8_t sel = s_sel[nn];
    const int pos = s_pos[nn];
    const float c = s_conf[nn];
    const int tok = s_arg[nn];
    const bool msk = s_msk[pos] != 0;
    const int ln = pos / B;
    const int k = (mode == 1) ? s_k[ln] : (s_cnt[ln] == 0 ? fallback_k : 0);
    const int lo = s_lo[ln], hi = s_hi[ln];
    const bool act = valid && (sel & SEL_CANDIDATE) && k > 0;
    int rank = 0;
    if (act) {
      for (int m0 = (lo & ~3) + 4 * sub; m0 < hi; m0 += 4 * tpr) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(&s_conf[m0]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = m0 + e;
          const bool in = m >= lo && m < hi;
          const bool ahead = m < n ? v[e] >= c : v[e] > c;
          rank += (in && ahead) ? 1 : 0;
        }
      }
    }
    for (int o = tpr >> 1; o > 0; o >>= 1) rank += __shfl_xor(rank, o, kWave);
    const bool lead = valid && sub == 0;
    const bool tr = lead && ((sel & SEL_TRANSFER) || (act && rank < k));
    const bool dr = lead && (sel & SEL_DRAFT);  // drafts lie outside [0, b_len): never transfers
    const bool fs = lead && !(tr || dr) && msk;
    if (lead) {
      unmask_flag[n] = (uint8_t)(tr ? 1 : (dr ? 2 : 0));
      s_sel[n] = sel | (tr ? SEL_TRANSFER : 0);
    }
    if (tr || dr) {
      tokens[pos] = tok;
      is_masked[pos] = 0;
      s_tok[pos] = tok;
      s_msk[pos] = 0;
      atomicAdd(tr ? &s_nsel[ln] : &s_ndraft[ln], 1);
    }
    const unsigned long long bu = __ballot(tr || dr);
    const unsigned long long bs = __ballot(fs);
    if (lane == 0) {
      s_wu[ps][w] = __popcll(bu);
      s_ws[ps][w] = __popcll(bs);
    }
  }
  __syncthreads();

  // Ordered compaction: a row's slot is the count of flagged rows in
  // earlier passes and wavefronts plus its rank in its own wavefront's
  // ballot (leaders only).  No barrier follows: nothing below writes LDS.
  // Wavefronts with no row in a pass skip it, so the last wavefronts,
  // which hold no rows unless N is large, start the lane statistics below
  // at once.
  {
    const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int tot_u = 0, tot_s = 0;
    for (int n0 = 0, ps = 0; n0 < N; n0 += rpp, ++ps) {
      if (n0 + w * (kWave / tpr) >= N) break;  // wavefront-uniform; later passes have no rows either
      const int n = n0 + tid / tpr;
      const bool lead = n < N && sub == 0;
      const int nn = n < N ? n : 0;
      const uint8_t f = s_sel[nn];
      const int pos = s_pos[nn];
      const bool fu = lead && (f & (SEL_TRANSFER | SEL_DRAFT));
      const bool fs = lead && !fu && s_msk[pos] != 0;
      const unsigned long long bu = __ballot(fu);
      const unsigned long long bs = __ballot(fs);
      int off_u = tot_u, off_s = tot_s;
#pragma unroll
      for (int ww = 0; ww < SEL_WAVES; ++ww) {
        const int cu = s_wu[ps][ww], cs = s_ws[ps][ww];
        off_u += ww < w ? cu : 0;
        off_s += ww < w ? cs : 0;
        tot_u += cu;
        tot_s += cs;
      }
      if (fu) unmasked_pos[off_u + __popcll(bu & lt)] = pos;
      if (fs) still_pos[off_s + __popcll(bs & lt)] = pos;
    }
    if (tid == 0) {
      // Wavefront 0 holds rows whenever N > 0 and so visits every pass.
      counts[0] = tot_u;
      counts[1] = tot_s;
    }
  }

  // Lane boundary statistics on the updated state: one wavefront per lane,
  // 64 positions per pass.  The last delimiter, the filled count and the
  // first masked / EOS position come from wavefront ballots (uniform
  // results, no shuffle reductions).  ValidBoundary: the bracket depth of
  // [0, i] is an inclusive wavefront prefix sum plus the depth carried
  // from earlier passes (only when bracket ids are given); the
  // numeric-period test reads position i-1.
  auto in_set = [](int tk, const int32_t* set, int n) {
    bool hit = false;
    for (int j = 0; j < n; ++j) hit |= (tk == set[j]);
    return hit;
  };
  const bool brackets = (n_open | n_close) != 0;
  for (int ln = SEL_WAVES - 1 - w; ln < L; ln += SEL_WAVES) {   // last wavefront first
    const int n = s_blen[ln];
    const bool gen = s_role[ln] == 0;
    const int t_ln = s_tlane[ln], nsel = s_nsel[ln], ndraft = s_ndraft[ln];
    int last = -1, filled = 0, stop = n, carry = 0;
    for (int i0 = 0; i0 < B; i0 += kWave) {
      const int i = i0 + lane;
      const int pos = ln * B + i;
      const bool in = i < n;
      // This position and the previous one, read together (clamped into
      // the lane's block; values outside [0, n) are not used).
      const int pc = ln * B + min(i, B - 1);
      const int pp = ln * B + max(min(i, B - 1) - 1, 0);
      const bool m = in ? s_msk[pc] != 0 : true;
      const int tk = s_tok[pc];
      const bool m_prev = s_msk[pp] != 0;
      const int tk_prev = s_tok[pp];
      int depth = 0;
      if (brackets) {
        if (in && !m) depth = in_set(tk, s_ids + ID_OPEN, n_open) ? 1 : (in_set(tk, s_ids + ID_CLOSE, n_close) ? -1 : 0);
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
          const int v = __shfl_up(depth, o, kWave);
          if (lane >= o) depth += v;
        }
        depth += carry;
        carry = __shfl(depth, kWave - 1, kWave);
      }
      bool isd = false;
      if (in && !m) {
        bool hit = false;
#pragma unroll
        for (int j = 0; j < kSelMaxDelims; ++j) hit |= j < n_delim && tk == delim[j];
        isd = hit && depth <= 0;
        if (isd && i > 0 && !m_prev && in_set(tk_prev, s_ids + ID_DIGIT, n_digit)) isd = false;
      }
      const unsigned long long bd = __ballot(isd);
      const unsigned long long bf = __ballot(in && !m);
      const unsigned long long bs = __ballot(in && (m || tk == eos_id));
      if (bd) last = i0 + 63 - __clzll((long long)bd);
      filled += __popcll(bf);
      if (bs) stop = min(stop, i0 + __ffsll((long long)bs) - 1);
      if (delim_flag && i < B) delim_flag[pos] = (uint8_t)isd;
    }
    if (lane == 0) {
      const int split = last + 1;
      const bool fork = gen && split > 0 && (float)filled >= rho_min * (float)n && t_ln >= t_min;
      int32_t* st = lane_stats + ln * 6;
      st[0] = split;
      st[1] = filled;
      st[2] = stop;
      st[3] = fork ? 1 : 0;
      st[4] = nsel;
      st[5] = ndraft;
    }
  }
}

hipError_t launch_select(const SelHost& h, const float* conf, const int32_t* argmax,
                         const int32_t* row_pos, int32_t* tokens, uint8_t* is_masked,
                         uint8_t* unmask_flag, int32_t* unmasked_pos, int32_t* still_pos,
                         int32_t* counts, int32_t* lane_stats, uint8_t* delim_flag,
                         hipStream_t stream) {
  SelParams p;
  p.h = h;
  p.conf = conf;
  p.argmax = argmax;
  p.row_pos = row_pos;
  p.tokens = tokens;
  p.is_masked = is_masked;
  p.unmask_flag = unmask_flag;
  p.unmasked_pos = unmasked_pos;
  p.still_pos = still_pos;
  p.counts = counts;
  p.lane_stats = lane_stats;
  p.delim_flag = delim_flag;
  hipLaunchKernelGGL(select_unmask_kernel, dim3(1), dim3(SEL_THREADS), 0, stream, p);
  return hipGetLastError();
}

}  // namespace al
