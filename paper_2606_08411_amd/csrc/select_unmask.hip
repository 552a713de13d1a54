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
  __shared__ float s_conf[kSelMaxPositions];
  __shared__ int s_arg[kSelMaxPositions];
  __shared__ int s_lo[kSelMaxLanes], s_hi[kSelMaxLanes], s_cnt[kSelMaxLanes], s_nsel[kSelMaxLanes];
  __shared__ int s_blen[kSelMaxLanes], s_k[kSelMaxLanes], s_role[kSelMaxLanes], s_ndraft[kSelMaxLanes];
  __shared__ int s_tlane[kSelMaxLanes];
  // Delimiter, digit, open- and close-bracket ids.
  constexpr int ID_DIGIT = kSelMaxDelims, ID_OPEN = ID_DIGIT + kSelMaxBoundaryIds;
  constexpr int ID_CLOSE = ID_OPEN + kSelMaxBoundaryIds, ID_ALL = ID_CLOSE + kSelMaxBoundaryIds;
  __shared__ int32_t s_ids[ID_ALL];
  __shared__ int s_wu[SEL_WAVES], s_ws[SEL_WAVES];

  const SelHost& h = p.h;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int L = h.L, B = h.B, N = h.N, LB = L * B;

  // Every input of the first SEL_THREADS positions / rows, the per-lane
  // limits and the id sets (kernel arguments) is loaded before anything is
  // stored, so the whole first pass costs one memory round trip (separate
  // loops would wait for each in turn); larger inputs continue below.
  {
    const bool pi = tid < LB, ri = tid < N, li = tid < L;
    const int tk = pi ? p.tokens[tid] : 0;
    const uint8_t mk = pi ? p.is_masked[tid] : 0;
    const int ps = ri ? p.row_pos[tid] : 0;
    const float cf = ri ? p.conf[tid] : 0.f;
    const int ag = ri ? p.argmax[tid] : 0;
    const int bl = li ? h.b_len[tid] : 0;
    const int kl = li ? h.k_lane[tid] : 0;
    const int rl = li ? h.role[tid] : 1;
    const int tl = li ? h.t_lane[tid] : 0;
    int id = 0;
    if (tid < ID_DIGIT) id = h.delim[tid];
    else if (tid < ID_OPEN) id = h.digit[tid - ID_DIGIT];
    else if (tid < ID_CLOSE) id = h.open[tid - ID_OPEN];
    else if (tid < ID_ALL) id = h.close[tid - ID_CLOSE];
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
      s_lo[tid] = 0;
      s_hi[tid] = 0;
      s_cnt[tid] = 0;
      s_nsel[tid] = 0;
      s_ndraft[tid] = 0;
      s_blen[tid] = bl;
      s_k[tid] = kl;
      s_role[tid] = rl;
      s_tlane[tid] = tl;
    }
    if (tid < ID_ALL) s_ids[tid] = id;
  }
  for (int i = tid + SEL_THREADS; i < LB; i += SEL_THREADS) {
    s_tok[i] = p.tokens[i];
    s_msk[i] = p.is_masked[i];
  }
  for (int n = tid + SEL_THREADS; n < N; n += SEL_THREADS) {
    s_pos[n] = p.row_pos[n];
    s_conf[n] = p.conf[n];
    s_arg[n] = p.argmax[n];
  }
  __syncthreads();

  // Candidates, lane row ranges (row_pos is ascending, so each lane's rows
  // are contiguous) and threshold passes.
  for (int n = tid; n < N; n += SEL_THREADS) {
    const int pos = s_pos[n];
    const int ln = pos / B;
    const int i = pos - ln * B;
    if (n == 0 || s_pos[n - 1] / B != ln) s_lo[ln] = n;
    if (n == N - 1 || s_pos[n + 1] / B != ln) s_hi[ln] = n + 1;
    const bool cand = i < s_blen[ln] && s_msk[pos];
    uint8_t f = cand ? SEL_CANDIDATE : 0;
    if (h.mode == 0 && cand && s_conf[n] >= h.tau) {
      f |= SEL_TRANSFER;
      atomicAdd(&s_cnt[ln], 1);
    }
    // Lookahead window of a generate lane (tau_future > 1 never passes).
    if (s_role[ln] == 0 && i >= s_blen[ln] && s_msk[pos] && s_conf[n] >= h.tau_future &&
        s_arg[n] != h.eos_id)
      f |= SEL_DRAFT;
    s_sel[n] = f;
    if (!cand) s_conf[n] = __builtin_nanf("");  // compares false in the ranking below
  }
  __syncthreads();

  // Top-k (TOPK mode) or fallback (THRESHOLD mode, lanes with no pass):
  // a candidate is chosen when fewer than k candidates of its lane come
  // first (higher confidence, or equal confidence and lower position).
  // row_pos is strictly ascending, so on equal confidence exactly the
  // lane's earlier rows come first; non-candidates hold NaN, which compares
  // false.  One LDS read per compared row, no branch.
  for (int n = tid; n < N; n += SEL_THREADS) {
    if (!(s_sel[n] & SEL_CANDIDATE)) continue;
    const int ln = s_pos[n] / B;
    const int k = (h.mode == 1) ? s_k[ln] : (s_cnt[ln] == 0 ? h.fallback_k : 0);
    if (k <= 0) continue;
    const float c = s_conf[n];
    const int lo = s_lo[ln], hi = s_hi[ln];
    int rank = 0;
#pragma unroll 8
    for (int m = lo; m < n; ++m) rank += s_conf[m] >= c;
#pragma unroll 8
    for (int m = n + 1; m < hi; ++m) rank += s_conf[m] > c;
    if (rank < k) s_sel[n] |= SEL_TRANSFER;
  }
  __syncthreads();

  // Write-back of transfers (flag 1) and drafts (flag 2).
  for (int n = tid; n < N; n += SEL_THREADS) {
    const uint8_t f = s_sel[n];
    const bool tr = f & SEL_TRANSFER;
    const bool dr = f & SEL_DRAFT;
    p.unmask_flag[n] = (uint8_t)(tr ? 1 : (dr ? 2 : 0));
    if (tr || dr) {
      const int pos = s_pos[n];
      const int tok = s_arg[n];
      p.tokens[pos] = tok;
      p.is_masked[pos] = 0;
      s_tok[pos] = tok;
      s_msk[pos] = 0;
      atomicAdd(tr ? &s_nsel[pos / B] : &s_ndraft[pos / B], 1);
    }
  }
  __syncthreads();

  // Ordered compaction of transferred / still-masked rows.
  int base_u = 0, base_s = 0;
  for (int b0 = 0; b0 < N; b0 += SEL_THREADS) {
    const int n = b0 + tid;
    const bool fu = n < N && (s_sel[n] & (SEL_TRANSFER | SEL_DRAFT));
    const bool fs = n < N && !fu && s_msk[s_pos[n]];
    const unsigned long long bu = __ballot(fu);
    const unsigned long long bs = __ballot(fs);
    const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    if (lane == 0) {
      s_wu[w] = __popcll(bu);
      s_ws[w] = __popcll(bs);
    }
    __syncthreads();
    int off_u = base_u, off_s = base_s, tot_u = 0, tot_s = 0;
    for (int ww = 0; ww < SEL_WAVES; ++ww) {
      if (ww < w) {
        off_u += s_wu[ww];
        off_s += s_ws[ww];
      }
      tot_u += s_wu[ww];
      tot_s += s_ws[ww];
    }
    if (fu) p.unmasked_pos[off_u + __popcll(bu & lt)] = s_pos[n];
    if (fs) p.still_pos[off_s + __popcll(bs & lt)] = s_pos[n];
    base_u += tot_u;
    base_s += tot_s;
    __syncthreads();
  }
  if (tid == 0) {
    p.counts[0] = base_u;
    p.counts[1] = base_s;
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
  const bool brackets = (h.n_open | h.n_close) != 0;
  for (int ln = w; ln < L; ln += SEL_WAVES) {
    const int n = s_blen[ln];
    int last = -1, filled = 0, stop = n, carry = 0;
    for (int i0 = 0; i0 < B; i0 += kWave) {
      const int i = i0 + lane;
      const int pos = ln * B + i;
      const bool in = i < n;
      const bool m = in ? s_msk[pos] != 0 : true;
      const int tk = in ? s_tok[pos] : 0;
      int depth = 0;
      if (brackets) {
        if (in && !m) depth = in_set(tk, s_ids + ID_OPEN, h.n_open) ? 1 : (in_set(tk, s_ids + ID_CLOSE, h.n_close) ? -1 : 0);
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
        isd = in_set(tk, s_ids, h.n_delim) && depth <= 0;
        if (isd && i > 0 && !s_msk[pos - 1] && in_set(s_tok[pos - 1], s_ids + ID_DIGIT, h.n_digit)) isd = false;
      }
      const unsigned long long bd = __ballot(isd);
      const unsigned long long bf = __ballot(in && !m);
      const unsigned long long bs = __ballot(in && (m || tk == h.eos_id));
      if (bd) last = i0 + 63 - __clzll((long long)bd);
      filled += __popcll(bf);
      if (bs) stop = min(stop, i0 + __ffsll((long long)bs) - 1);
      if (p.delim_flag && i < B) p.delim_flag[pos] = (uint8_t)isd;
    }
    if (lane == 0) {
      const int split = last + 1;
      const bool fork = s_role[ln] == 0 && split > 0 &&
                        (float)filled >= h.rho_min * (float)n && s_tlane[ln] >= h.t_min;
      int32_t* st = p.lane_stats + ln * 6;
      st[0] = split;
      st[1] = filled;
      st[2] = stop;
      st[3] = fork ? 1 : 0;
      st[4] = s_nsel[ln];
      st[5] = s_ndraft[ln];
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
