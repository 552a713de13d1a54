/*
 * asynclane.h -- C ABI of the AsyncLane decode-step hot path on MI355X (gfx950).
 *
 * One decode step of AsyncLane (arXiv 2606.08411) evaluates every active lane
 * of one prefix-sharing group in a single batched model call (Section 3.4,
 * "Shared-prefix lane batching"), then applies the block-wise sampler's
 * confidence-based transfer rule inside each lane's valid update region and
 * reads the lane boundary state that drives forking and advancement
 * (Section 3.2).  This library provides the data-parallel part of that step
 * as three calls:
 *
 *   lane_attn_forward   shared-prefix lane-batched bidirectional attention
 *                       (+ compact-refresh row rewrite and refresh rows)
 *   lmhead_confidence   fused hidden->vocab GEMM + online softmax: per masked
 *                       position the max probability and its token id,
 *                       without writing the logits
 *   select_unmask       per-lane threshold / top-k transfer, lookahead
 *                       drafts, write-back, ordered compaction and
 *                       boundary statistics
 *
 * Conventions shared by every call
 * --------------------------------
 * - bf16 tensors are passed as uint16_t bit patterns (al_bf16), row-major,
 *   innermost index last as written in each shape.
 * - "dev" pointers are device memory of the current HIP device; "host"
 *   pointers are read during the call only (their contents are copied into
 *   kernel arguments before the call returns).
 * - The caller owns every buffer, including workspaces; the library never
 *   allocates, frees or keeps a pointer after a call returns
 *   (lmhead_confidence_noalloc keeps its partials in a fixed device array
 *   of the library instead of a caller workspace).
 * - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *   the call returns before it completes.  Inputs must stay valid until the
 *   stream reaches that point.
 * - Return value: AL_OK (0), or a negative AL_ERR_* status.  Argument errors
 *   are detected before anything is enqueued; AL_ERR_HIP reports a failed
 *   launch (hipGetLastError after the enqueue).  Nothing is printed and no
 *   exception crosses the boundary.
 * - Preconditions that are NOT checked: finite inputs; refresh indices unique
 *   and in [0, P); row_idx values in [0, n_rows); row_pos strictly ascending
 *   and in [0, L*B); no overlap between output and input buffers unless a
 *   parameter is documented as in/out.
 */
#ifndef ASYNCLANE_H
#define ASYNCLANE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t al_bf16;

#define AL_OK 0
#define AL_ERR_NULL (-1)        /* a required pointer is NULL                     */
#define AL_ERR_SHAPE (-2)       /* a size or scalar is out of the supported range */
#define AL_ERR_TREE (-3)        /* parent[i] not in [-1, i)                        */
#define AL_ERR_WORKSPACE (-4)   /* workspace smaller than the *_workspace_size()   */
#define AL_ERR_ALIGN (-5)       /* a device pointer is not 16-byte aligned         */
#define AL_ERR_UNSUPPORTED (-6) /* valid request this build does not implement     */
#define AL_ERR_HIP (-7)         /* the HIP runtime reported a launch error         */

#define AL_ROLE_GEN 0           /* generate lane: advances the frontier          */
#define AL_ROLE_REF 1           /* refine lane: polishes a discovered prefix     */
#define AL_MODE_THRESHOLD 0     /* conf >= tau, optional top-fallback_k          */
#define AL_MODE_TOPK 1          /* the k_lane[l] most confident positions        */

#define AL_MAX_LANES 64         /* one ancestor set per lane fits a uint64       */
#define AL_MAX_DELIMS 16
#define AL_MAX_BOUNDARY_IDS 32  /* per ValidBoundary id set of select_unmask  */
#define AL_MAX_SELECT_POSITIONS 8192  /* L*B limit of select_unmask              */

/* lane_stats columns (int32 [L][AL_LANE_STATS]) */
#define AL_STAT_SPLIT 0   /* 0-indexed start of the continuation after the last
                             delimiter in [0, b_len), 0 if none (eq. split_point) */
#define AL_STAT_FILLED 1  /* filled (unmasked) positions in [0, b_len)           */
#define AL_STAT_VALID 2   /* index of the first masked or EOS position, else
                             b_len (valid prefix length, "Advancement control")   */
#define AL_STAT_FORK 3    /* 1 iff role = gen, split > 0,
                             (float)filled >= rho_min * (float)b_len (fp32) and
                             t_lane >= t_min (eq. fork_condition)                  */
#define AL_STAT_NSEL 4    /* positions of this lane transferred by this call      */
#define AL_STAT_NDRAFT 5  /* lookahead drafts written into this lane by this call */
#define AL_LANE_STATS 6

/* Human-readable name of a status code (static string, never NULL). */
const char* al_status_string(int status);

/* ------------------------------------------------------------------------
 * lane_attn_forward -- shared-prefix lane-batched bidirectional attention.
 *
 * Defined by Section 3.2 ("Lane-local denoising": a lane is evaluated on its
 * input given the cached prefix state before the lane) and Section 3.4
 * ("Shared-prefix lane batching": lanes sharing a prefix state form one
 * batched call; "Compact cache refresh and reuse": stale prefix rows are
 * recomputed).  Query row a of lane i and query head h attend, with softmax
 * scale `scale`, to the key/value rows
 *     every prefix row 0..P-1
 *   + every row of the block of each lane j that is i or an ancestor of i
 *     in the lane tree (parent links), bidirectionally inside the block.
 * Siblings and descendants are not visible.  K/V head of query head h is
 * h / (Hq/Hkv).  No bias, soft-cap or positional term is applied (rotary
 * embedding is the caller's).  Masked positions are ordinary keys.
 *
 * With n_refresh > 0 the call first rewrites prefix rows in place,
 *     k_prefix[refresh_idx[r]] = k_ref[r],  v_prefix[refresh_idx[r]] = v_ref[r],
 * then computes the lanes over the updated prefix, and computes the
 * refreshed rows' queries q_ref over all P rows of the updated prefix only.
 *
 * Compact cache refresh (Section 3.4): with L = 0 and n_refresh > 0 the call
 * only refreshes.  Passing the window [0, L_refresh) as the prefix
 * (P = L_refresh, see al_refresh_window) with refresh_idx = 0..P-1 is the
 * bidirectional refresh forward over the window.
 *
 * q        dev  [L*B][Hq][D]   lane query rows, lane-major (row = i*B + a)
 * k_lane   dev  [L*B][Hkv][D]  lane block keys (same row order)
 * v_lane   dev  [L*B][Hkv][D]
 * k_prefix dev  [P][Hkv][D]    shared cached prefix; in/out when n_refresh>0
 * v_prefix dev  [P][Hkv][D]
 * parent   host [L]            parent lane, -1 for a lane attached directly
 *                              to the prefix; parent[i] must be < i
 * L        0..AL_MAX_LANES (0 only with n_refresh > 0: q, k_lane, v_lane,
 *          parent, o, lse may then be NULL and B is ignored);
 *          B: 16..1024, multiple of 16;  P >= 0
 * Hq, Hkv  Hq % Hkv == 0, Hq/Hkv <= 16;  D: 64 or 128
 * scale    softmax scale; <= 0 selects 1/sqrt(D)
 * refresh_idx dev [n_refresh] int32, unique rows in [0, P); n_refresh >= 0
 * q_ref    dev  [n_refresh][Hq][D];  k_ref, v_ref dev [n_refresh][Hkv][D]
 * o_ref    dev  [n_refresh][Hq][D]  out;  lse_ref dev [n_refresh][Hq] fp32 out
 *          or NULL (all refresh pointers may be NULL when n_refresh == 0)
 * o        dev  [L*B][Hq][D] out (bf16, round-to-nearest-even)
 * lse      dev  [L*B][Hq] fp32 out (natural-log sum of exp of scaled
 *          scores), or NULL
 * workspace dev, >= lane_attn_workspace_size(...) bytes (may be NULL when
 *          that size is 0); contents need not be initialised
 * ------------------------------------------------------------------------ */
size_t lane_attn_workspace_size(int L, int B, int P, int Hq, int Hkv, int D, int n_refresh);

int lane_attn_forward(const al_bf16* q, const al_bf16* k_lane, const al_bf16* v_lane,
                      al_bf16* k_prefix, al_bf16* v_prefix,
                      const int32_t* parent, int L, int B, int P,
                      int Hq, int Hkv, int D, float scale,
                      const int32_t* refresh_idx, int n_refresh,
                      const al_bf16* q_ref, const al_bf16* k_ref, const al_bf16* v_ref,
                      al_bf16* o_ref, float* lse_ref,
                      al_bf16* o, float* lse,
                      void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * lmhead_confidence -- LM-head GEMM fused with an online softmax.
 *
 * Defined by Section 3.2 ("Lane-local denoising"): a lane's outputs feed the
 * block-wise sampler's confidence-based transfer rule, whose confidence is
 * the probability of the most likely token; refine lanes suppress EOS.  For
 * n in [0, N), with r = row_idx[n] (or n when row_idx is NULL):
 *     z[v]     = sum_k hidden[r][k] * W[v][k]          (fp32 accumulation)
 *     C        = [0, V) minus eos_id if suppress_eos[n] != 0
 *     argmax[n]= smallest v in C with z[v] = max_C z
 *     lse[n]   = log sum_{v in C} exp(z[v])   (natural log)
 *     conf[n]  = exp(max_C z - lse[n])
 * The logits are never written to memory.  Results are bitwise
 * reproducible from call to call (fixed reduction order, no float atomics).
 *
 * hidden   dev [n_rows][d]        bf16 hidden states
 * row_idx  dev [N] int32 or NULL  rows of `hidden` to score (masked positions)
 * N        0..n_rows (N == 0 enqueues nothing)
 * W        dev [V][d]             bf16 LM-head weight (nn.Linear layout)
 * d        multiple of 8, 8..65536;  n_rows * d < 2^31;  V: 1..2^30
 * suppress_eos dev [N] uint8 or NULL (NULL = no row suppresses EOS)
 * eos_id   in [-1, V); -1 = no EOS id.  V == 1 with eos_id == 0 and
 *          suppress_eos given is AL_ERR_SHAPE (a suppressed row would have
 *          no candidate token).
 * conf, argmax  dev [N] fp32 / int32 out;  lse dev [N] fp32 out or NULL
 * workspace dev, >= lmhead_confidence_workspace_size(N, d, V) bytes of
 *          scratch (per-vocab-tile partial maxima, sums and indices);
 *          contents need not be initialised.  Calls that share a workspace
 *          must not run concurrently.  The size depends on the compute-unit
 *          count of the current device: query it with that device current.
 * ------------------------------------------------------------------------ */
size_t lmhead_confidence_workspace_size(int N, int d, int V);

int lmhead_confidence(const al_bf16* hidden, int n_rows,
                      const int32_t* row_idx, int N,
                      const al_bf16* W, int d, int V,
                      const uint8_t* suppress_eos, int eos_id,
                      float* conf, int32_t* argmax, float* lse,
                      void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Packed LM-head weight: lmhead_pack_weight + lmhead_confidence_packed.
 *
 * The same computation as lmhead_confidence (Section 3.2), reading W from a
 * one-time repacked copy (weights do not change between decode steps, so
 * the copy is made once, e.g. at model load).  Layout: W is cut into
 * 32-row units u = v / 32 and 64-element K chunks c = k / 64; block (c, u)
 * holds 4 x 64 x 8 elements in the order the kernel's registers take them
 * (step s = (k % 64) / 16, lane l = 32 * ((k % 16) / 8) + v % 32, element
 * k % 8), and blocks are stored K-chunk-major: element offset
 *     (((c * ceil(V/32) + u) * 4 + s) * 64 + l) * 8 + k % 8.
 * Rows past V and K past d are zero.  Reading W chunk by chunk across the
 * whole vocabulary this way is a near-linear stream of HBM.
 *
 * lmhead_packed_weight_size returns the bytes of the packed copy
 * (ceil(d/64)*64 * ceil(V/32)*32 * 2), 0 for bad arguments.
 * lmhead_pack_weight: W dev [V][d] in, W_packed dev out (packed_bytes >=
 * that size, else AL_ERR_WORKSPACE); d, V as for lmhead_confidence.
 * lmhead_confidence_packed: arguments, results and errors of
 * lmhead_confidence with W_packed in place of W; the workspace size is
 * lmhead_confidence_workspace_size(N, d, V).  Results equal
 * lmhead_confidence's within rounding (the vocabulary is tiled in 32-row
 * units, so the fp32 sums are grouped and ordered differently); argmax
 * ties still go to the lowest id.
 * ------------------------------------------------------------------------ */
size_t lmhead_packed_weight_size(int d, int V);

int lmhead_pack_weight(const al_bf16* W, int d, int V, al_bf16* W_packed, size_t packed_bytes,
                       void* stream);

int lmhead_confidence_packed(const al_bf16* hidden, int n_rows,
                             const int32_t* row_idx, int N,
                             const al_bf16* W_packed, int d, int V,
                             const uint8_t* suppress_eos, int eos_id,
                             float* conf, int32_t* argmax, float* lse,
                             void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * lmhead_confidence_noalloc -- lmhead_confidence without a workspace.
 *
 * For callers that cannot allocate device memory at call time: code being
 * captured into a HIP graph, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, results and errors as lmhead_confidence
 * (bitwise the same outputs: the same kernels run), minus the workspace.
 * The per-vocab-tile partials go to a fixed device array inside the library
 * (AL_NOALLOC_SCRATCH_BYTES per GPU, held until the process ends; its
 * device address is looked up once per device on the first call).  The
 * call allocates nothing.
 *
 * Limit: lmhead_confidence_workspace_size(N, d, V) must not exceed
 * AL_NOALLOC_SCRATCH_BYTES (with 256 compute units: N <= 960 at
 * V = 126464, N <= 672 at V = 152064), else AL_ERR_WORKSPACE before
 * anything is enqueued.
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (two streams, or two host threads) race and must be serialised by
 * the caller.  Nothing in the array needs to start at zero.
 * ------------------------------------------------------------------------ */
#define AL_NOALLOC_SCRATCH_BYTES (8u << 20)

int lmhead_confidence_noalloc(const al_bf16* hidden, int n_rows,
                              const int32_t* row_idx, int N,
                              const al_bf16* W, int d, int V,
                              const uint8_t* suppress_eos, int eos_id,
                              float* conf, int32_t* argmax, float* lse, void* stream);

/* ------------------------------------------------------------------------
 * select_unmask -- per-lane transfer, lookahead drafts, write-back and
 * boundary statistics.
 *
 * Defined by Section 3.2: the transfer rule is applied to each lane's valid
 * update region [0, b_len[l]) (refine lanes: the discovered prefix); the
 * transferred positions take their argmax token and are written back; then
 * the lane's split point (eq. split_point, with the ValidBoundary id sets below),
 * fill ratio and step condition (eq. fork_condition) and valid prefix length
 * ("Advancement control") are computed on the updated state.
 *
 * Lookahead drafts ("Advancement control", eq. lane_input): positions
 * [b_len[l], B) of a generate lane are its lookahead window.  A masked
 * window row with conf >= tau_future (fp32) whose argmax is not eos_id is
 * written back as a draft.  Refine lanes never draft.  Drafting is off
 * when tau_future > 1 (conf never exceeds 1), e.g. +inf.
 *
 * Row n describes flat position row_pos[n] = lane*B + i.  A row is a
 * candidate of lane l = row_pos[n]/B when i < b_len[l] and the position is
 * masked.  Order "most confident first": conf descending, then position
 * ascending.  THRESHOLD mode selects every candidate with conf >= tau (fp32
 * compare); a lane with none selects its fallback_k most confident
 * candidates when fallback_k > 0.  TOPK mode selects the min(k_lane[l],
 * #candidates) most confident candidates of each lane.
 *
 * conf, argmax  dev [N] fp32 / int32 (from lmhead_confidence)
 * row_pos  dev [N] int32, strictly ascending in [0, L*B)
 * N        0..L*B
 * tokens   dev [L*B] int32 in/out;  is_masked dev [L*B] uint8 in/out
 * L        1..AL_MAX_LANES;  B >= 1;  L*B <= AL_MAX_SELECT_POSITIONS
 * role     host [L] uint8 AL_ROLE_*;  b_len host [L] in [0, B] or NULL (= B);
 * t_lane   host [L] local denoising steps or NULL (= 0)
 * mode     AL_MODE_THRESHOLD or AL_MODE_TOPK;  tau fp32 (not NaN)
 * fallback_k >= 0;  k_lane host [L] >= 0 (required in TOPK mode, else unused)
 * delim_ids host [n_delim] token ids, 0 <= n_delim <= AL_MAX_DELIMS
 * digit_ids, open_ids, close_ids  host [n_digit] / [n_open] / [n_close]
 *          token ids (each count 0..AL_MAX_BOUNDARY_IDS; NULL when 0) of
 *          ValidBoundary (Section 3.2, Section 4 setup): a delimiter at
 *          lane position i counts only if position i-1 is not filled with a
 *          digit id (numeric-period exclusion) and the filled positions of
 *          [0, i] hold no more open- than close-bracket ids (no split inside
 *          unclosed brackets).  Masked positions are neither.  All sets
 *          empty: every delimiter counts.
 * eos_id   token id ending the valid prefix (-1 = none)
 * rho_min, t_min  fork condition parameters
 * tau_future fp32 (not NaN): lookahead draft threshold, > 1 = off
 * unmask_flag dev [N] uint8 out: 1 row n was transferred, 2 drafted, else 0
 * unmasked_pos dev [N] int32 out: transferred and drafted positions,
 *          ascending
 * still_masked_pos dev [N] int32 out: positions of rows still masked,
 *          ascending (the next step's row list)
 * counts   dev [2] int32 out: {#unmasked_pos, #still_masked_pos}
 * lane_stats dev [L][AL_LANE_STATS] int32 out
 * delim_flag dev [L*B] uint8 out or NULL: 1 iff the position is < b_len of
 *          its lane, filled, holds a delimiter id and passes ValidBoundary
 * ------------------------------------------------------------------------ */
int select_unmask(const float* conf, const int32_t* argmax, const int32_t* row_pos, int N,
                  int32_t* tokens, uint8_t* is_masked, int L, int B,
                  const uint8_t* role, const int32_t* b_len, const int32_t* t_lane,
                  int mode, float tau, int fallback_k, const int32_t* k_lane,
                  const int32_t* delim_ids, int n_delim,
                  const int32_t* digit_ids, int n_digit, const int32_t* open_ids, int n_open,
                  const int32_t* close_ids, int n_close, int eos_id,
                  float rho_min, int t_min, float tau_future,
                  uint8_t* unmask_flag, int32_t* unmasked_pos, int32_t* still_masked_pos,
                  int32_t* counts, int32_t* lane_stats, uint8_t* delim_flag,
                  void* stream);

/* ------------------------------------------------------------------------
 * al_refresh_window -- length of the compact cache refresh window.
 *
 * Defined by Section 3.4 ("Compact cache refresh and reuse"):
 *     L_refresh = min(P + L_gen, P + L_eff + margin),
 *     L_eff = max over lanes of (lane_start[i] + valid_len[i])   (0 if none)
 * P is the prompt length, L_gen the generation length, lane_start the
 * lanes' starts and valid_len their valid prefix lengths (the
 * AL_STAT_VALID column of select_unmask) in generation coordinates.
 *
 * lane_start, valid_len  host [n_lanes] int32 (>= 0), read during the call
 * Returns L_refresh (>= 0) or a negative status: AL_ERR_SHAPE for a
 * negative argument or a result above INT32_MAX, AL_ERR_NULL for missing
 * arrays.  Host computation only; no device work.
 * ------------------------------------------------------------------------ */
int al_refresh_window(int P, int L_gen, const int32_t* lane_start, const int32_t* valid_len,
                      int n_lanes, int margin);

/* ------------------------------------------------------------------------
 * Active-lane scheduler (host) -- Section 3.3, the paper's active-lane
 * decoding algorithm, with the fork operator (eq. fork_operator), the
 * fork condition (eq. fork_condition, via select_unmask's lane_stats),
 * cascading termination ("Advancement control"), output reconstruction and
 * model-call NFE accounting (Section 3.4).
 *
 * Generation positions are 0..L_gen-1.  A lane has a role, a start s and a
 * length b (its update region [s, s+b)); its block for select_unmask is the
 * W = B + window positions [s, s+W) (region plus lookahead window; positions
 * past L_gen are filled with pad_id).  One iteration:
 *   n = al_sched_plan(...)            active lanes, depth-first, refine
 *                                     children before generate children,
 *                                     at most max_lanes
 *   al_sched_blocks(...)              their [n][W] token / mask blocks
 *   lane_attn_forward per group       (call_parent gives the in-call lane
 *                                     tree), lmhead_confidence on the
 *                                     masked rows, select_unmask with
 *                                     L = n, B = W, b_len, role, t_lane =
 *                                     t_step
 *   al_sched_commit(...)              write-back (regions first, then
 *                                     drafts into still-masked positions)
 *                                     and transitions: a generate lane
 *                                     with fork_ok forks at p = split into
 *                                     refine (s, p) and generate (s+p,
 *                                     min(B, L-s-p)) sharing a new group;
 *                                     otherwise a filled lane completes and
 *                                     a completed generate lane stops when
 *                                     v = 0 or s+v >= L, else spawns a
 *                                     generate successor at s+v (new group)
 * NFE = 1 + sum over iterations of the number of groups evaluated.
 *
 * The scheduler object owns host memory only (created by al_sched_create,
 * released by al_sched_destroy); every array argument is caller-owned host
 * memory read or written during the call.  Not thread-safe per object.
 * Errors: AL_ERR_NULL, AL_ERR_SHAPE (capacity too small, bad arguments).
 * ------------------------------------------------------------------------ */
typedef struct al_sched al_sched;

/* NULL on bad arguments (P >= 0, L_gen >= 1, B >= 1, window >= 0,
 * 1 <= max_lanes <= AL_MAX_LANES) or allocation failure. */
al_sched* al_sched_create(int P, int L_gen, int B, int window, int max_lanes, int pad_id);
void al_sched_destroy(al_sched* s);
/* Next plan: returns n (0 = no active lane).  Per lane k < n: lane id,
 * role (AL_ROLE_*), start, b_len, t_step (local steps including this one),
 * group (prefix-state id) and call_parent (index in this plan of the lane
 * whose block lane k sees -- its refine sibling -- or -1). */
int al_sched_plan(al_sched* s, int32_t* lane_id, uint8_t* role, int32_t* start, int32_t* b_len,
                  int32_t* t_step, int32_t* group, int32_t* call_parent, int cap);
/* Blocks of the last plan: tokens [n][W] int32, masked [n][W] uint8. */
int al_sched_blocks(const al_sched* s, int32_t* tokens, uint8_t* masked);
/* Results of the last plan: blocks after select_unmask and its lane_stats
 * [n][AL_LANE_STATS].  Returns the number of active lanes afterwards, or
 * AL_ERR_SHAPE (state unchanged) when a lane's split, filled count or
 * valid length lies outside [0, b_len] or a fork has split 0. */
int al_sched_commit(al_sched* s, const int32_t* tokens, const uint8_t* masked,
                    const int32_t* lane_stats);
/* Output reconstruction into out [cap]; returns its length. */
int al_sched_collect(const al_sched* s, int eos_id, int32_t* out, int cap);
/* out [6]: iterations, nfe, forks, spawns, stops, lanes created. */
int al_sched_counters(const al_sched* s, int32_t* out);
/* Lane tree, lanes in creation order: role, start, length, parent (-1 for
 * the root), kind (0 open/leaf, 1 forked, 2 spawned a successor) and v
 * (valid length at spawn, else -1).  Returns the lane count. */
int al_sched_tree(const al_sched* s, uint8_t* role, int32_t* start, int32_t* length,
                  int32_t* parent, int32_t* kind, int32_t* v, int cap);
/* Global generation state: tokens [L_gen] int32, masked [L_gen] uint8. */
int al_sched_state(const al_sched* s, int32_t* tokens, uint8_t* masked);

#ifdef __cplusplus
}
#endif
#endif /* ASYNCLANE_H */
