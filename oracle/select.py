"""fp64/fp32 oracle: per-lane unmasking and lane boundary statistics.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Transfer rule (paper Section 3.2, "Lane-local denoising"): a lane is updated
with the block-wise sampler's confidence-based transfer rule, restricted to
its valid update region (positions [0, b_len) of the lane; refine lanes
suppress EOS, which is handled by the LM head).  Two modes:

* THRESHOLD: transfer every eligible masked position whose confidence is at
  least tau; if none passes and fallback_k > 0, transfer the fallback_k most
  confident eligible positions (so every lane makes progress).
* TOPK: transfer the k_lane[l] most confident eligible positions.

Order for "most confident": confidence descending, then position ascending.
Transferred positions take the argmax token and become unmasked.

Boundary statistics per lane on the updated state (0-indexed positions
i < b_len; delimiters and EOS as in Section 3.2):

* delim_i   = position i is filled, holds a delimiter id and passes
              ValidBoundary on the prefix [0, i]
* split     = 1 + the last i with delim_i, or 0 when there is none
              (eq. split_point: the 0-indexed start of the continuation
              lane)
* n_filled  = number of filled positions (eq. fork_condition's numerator)
* valid_len = the first i that is masked or holds EOS, or b_len if none
              (the valid prefix length of "Advancement control")
* fork_ok   = generate lane, split > 0, n_filled >= rho_min * b_len and
              t_lane >= t_min (eq. fork_condition); the product is formed
              in fp32.
* n_sel     = number of positions of the lane transferred by this call.
* n_draft   = number of lookahead drafts written into the lane this call.

Lookahead drafts (Section 3.2, "Advancement control", and eq. lane_input):
the input of a generate lane is its state followed by an optional lookahead
window; only the first b_len logits drive the transfer rule.  Here a lane
block holds B positions, so the window is positions [b_len, B).  A masked
window position of a generate lane whose confidence reaches tau_future and
whose predicted token is not EOS takes that token as a draft (unmask_flag
2; it becomes unmasked and is listed in unmasked_pos).  Refine lanes never
draft.  tau_future None (or above 1, since conf <= 1) disables drafting.
The paper gives no value for tau_future.

ValidBoundary (Section 3.2; the experimental setup of Section 4): the
paper names numeric-period exclusion for the math tasks and no split inside
unclosed brackets for code, as predicates of the prefix z_{1:i}.  Read here
with token-id sets (empty sets: always valid):

* numeric period: invalid when position i-1 is filled with a digit id;
* bracket balance: invalid when the filled positions of [0, i] hold more
  open-bracket ids than close-bracket ids.

Decisions that compare floating point values (threshold, ordering, fill
ratio) are taken in fp32, the precision the device kernel uses.
"""
import numpy as np

ROLE_GEN = 0
ROLE_REF = 1
MODE_THRESHOLD = 0
MODE_TOPK = 1

STAT_SPLIT, STAT_FILLED, STAT_VALID, STAT_FORK, STAT_NSEL, STAT_NDRAFT = range(6)
N_STATS = 6


def valid_boundary(tokens, is_masked, start, i, digit_ids=(), open_ids=(), close_ids=()):
    """ValidBoundary of the delimiter at lane position i, whose lane block
    starts at flat position start: a predicate of the prefix [0, i]."""
    if i > 0 and not is_masked[start + i - 1] and int(tokens[start + i - 1]) in set(digit_ids):
        return False
    depth = 0
    for j in range(i + 1):
        if is_masked[start + j]:
            continue
        t = int(tokens[start + j])
        if t in set(open_ids):
            depth += 1
        elif t in set(close_ids):
            depth -= 1
    return depth <= 0


def lane_boundary_stats(tokens, is_masked, B, role, b_len, t_lane, delim_ids,
                        eos_id, rho_min, t_min, digit_ids=(), open_ids=(), close_ids=()):
    """Returns (lane_stats [L][6] int32, delim_flag [L*B] uint8); the
    n_sel and n_draft columns are left at zero here."""
    L = len(role)
    stats = np.zeros((L, N_STATS), dtype=np.int32)
    dflag = np.zeros(L * B, dtype=np.uint8)
    dset = set(int(x) for x in delim_ids)
    for lane in range(L):
        n = int(b_len[lane])
        split = 0
        filled = 0
        valid = n
        for i in range(n):
            pos = lane * B + i
            masked = bool(is_masked[pos])
            tok = int(tokens[pos])
            if not masked:
                filled += 1
                if tok in dset and valid_boundary(tokens, is_masked, lane * B, i,
                                                  digit_ids, open_ids, close_ids):
                    dflag[pos] = 1
                    split = i + 1
            if valid == n and (masked or tok == eos_id):
                valid = i
        ratio_ok = np.float32(filled) >= np.float32(rho_min) * np.float32(n)
        fork = (int(role[lane]) == ROLE_GEN and split > 0 and bool(ratio_ok)
                and int(t_lane[lane]) >= int(t_min))
        stats[lane, STAT_SPLIT] = split
        stats[lane, STAT_FILLED] = filled
        stats[lane, STAT_VALID] = valid
        stats[lane, STAT_FORK] = int(fork)
    return stats, dflag


def select_unmask(conf, argmax, row_pos, tokens, is_masked, B, role, b_len, t_lane,
                  mode, tau, fallback_k=0, k_lane=None, delim_ids=(0, 1), eos_id=2,
                  rho_min=0.5, t_min=2, tau_future=None, digit_ids=(), open_ids=(),
                  close_ids=()):
    """Per-lane transfer on the rows row_pos (flat positions lane*B + i,
    ascending), lookahead drafts, then the boundary statistics.

    Returns dict(tokens, is_masked, unmask_flag [N] u8 (1 transfer,
    2 draft), unmasked_pos, still_masked_pos, counts [2], lane_stats [L][6],
    delim_flag [L*B])."""
    conf32 = np.asarray(conf, dtype=np.float32)
    tau32 = np.float32(tau)
    row_pos = np.asarray(row_pos, dtype=np.int64)
    tokens = np.array(tokens, dtype=np.int32, copy=True)
    is_masked = np.array(is_masked, dtype=np.uint8, copy=True)
    L = len(role)
    N = len(row_pos)
    flag = np.zeros(N, dtype=np.uint8)
    for lane in range(L):
        cand = [n for n in range(N)
                if row_pos[n] // B == lane and row_pos[n] % B < b_len[lane]
                and is_masked[row_pos[n]]]
        order = sorted(cand, key=lambda n: (-float(conf32[n]), int(row_pos[n])))
        if mode == MODE_THRESHOLD:
            chosen = [n for n in cand if conf32[n] >= tau32]
            if not chosen and fallback_k > 0:
                chosen = order[:fallback_k]
        elif mode == MODE_TOPK:
            chosen = order[:max(0, min(int(k_lane[lane]), len(cand)))]
        else:
            raise ValueError(mode)
        for n in chosen:
            flag[n] = 1
    if tau_future is not None:
        tf32 = np.float32(tau_future)
        for n in range(N):
            pos = int(row_pos[n])
            lane, i = pos // B, pos % B
            if (int(role[lane]) == ROLE_GEN and i >= int(b_len[lane]) and is_masked[pos]
                    and conf32[n] >= tf32 and int(argmax[n]) != int(eos_id)):
                flag[n] = 2
    for n in range(N):
        if flag[n]:
            tokens[row_pos[n]] = argmax[n]
            is_masked[row_pos[n]] = 0
    unmasked_pos = row_pos[flag != 0].astype(np.int32)
    still = np.array([row_pos[n] for n in range(N) if not flag[n] and is_masked[row_pos[n]]],
                     dtype=np.int32)
    stats, dflag = lane_boundary_stats(tokens, is_masked, B, role, b_len, t_lane,
                                       delim_ids, eos_id, rho_min, t_min,
                                       digit_ids, open_ids, close_ids)
    for n in range(N):
        if flag[n] == 1:
            stats[row_pos[n] // B, STAT_NSEL] += 1
        elif flag[n] == 2:
            stats[row_pos[n] // B, STAT_NDRAFT] += 1
    return dict(tokens=tokens, is_masked=is_masked, unmask_flag=flag,
                unmasked_pos=unmasked_pos, still_masked_pos=still,
                counts=np.array([len(unmasked_pos), len(still)], dtype=np.int32),
                lane_stats=stats, delim_flag=dflag)
