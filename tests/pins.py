"""Checks that pin the oracle to facts other than itself.

Every check takes the oracle module(s) as arguments so the same checks can be
run against deliberately broken copies of the oracle (see
test_oracle_mutants.py): a plausible mistake in the oracle must fail at least
one of them.  Nothing here imports the HIP library.

Pins used (paper passages in each docstring):
* library routines on special cases (torch scaled_dot_product_attention,
  scipy logsumexp / softmax),
* closed forms (V = 1 gives O = 1, K = 0 gives the mean of the visible V
  rows, W = 0 gives conf = 1/V),
* invariants (prefix-row permutation, lane relabelling, GQA = repeated MHA,
  forest = independent lanes),
* brute force with explicit Python loops on tiny inputs,
* hand-worked lane statistics from the paper's formulas (golden file).
"""
import itertools
import math
import os

import numpy as np
import scipy.special
import torch

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(seed, *shape, scale=1.0):
    g = np.random.default_rng([seed, 99])
    # bf16-exact values, as the device path sees them
    return synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(
        g.standard_normal(int(np.prod(shape)), dtype=np.float32) * np.float32(scale))
    ).reshape(shape).astype(np.float64)


def _lane_inputs(seed, L, B, P, Hq, Hkv, D):
    return (_rand(seed, L * B, Hq, D), _rand(seed + 1, L * B, Hkv, D),
            _rand(seed + 2, L * B, Hkv, D), _rand(seed + 3, P, Hkv, D),
            _rand(seed + 4, P, Hkv, D))


def _visible_rows(parent, i, B, P):
    """Indices into concat(prefix, lane rows) that lane i sees, by walking
    the parent links (Section 3.2: prefix state + own block)."""
    lanes = [i]
    j = int(parent[i])
    while j >= 0:
        lanes.append(j)
        j = int(parent[j])
    rows = list(range(P))
    for j in sorted(lanes):
        rows += [P + j * B + b for b in range(B)]
    return rows


def _sdpa(q, k, v, mask=None):
    """torch fp32 CPU reference: q [M][Hq][D], k/v [S][Hq][D]."""
    tq = torch.tensor(q, dtype=torch.float32).permute(1, 0, 2)[None]
    tk = torch.tensor(k, dtype=torch.float32).permute(1, 0, 2)[None]
    tv = torch.tensor(v, dtype=torch.float32).permute(1, 0, 2)[None]
    am = None if mask is None else torch.tensor(mask)
    o = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=am)
    scores = (tq @ tk.transpose(-1, -2)) / math.sqrt(q.shape[-1])
    if am is not None:
        scores = scores.masked_fill(~am, float("-inf"))
    lse = torch.logsumexp(scores, dim=-1)
    return o[0].permute(1, 0, 2).numpy().astype(np.float64), lse[0].T.numpy().astype(np.float64)


# ------------------------------------------------------------------ attention
def check_single_lane_is_blockwise(att):
    """One lane, no fork = ordinary block-wise attention over [prefix; block]
    (Section 3.1: the block-wise baseline is the single-frontier case)."""
    for (P, B, Hq, Hkv, D) in [(16, 8, 2, 2, 16), (13, 16, 4, 2, 8), (0, 4, 2, 1, 4)]:
        q, kl, vl, kp, vp = _lane_inputs(3, 1, B, P, Hq, Hkv, D)
        O, LSE = att.lane_attention_concat(q, kl, vl, kp, vp, np.array([-1]), B)
        g = Hq // Hkv
        k = np.repeat(np.concatenate([kp, kl]), g, axis=1)
        v = np.repeat(np.concatenate([vp, vl]), g, axis=1)
        ro, rl = _sdpa(q, k, v)
        assert np.abs(O - ro).max() < 2e-5, np.abs(O - ro).max()
        assert np.abs(LSE - rl).max() < 2e-5


def check_chain_is_block_causal(att):
    """A chain of lanes (each lane forked off the previous one) attends
    block-causally over the lane blocks and fully over the prefix."""
    L, B, P, Hq, Hkv, D = 4, 4, 6, 2, 2, 8
    q, kl, vl, kp, vp = _lane_inputs(5, L, B, P, Hq, Hkv, D)
    parent = np.arange(-1, L - 1)
    O, LSE = att.lane_attention_concat(q, kl, vl, kp, vp, parent, B)
    qb = np.arange(L * B)[:, None] // B
    kb = np.arange(L * B)[None, :] // B
    mask = np.concatenate([np.ones((L * B, P), bool), kb <= qb], axis=1)
    ro, rl = _sdpa(q, np.concatenate([kp, kl]), np.concatenate([vp, vl]),
                   np.broadcast_to(mask, (Hq, L * B, P + L * B)).copy())
    assert np.abs(O - ro).max() < 2e-5
    assert np.abs(LSE - rl).max() < 2e-5


def _trees():
    return [np.array([-1]), np.array([-1, 0]), np.array([-1, -1, -1]),
            np.array([-1, 0, 1, 2, 3]), np.array([-1, 0, 0, 1, 1, 2]),
            np.array([-1, 0, -1, 2, 1, 4, 0]),
            synth.lane_tree("random", 9, 4, 3)]


def check_forms_agree(att):
    """Lane-batched (dense masked) = each lane run on its concatenated context."""
    for t, parent in enumerate(_trees()):
        for (Hq, Hkv) in [(2, 2), (4, 2), (3, 1)]:
            L, B, P, D = len(parent), 4, 5, 8
            q, kl, vl, kp, vp = _lane_inputs(10 + t, L, B, P, Hq, Hkv, D)
            oa, la = att.lane_attention_concat(q, kl, vl, kp, vp, parent, B)
            ob, lb = att.lane_attention_dense(q, kl, vl, kp, vp, parent, B)
            assert np.abs(oa - ob).max() < 1e-12
            assert np.abs(la - lb).max() < 1e-12


def check_v_ones(att):
    """Softmax rows sum to one: V = 1 everywhere gives O = 1 exactly."""
    parent = np.array([-1, 0, 0, 2])
    L, B, P, Hq, Hkv, D = 4, 4, 7, 2, 1, 8
    q, kl, _, kp, _ = _lane_inputs(21, L, B, P, Hq, Hkv, D)
    for fn in (att.lane_attention_concat, att.lane_attention_dense):
        O, _ = fn(q, kl, np.ones_like(kl), kp, np.ones((P, Hkv, D)), parent, B)
        assert np.abs(O - 1.0).max() < 1e-12


def check_k_zero_mean(att):
    """K = 0 makes every visible key equally likely: O is the plain mean of
    the visible V rows and LSE = log(#visible)."""
    parent = np.array([-1, 0, 1, 0, -1])
    L, B, P, Hq, Hkv, D = 5, 2, 3, 2, 2, 4
    q, kl, vl, kp, vp = _lane_inputs(31, L, B, P, Hq, Hkv, D)
    for fn in (att.lane_attention_concat, att.lane_attention_dense):
        O, LSE = fn(q, np.zeros_like(kl), vl, np.zeros_like(kp), vp, parent, B)
        vall = np.concatenate([vp, vl])
        for i in range(L):
            rows = _visible_rows(parent, i, B, P)
            for h in range(Hq):
                mean = vall[rows, h].mean(axis=0)
                for a in range(B):
                    assert np.abs(O[i * B + a, h] - mean).max() < 1e-12
                    assert abs(LSE[i * B + a, h] - math.log(len(rows))) < 1e-12


def check_brute_force(att):
    """Pure-Python loops over (lane, head, query, key) on a tiny case."""
    parent = np.array([-1, 0, 0])
    L, B, P, Hq, Hkv, D = 3, 2, 3, 2, 1, 4
    q, kl, vl, kp, vp = _lane_inputs(41, L, B, P, Hq, Hkv, D)
    kall = np.concatenate([kp, kl])
    vall = np.concatenate([vp, vl])
    O, LSE = att.lane_attention_concat(q, kl, vl, kp, vp, parent, B)
    for i in range(L):
        rows = _visible_rows(parent, i, B, P)
        for h in range(Hq):
            for a in range(B):
                t = i * B + a
                s = [sum(q[t, h, x] * kall[r, 0, x] for x in range(D)) / math.sqrt(D)
                     for r in rows]
                mx = max(s)
                w = [math.exp(x - mx) for x in s]
                tot = math.fsum(w)
                for x in range(D):
                    ref = math.fsum(w[j] * vall[rows[j], 0, x] for j in range(len(rows))) / tot
                    assert abs(O[t, h, x] - ref) < 1e-12
                assert abs(LSE[t, h] - (mx + math.log(tot))) < 1e-12


def check_prefix_permutation(att):
    """Attention is a set function of its keys: permuting prefix rows
    leaves every output unchanged."""
    parent = np.array([-1, 0, 1])
    L, B, P, Hq, Hkv, D = 3, 4, 9, 2, 2, 8
    q, kl, vl, kp, vp = _lane_inputs(51, L, B, P, Hq, Hkv, D)
    perm = np.random.default_rng(0).permutation(P)
    o1, _ = att.lane_attention_concat(q, kl, vl, kp, vp, parent, B)
    o2, _ = att.lane_attention_concat(q, kl, vl, kp[perm], vp[perm], parent, B)
    assert np.abs(o1 - o2).max() < 1e-12


def check_lane_relabel(att):
    """Relabelling lanes consistently (any order that keeps parents before
    children) permutes the outputs the same way."""
    parent = np.array([-1, 0, 0, 1, 2, 2, -1])
    L, B, P, Hq, Hkv, D = 7, 2, 4, 2, 2, 4
    q, kl, vl, kp, vp = _lane_inputs(61, L, B, P, Hq, Hkv, D)
    order = [6, 0, 2, 5, 1, 4, 3]          # a topological order
    new = {old: n for n, old in enumerate(order)}
    parent2 = np.array([-1 if parent[o] < 0 else new[int(parent[o])] for o in order])
    rows = np.concatenate([np.arange(o * B, (o + 1) * B) for o in order])
    o1, l1 = att.lane_attention_concat(q, kl, vl, kp, vp, parent, B)
    o2, l2 = att.lane_attention_concat(q[rows], kl[rows], vl[rows], kp, vp, parent2, B)
    assert np.abs(o1[rows] - o2).max() < 1e-12
    assert np.abs(l1[rows] - l2).max() < 1e-12


def check_gqa_is_repeated_mha(att):
    """Grouped-query attention = multi-head attention with each K/V head
    repeated for its Hq/Hkv contiguous query heads."""
    parent = np.array([-1, 0, 1, 0])
    L, B, P, Hq, Hkv, D = 4, 4, 5, 6, 2, 8
    q, kl, vl, kp, vp = _lane_inputs(71, L, B, P, Hq, Hkv, D)
    g = Hq // Hkv
    o1, _ = att.lane_attention_dense(q, kl, vl, kp, vp, parent, B)
    o2, _ = att.lane_attention_dense(q, np.repeat(kl, g, 1), np.repeat(vl, g, 1),
                                     np.repeat(kp, g, 1), np.repeat(vp, g, 1), parent, B)
    assert np.abs(o1 - o2).max() < 1e-12
    o3, _ = att.lane_attention_concat(q, kl, vl, kp, vp, parent, B)
    o4, _ = att.lane_attention_concat(q, np.repeat(kl, g, 1), np.repeat(vl, g, 1),
                                      np.repeat(kp, g, 1), np.repeat(vp, g, 1), parent, B)
    assert np.abs(o3 - o4).max() < 1e-12


def check_forest_is_independent(att):
    """Lanes with no common ancestor lane (a forest of roots) see only the
    shared prefix and their own block: the same as separate single-lane
    calls."""
    L, B, P, Hq, Hkv, D = 3, 4, 6, 2, 1, 8
    q, kl, vl, kp, vp = _lane_inputs(81, L, B, P, Hq, Hkv, D)
    O, _ = att.lane_attention_dense(q, kl, vl, kp, vp, np.full(L, -1), B)
    for i in range(L):
        r = slice(i * B, (i + 1) * B)
        oi, _ = att.lane_attention_concat(q[r], kl[r], vl[r], kp, vp, np.array([-1]), B)
        assert np.abs(O[r] - oi).max() < 1e-12


def check_refresh(att):
    """Compact refresh (Section 3.4): refreshed rows are rewritten in place,
    lanes attend over the rebuilt prefix and refresh rows attend over the
    rebuilt prefix only (torch SDPA on an explicitly rebuilt prefix)."""
    parent = np.array([-1, 0, 0])
    L, B, P, Hq, Hkv, D = 3, 4, 10, 2, 2, 8
    q, kl, vl, kp, vp = _lane_inputs(91, L, B, P, Hq, Hkv, D)
    idx = np.array([1, 4, 9])
    qr, kr, vr = _rand(92, 3, Hq, D), _rand(93, 3, Hkv, D), _rand(94, 3, Hkv, D)
    out = att.decode_attention(q, kl, vl, kp, vp, parent, B, idx, qr, kr, vr)
    kp2 = kp.copy()
    vp2 = vp.copy()
    sel = np.zeros(P, bool)
    sel[idx] = True
    kp2[sel] = kr
    vp2[sel] = vr
    assert np.array_equal(out["k_pre"], kp2) and np.array_equal(out["v_pre"], vp2)
    o_ref, l_ref = _sdpa(qr, kp2, vp2)
    assert np.abs(out["o_ref"] - o_ref).max() < 2e-5
    assert np.abs(out["lse_ref"] - l_ref).max() < 2e-5
    o_l, _ = att.lane_attention_dense(q, kl, vl, kp2, vp2, parent, B)
    assert np.abs(out["o"] - o_l).max() < 1e-12


def check_rows_agree(att):
    """The one-row-at-a-time form equals the lane-batched forms."""
    parent = np.array([-1, 0, 1, 0, 3])
    L, B, P, Hq, Hkv, D = 5, 4, 6, 4, 2, 8
    q, kl, vl, kp, vp = _lane_inputs(101, L, B, P, Hq, Hkv, D)
    ob, lb = att.lane_attention_dense(q, kl, vl, kp, vp, parent, B)
    rows = [0, 3, 5, 9, 12, 19]
    heads = [3, 0, 2]
    o, l = att.lane_attention_rows(q, kl, vl, kp, vp, parent, B, rows, heads)
    assert np.abs(o - ob[rows][:, heads]).max() < 1e-12
    assert np.abs(l - lb[rows][:, heads]).max() < 1e-12


ATTENTION_CHECKS = [check_single_lane_is_blockwise, check_rows_agree, check_chain_is_block_causal,
                    check_forms_agree, check_v_ones, check_k_zero_mean, check_brute_force,
                    check_prefix_permutation, check_lane_relabel, check_gqa_is_repeated_mha,
                    check_forest_is_independent, check_refresh]


# -------------------------------------------------------------------- LM head
def _lm_forms(lm):
    return [lambda *a, **k: lm.lmhead_confidence_full(*a, **k),
            lambda *a, **k: lm.lmhead_confidence_chunked(*a, chunk=3, **k),
            lambda *a, **k: lm.lmhead_confidence_chunked(*a, chunk=256, **k)]


def check_lm_brute_force(lm):
    """Explicit loops: z = dot products (math.fsum), m = first maximum, full
    softmax; EOS removed from suppressed rows (Section 3.2)."""
    for V in (2, 3, 7, 16, 40):
        d, N = 8, 5
        H = _rand(100 + V, N, d)
        W = _rand(200 + V, V, d, scale=1 / math.sqrt(d))
        rows = np.array([4, 0, 2, 2, 1])
        sup = np.array([0, 1, 0, 1, 1], np.uint8)
        eos = 1
        for form in _lm_forms(lm):
            out = form(H, rows, W, suppress_eos=sup, eos_id=eos)
            for n in range(N):
                z = [math.fsum(H[rows[n], k] * W[v, k] for k in range(d)) for v in range(V)]
                ids = [v for v in range(V) if not (sup[n] and v == eos)]
                best = ids[0]
                for v in ids:
                    if z[v] > z[best]:
                        best = v
                tot = math.fsum(math.exp(z[v] - z[best]) for v in ids)
                assert out["argmax"][n] == best
                assert abs(out["conf"][n] - 1.0 / tot) < 1e-12
                assert abs(out["lse"][n] - (z[best] + math.log(tot))) < 1e-12
                if "gap" in out and len(ids) > 1:
                    second = max(z[v] for v in ids if v != best)
                    assert abs(out["gap"][n] - (z[best] - second)) < 1e-12


def check_lm_library(lm):
    """lse equals scipy's logsumexp and conf equals the max of scipy's
    softmax of the same logits (computed here with a float64 einsum)."""
    V, d, N = 700, 16, 6
    H = _rand(301, N, d, scale=3.0)
    W = _rand(302, V, d, scale=1 / 4)
    rows = np.arange(N)
    z = np.einsum("nk,vk->nv", H, W)
    for form in _lm_forms(lm):
        out = form(H, rows, W)
        assert np.abs(out["lse"] - scipy.special.logsumexp(z, axis=1)).max() < 1e-10
        sm = scipy.special.softmax(z, axis=1)
        assert np.abs(out["conf"] - sm.max(axis=1)).max() < 1e-12
        assert np.array_equal(out["argmax"], sm.argmax(axis=1))


def check_lm_zero_weight(lm):
    """W = 0: every logit is 0, so conf = 1/|C| and the argmax is the
    smallest allowed id (0, or 1 when EOS = 0 is suppressed)."""
    V, d = 37, 8
    H = _rand(311, 3, d)
    W = np.zeros((V, d))
    for form in _lm_forms(lm):
        out = form(H, np.arange(3), W, suppress_eos=np.array([0, 1, 0]), eos_id=0)
        assert list(out["argmax"]) == [0, 1, 0]
        assert np.abs(out["conf"] - np.array([1 / V, 1 / (V - 1), 1 / V])).max() < 1e-15


def check_lm_duplicate_rows(lm):
    """Two identical vocabulary rows holding the maximum: the lower id wins,
    also when the duplicates fall in different chunks."""
    V, d = 600, 8
    H = np.zeros((4, d))
    H[np.arange(4), np.arange(4)] = 1.0
    W = _rand(322, V, d, scale=0.1)
    for n in range(4):
        W[[5 + 100 * n, 260 + 80 * n]] = 10.0 * H[n]
    for form in _lm_forms(lm):
        out = form(H, np.arange(4), W)
        assert list(out["argmax"]) == [5 + 100 * n for n in range(4)]


def check_lm_integer_closed_form(lm):
    """One-hot hidden rows and small-integer weights make every logit an
    exact integer, so conf and lse have closed forms."""
    V, d = 9, 4
    W = np.array([[(3 * v + 2 * k) % 7 - 3 for k in range(d)] for v in range(V)], float)
    H = np.zeros((d, d))
    H[np.arange(d), np.arange(d)] = [1, 2, -1, 3]
    for form in _lm_forms(lm):
        out = form(H, np.arange(d), W)
        for n in range(d):
            z = H[n, n] * W[:, n]
            m = z.max()
            assert out["argmax"][n] == int(np.flatnonzero(z == m)[0])
            assert abs(out["conf"][n] - 1.0 / np.exp(z - m).sum()) < 1e-15


def check_lm_eos_is_row_deletion(lm):
    """Suppressing EOS = deleting its vocabulary row and mapping the ids
    above it down by one."""
    V, d, N, eos = 50, 8, 6, 17
    H = _rand(331, N, d, scale=2)
    W = _rand(332, V, d, scale=0.5)
    W[eos] = H.mean(axis=0) * 3       # make EOS a strong competitor
    keep = np.array([v for v in range(V) if v != eos])
    for form in _lm_forms(lm):
        out = form(H, np.arange(N), W, suppress_eos=np.ones(N, np.uint8), eos_id=eos)
        ref = form(H, np.arange(N), W[keep])
        assert np.array_equal(out["argmax"], keep[ref["argmax"]])
        assert np.abs(out["conf"] - ref["conf"]).max() < 1e-14


def check_lm_row_gather(lm):
    """row_idx selects hidden rows: the result for a gathered row equals the
    result for that row alone."""
    V, d = 64, 8
    H = _rand(341, 10, d)
    W = _rand(342, V, d)
    rows = np.array([7, 2, 9])
    for form in _lm_forms(lm):
        out = form(H, rows, W)
        for n, r in enumerate(rows):
            one = form(H[r:r + 1], np.array([0]), W)
            assert out["argmax"][n] == one["argmax"][0]
            assert abs(out["conf"][n] - one["conf"][0]) < 1e-15


LMHEAD_CHECKS = [check_lm_brute_force, check_lm_library, check_lm_zero_weight,
                 check_lm_duplicate_rows, check_lm_integer_closed_form,
                 check_lm_eos_is_row_deletion, check_lm_row_gather]


# ------------------------------------------------------------------ selection
def _topk_set_by_definition(cand, conf, pos, k):
    """The unique subset S of size min(k, |cand|) in which every member beats
    every non-member on (higher confidence, then lower position) -- found by
    enumerating subsets, not by sorting."""
    k = min(k, len(cand))

    def beats(a, b):
        return conf[a] > conf[b] or (conf[a] == conf[b] and pos[a] < pos[b])

    found = [set(S) for S in itertools.combinations(cand, k)
             if all(beats(a, b) for a in S for b in cand if b not in S)]
    assert len(found) == 1
    return found[0]


def check_select_brute_force(sel):
    """Exhaustive small cases, random and exactly tied confidences."""
    rng = np.random.default_rng(7)
    for trial in range(60):
        L = int(rng.integers(1, 4))
        B = int(rng.integers(1, 7))
        LB = L * B
        is_masked = (rng.random(LB) < 0.7).astype(np.uint8)
        row_pos = np.flatnonzero(rng.random(LB) < 0.9)   # may include unmasked rows
        N = len(row_pos)
        conf = (rng.integers(0, 17, N) / 16).astype(np.float32)
        arg = rng.integers(3, 50, N).astype(np.int32)
        tokens = rng.integers(3, 50, LB).astype(np.int32)
        b_len = rng.integers(0, B + 1, L).astype(np.int32)
        role = rng.integers(0, 2, L).astype(np.uint8)
        t_lane = rng.integers(0, 5, L).astype(np.int32)
        tau = float(rng.choice([0.5, 0.75, 1.0, 1.5]))
        fb = int(rng.integers(0, 3))
        k_lane = rng.integers(0, B + 2, L).astype(np.int32)
        for mode in (sel.MODE_THRESHOLD, sel.MODE_TOPK):
            out = sel.select_unmask(conf, arg, row_pos, tokens, is_masked, B, role, b_len,
                                    t_lane, mode, tau, fb, k_lane)
            expect = set()
            for lane in range(L):
                cand = [n for n in range(N) if row_pos[n] // B == lane
                        and row_pos[n] % B < b_len[lane] and is_masked[row_pos[n]]]
                if mode == sel.MODE_THRESHOLD:
                    S = {n for n in cand if conf[n] >= np.float32(tau)}
                    if not S and fb > 0:
                        S = _topk_set_by_definition(cand, conf, row_pos, fb)
                else:
                    S = _topk_set_by_definition(cand, conf, row_pos, int(k_lane[lane]))
                expect |= S
            got = set(np.flatnonzero(out["unmask_flag"]).tolist())
            assert got == expect, (trial, mode, got, expect)
            # write-back and compaction follow from the chosen set
            tk = tokens.copy()
            mk = is_masked.copy()
            for n in expect:
                tk[row_pos[n]] = arg[n]
                mk[row_pos[n]] = 0
            assert np.array_equal(out["tokens"], tk) and np.array_equal(out["is_masked"], mk)
            up = sorted(int(row_pos[n]) for n in expect)
            sp = sorted(int(row_pos[n]) for n in range(N) if n not in expect and mk[row_pos[n]])
            assert list(out["unmasked_pos"]) == up and list(out["still_masked_pos"]) == sp
            assert list(out["counts"]) == [len(up), len(sp)]
            nsel = [sum(1 for n in expect if row_pos[n] // B == lane) for lane in range(L)]
            assert list(out["lane_stats"][:, 4]) == nsel


def check_select_threshold_extremes(sel):
    """tau above 1 transfers only the fallback; tau = 0 transfers every
    eligible masked position (conf is never negative)."""
    step = synth.make_step("tiny", 3, with_weight=False)
    conf, arg = synth.random_confidences(3, step.N, step.V)
    args = (step.row_pos, step.tokens, step.is_masked, step.B, step.role, step.b_len,
            step.t_lane)
    out = sel.select_unmask(conf, arg, *args, sel.MODE_THRESHOLD, 1.01, 1)
    lanes = sorted(set((step.row_pos // step.B).tolist()))
    assert out["counts"][0] == len(lanes)
    for lane in lanes:
        rows = np.flatnonzero(step.row_pos // step.B == lane)
        best = rows[np.lexsort((step.row_pos[rows], -conf[rows]))[0]]
        assert out["unmask_flag"][best] == 1
    out = sel.select_unmask(conf, arg, *args, sel.MODE_THRESHOLD, 1.01, 0)
    assert out["counts"][0] == 0 and np.array_equal(out["tokens"], step.tokens)
    out = sel.select_unmask(conf, arg, *args, sel.MODE_THRESHOLD, 0.0, 0)
    assert out["counts"][0] == step.N and out["counts"][1] == 0
    assert not out["is_masked"].any()


def _parse_golden():
    cases = []
    with open(os.path.join(GOLDEN, "lane_stats_cases.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            lhs, rhs = line.split("||")
            toks, b_len, role, t, rho, tmin = [x.strip() for x in lhs.split("|")]
            split, filled, valid, fork, dpos = [x.strip() for x in rhs.split("|")]
            tk = toks.split(",")
            cases.append(dict(
                tokens=np.array([-1 if x == "M" else int(x) for x in tk], np.int32),
                masked=np.array([x == "M" for x in tk], np.uint8),
                b_len=int(b_len), role=0 if role == "gen" else 1, t=int(t),
                rho=float(rho), tmin=int(tmin),
                expect=[int(split), int(filled), int(valid), int(fork)],
                dpos=[int(x) for x in dpos.split(",")] if dpos else []))
    return cases


def check_lane_stats_golden(sel):
    """Hand-worked cases of eq. split_point, eq. fork_condition and the
    valid prefix length (tests/golden/lane_stats_cases.txt)."""
    cases = _parse_golden()
    assert len(cases) >= 10
    for c in cases:
        B = len(c["tokens"])
        stats, dflag = sel.lane_boundary_stats(
            c["tokens"], c["masked"], B, np.array([c["role"]]), np.array([c["b_len"]]),
            np.array([c["t"]]), (0, 1), 2, c["rho"], c["tmin"])
        assert list(stats[0, :4]) == c["expect"], (c, stats)
        assert list(np.flatnonzero(dflag)) == c["dpos"], (c, dflag)


def check_lane_stats_scan(sel):
    """Lane statistics on random states equal direct vectorised scans."""
    rng = np.random.default_rng(11)
    L, B = 6, 16
    for _ in range(20):
        tokens = rng.integers(0, 6, L * B).astype(np.int32)
        masked = (rng.random(L * B) < 0.4).astype(np.uint8)
        b_len = rng.integers(0, B + 1, L).astype(np.int32)
        role = rng.integers(0, 2, L).astype(np.uint8)
        t_lane = rng.integers(0, 4, L).astype(np.int32)
        stats, dflag = sel.lane_boundary_stats(tokens, masked, B, role, b_len, t_lane,
                                               (0, 1), 2, 0.5, 2)
        for lane in range(L):
            n = b_len[lane]
            tk = tokens[lane * B:lane * B + n]
            mk = masked[lane * B:lane * B + n].astype(bool)
            d = (~mk) & np.isin(tk, [0, 1])
            split = int(np.flatnonzero(d)[-1]) + 1 if d.any() else 0
            stop = mk | (tk == 2)
            valid = int(np.argmax(stop)) if stop.any() else int(n)
            filled = int((~mk).sum())
            fork = int(role[lane] == 0 and split > 0 and t_lane[lane] >= 2
                       and np.float32(filled) >= np.float32(0.5) * np.float32(n))
            assert list(stats[lane, :4]) == [split, filled, valid, fork]
            assert np.array_equal(dflag[lane * B:lane * B + n], d.astype(np.uint8))
            assert not dflag[lane * B + n:(lane + 1) * B].any()


def _parse_lookahead_golden():
    cases = []
    with open(os.path.join(GOLDEN, "lookahead_cases.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            lhs, rhs = line.split("||")
            roles, b_len, toks, rows, mode, tau, fb, k_lane, tauf = [x.strip() for x in lhs.split("|")]
            flags, nsel, ndraft = [x.strip() for x in rhs.split("|")]
            lanes = [t.split(",") for t in toks.split("/")]
            B = len(lanes[0])
            assert all(len(t) == B for t in lanes)
            flat = [x for t in lanes for x in t]
            rws = [r.split(":") for r in rows.split(",")]
            cases.append(dict(
                role=np.array([0 if r == "gen" else 1 for r in roles.split(",")], np.uint8),
                b_len=np.array([int(x) for x in b_len.split(",")], np.int32), B=B,
                tokens=np.array([-1 if x == "M" else int(x) for x in flat], np.int32),
                masked=np.array([x == "M" for x in flat], np.uint8),
                row_pos=np.array([int(r[0]) for r in rws], np.int64),
                conf=np.array([float(r[1]) for r in rws], np.float32),
                arg=np.array([int(r[2]) for r in rws], np.int32),
                mode=0 if mode == "threshold" else 1, tau=float(tau), fb=int(fb),
                k_lane=np.array([int(x) for x in k_lane.split(",")], np.int32),
                tau_future=float(tauf),
                flags=[int(x) for x in flags.split(",")],
                nsel=[int(x) for x in nsel.split(",")],
                ndraft=[int(x) for x in ndraft.split(",")]))
    return cases


def check_lookahead_golden(sel):
    """Hand-worked transfers and lookahead drafts
    (tests/golden/lookahead_cases.txt), with the write-back they imply."""
    cases = _parse_lookahead_golden()
    assert len(cases) >= 5
    for c in cases:
        L = len(c["role"])
        out = sel.select_unmask(c["conf"], c["arg"], c["row_pos"], c["tokens"], c["masked"],
                                c["B"], c["role"], c["b_len"], np.full(L, 3, np.int32),
                                c["mode"], c["tau"], c["fb"], c["k_lane"], eos_id=2,
                                tau_future=c["tau_future"])
        assert list(out["unmask_flag"]) == c["flags"], (c, out["unmask_flag"])
        assert list(out["lane_stats"][:, 4]) == c["nsel"]
        assert list(out["lane_stats"][:, 5]) == c["ndraft"]
        hit = [n for n, f in enumerate(c["flags"]) if f]
        tk = c["tokens"].copy()
        mk = c["masked"].copy()
        for n in hit:
            tk[c["row_pos"][n]] = c["arg"][n]
            mk[c["row_pos"][n]] = 0
        assert np.array_equal(out["tokens"], tk) and np.array_equal(out["is_masked"], mk)
        assert list(out["unmasked_pos"]) == [int(c["row_pos"][n]) for n in hit]


def check_lookahead_properties(sel):
    """On random states: drafting off (None, or tau_future above 1 since
    conf <= 1) is the plain call; drafting never changes the in-region
    decision or the boundary statistics (they read [0, b_len) only);
    drafts lie in generate-lane windows on masked, non-EOS rows; lowering
    tau_future only adds drafts."""
    rng = np.random.default_rng(23)
    for trial in range(40):
        L = int(rng.integers(1, 5))
        B = int(rng.integers(2, 9))
        LB = L * B
        is_masked = (rng.random(LB) < 0.7).astype(np.uint8)
        row_pos = np.flatnonzero(rng.random(LB) < 0.9)
        N = len(row_pos)
        conf = (rng.integers(0, 17, N) / 16).astype(np.float32)
        arg = rng.integers(2, 9, N).astype(np.int32)     # id 2 (EOS) occurs
        tokens = rng.integers(0, 9, LB).astype(np.int32)
        b_len = rng.integers(0, B + 1, L).astype(np.int32)
        role = rng.integers(0, 2, L).astype(np.uint8)
        t_lane = rng.integers(0, 5, L).astype(np.int32)
        mode = int(rng.integers(0, 2))
        k_lane = rng.integers(0, B + 1, L).astype(np.int32)
        args = (conf, arg, row_pos, tokens, is_masked, B, role, b_len, t_lane, mode, 0.75, 1, k_lane)
        plain = sel.select_unmask(*args)
        for off in (None, 1.5):
            o = sel.select_unmask(*args, tau_future=off)
            for key in plain:
                assert np.array_equal(o[key], plain[key]), (trial, key)
        prev = None
        for tf in (1.0, 0.75, 0.5, 0.0):
            o = sel.select_unmask(*args, tau_future=tf)
            f = o["unmask_flag"]
            assert np.array_equal(f == 1, plain["unmask_flag"] == 1)
            assert np.array_equal(o["lane_stats"][:, :5], plain["lane_stats"][:, :5])
            assert np.array_equal(o["delim_flag"], plain["delim_flag"])
            for n in np.flatnonzero(f == 2):
                pos = int(row_pos[n])
                assert role[pos // B] == 0 and pos % B >= b_len[pos // B]
                assert is_masked[pos] and arg[n] != 2 and conf[n] >= np.float32(tf)
            d = set(np.flatnonzero(f == 2).tolist())
            if prev is not None:
                assert prev <= d
            prev = d
        # tau_future = 0: every masked window row of a generate lane that
        # does not predict EOS is drafted.
        want = {n for n in range(N) if role[row_pos[n] // B] == 0
                and row_pos[n] % B >= b_len[row_pos[n] // B]
                and is_masked[row_pos[n]] and arg[n] != 2}
        assert prev == want


def _id_set(field):
    if field == "-":
        return ()
    out = []
    for part in field.split(","):
        if "-" in part:
            lo, hi = part.split("-")
            out += list(range(int(lo), int(hi) + 1))
        else:
            out.append(int(part))
    return tuple(out)


def check_valid_boundary_golden(sel):
    """Hand-worked numeric-period and bracket-balance cases
    (tests/golden/valid_boundary_cases.txt)."""
    n = 0
    with open(os.path.join(GOLDEN, "valid_boundary_cases.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            lhs, rhs = line.split("||")
            toks, b_len, role, t, rho, tmin, dig, opn, cls = [x.strip() for x in lhs.split("|")]
            split, filled, valid, fork, dpos = [x.strip() for x in rhs.split("|")]
            tk = toks.split(",")
            # "M" = masked; "M<id>" = masked position still holding a stale id
            tokens = np.array([(int(x[1:]) if len(x) > 1 else -1) if x.startswith("M") else int(x)
                               for x in tk], np.int32)
            masked = np.array([x.startswith("M") for x in tk], np.uint8)
            stats, dflag = sel.lane_boundary_stats(
                tokens, masked, len(tk), np.array([0 if role == "gen" else 1]),
                np.array([int(b_len)]), np.array([int(t)]), (0, 1), 2, float(rho), int(tmin),
                _id_set(dig), _id_set(opn), _id_set(cls))
            want = [int(split), int(filled), int(valid), int(fork)]
            assert list(stats[0, :4]) == want, (line, stats)
            assert list(np.flatnonzero(dflag)) == ([int(x) for x in dpos.split(",")] if dpos else []), line
            n += 1
    assert n >= 10


def check_valid_boundary_properties(sel):
    """Empty id sets are the plain statistics; a rule can only remove
    delimiters (split never grows); brackets never inside an open scope."""
    rng = np.random.default_rng(31)
    L, B = 5, 24
    for _ in range(30):
        tokens = rng.integers(0, 26, L * B).astype(np.int32)
        masked = (rng.random(L * B) < 0.3).astype(np.uint8)
        b_len = rng.integers(0, B + 1, L).astype(np.int32)
        role = rng.integers(0, 2, L).astype(np.uint8)
        t_lane = rng.integers(0, 4, L).astype(np.int32)
        base = sel.lane_boundary_stats(tokens, masked, B, role, b_len, t_lane, (0, 1), 2, 0.5, 2)
        same = sel.lane_boundary_stats(tokens, masked, B, role, b_len, t_lane, (0, 1), 2, 0.5, 2,
                                       (), (), ())
        assert np.array_equal(base[0], same[0]) and np.array_equal(base[1], same[1])
        for sets in [((10, 11, 12), (), ()), ((), (20,), (22,)), ((10, 13), (20, 21), (22, 23))]:
            st, df = sel.lane_boundary_stats(tokens, masked, B, role, b_len, t_lane, (0, 1), 2,
                                             0.5, 2, *sets)
            assert np.all(df <= base[1])
            assert np.all(st[:, 0] <= base[0][:, 0])
            assert np.array_equal(st[:, 1:3], base[0][:, 1:3])   # filled, valid_len unchanged
            for pos in np.flatnonzero(df):
                lane, i = pos // B, pos % B
                seg_t = tokens[lane * B:pos + 1]
                seg_m = masked[lane * B:pos + 1].astype(bool)
                opens = int(np.isin(seg_t[~seg_m], sets[1]).sum())
                closes = int(np.isin(seg_t[~seg_m], sets[2]).sum())
                assert opens <= closes
                if i > 0 and not masked[pos - 1]:
                    assert tokens[pos - 1] not in sets[0]


SELECT_CHECKS = [check_select_brute_force, check_select_threshold_extremes,
                 check_lane_stats_golden, check_lane_stats_scan,
                 check_lookahead_golden, check_lookahead_properties,
                 check_valid_boundary_golden, check_valid_boundary_properties]


# ------------------------------------------------------------------ refresh
# Hand-worked L_refresh = min(P + L, P + max(s + v) + m) (Section 3.4).
REFRESH_CASES = [
    # P, L, lane starts, valid lengths, margin -> L_refresh
    (100, 256, [0, 32, 64], [32, 10, 0], 16, 180),   # L_eff = max(32, 42, 64) = 64
    (100, 256, [0, 32, 64], [32, 10, 0], 200, 356),  # margin runs past the end: P + L
    (512, 128, [0], [0], 0, 512),                    # nothing valid yet: the prompt only
    (512, 128, [], [], 8, 520),                      # no lanes: L_eff = 0
    (7, 64, [40, 8], [24, 50], 3, 71),               # L_eff = max(64, 58) = 64 -> 7+64+3 = 74 > 71
    (0, 64, [16, 0], [16, 8], 4, 36),                # no prompt: 0 + 32 + 4
]


def check_refresh_window_golden(rf):
    for P, L, s, v, m, want in REFRESH_CASES:
        assert rf.refresh_window_len(P, L, s, v, m) == want, (P, L, s, v, m)


def check_refresh_window_properties(rf):
    """P <= L_refresh <= P + L; monotone in the margin and in every lane's
    frontier; independent of lane order."""
    rng = np.random.default_rng(3)
    for _ in range(200):
        P = int(rng.integers(0, 600))
        L = int(rng.integers(1, 1025))
        n = int(rng.integers(0, 9))
        s = rng.integers(0, L, n)
        v = np.array([int(rng.integers(0, L - x + 1)) for x in s], dtype=np.int64)
        m = int(rng.integers(0, 64))
        r = rf.refresh_window_len(P, L, s, v, m)
        assert P <= r <= P + L
        assert rf.refresh_window_len(P, L, s, v, m + 1) >= r
        perm = rng.permutation(n)
        assert rf.refresh_window_len(P, L, s[perm], v[perm], m) == r
        if n:
            v2 = v.copy()
            v2[0] = min(v2[0] + 5, L - s[0])
            assert rf.refresh_window_len(P, L, s, v2, m) >= r


REFRESH_CHECKS = [check_refresh_window_golden, check_refresh_window_properties]


# ------------------------------------------------------------------ scheduler
def _script_conf(sc):
    script = {(it, pos): (c, t) for it, pos, c, t in sc["script"]}
    W = sc["B"] + sc["window"]

    def conf_fn(it, order, lanes, rows):
        conf, arg = [], []
        for r in rows:
            pos = lanes[order[r // W]].s + r % W
            c, t = script.get((it, pos), (0.1, 20 + pos))
            conf.append(c)
            arg.append(t)
        return np.array(conf, np.float32), np.array(arg, np.int32)
    return conf_fn


def _run_scenario(sch, sc, conf_fn=None):
    return sch.run(sc["P"], sc["L"], sc["B"], sc["window"], conf_fn or _script_conf(sc),
                   sc["max_iters"], tau=sc["tau"], fallback_k=sc["fallback_k"],
                   tau_future=sc["tau_future"], rho_min=sc["rho_min"], t_min=sc["t_min"])


def check_scheduler_golden(sch):
    """Two hand-traced runs (tests/golden/scheduler_scenarios.json)."""
    import json
    G = json.load(open(os.path.join(GOLDEN, "scheduler_scenarios.json")))
    assert len(G["scenarios"]) >= 2
    for sc in G["scenarios"]:
        S = _run_scenario(sch, sc)
        lanes = [["gen" if ln.role == 0 else "ref", ln.s, ln.b, ln.kind, ln.v] for ln in S.lanes]
        ex = sc["expect"]
        assert lanes == ex["lanes"], (sc["name"], lanes)
        assert S.collect() == ex["output"], (sc["name"], S.collect())
        tk = [int(t) if not m else -1 for t, m in zip(S.tokens, S.masked)]
        assert tk == ex["tokens"], (sc["name"], tk)
        plans = [[[["gen" if S.lanes[x].role == 0 else "ref", S.lanes[x].s] for x in order], cp]
                 for order, cp in S.plans if order]
        assert plans == ex["plans"], (sc["name"], plans)
        got = [S.iterations, S.nfe, S.forks, S.spawns, S.stops]
        assert got == [ex[k] for k in ("iterations", "nfe", "forks", "spawns", "stops")], (sc["name"], got)


def _random_conf(seed, p_delim=0.08, p_eos=0.02):
    def conf_fn(it, order, lanes, rows):
        rng = np.random.default_rng([seed, it])
        n = len(rows)
        conf = rng.uniform(0, 1, n).astype(np.float32)
        arg = rng.integers(3, 50, n).astype(np.int32)
        u = rng.random(n)
        arg[u < p_delim] = rng.integers(0, 2, int((u < p_delim).sum()))
        arg[(u >= p_delim) & (u < p_delim + p_eos)] = 2
        return conf, arg
    return conf_fn


def check_scheduler_blockwise(sch):
    """No delimiter ever predicted and no lookahead: no fork can happen, so
    the lanes are the consecutive blocks [kB, (k+1)B) of block-wise
    semi-autoregressive decoding (Section 3.1), one model call each
    iteration, and the output is the whole sequence up to the first EOS."""
    for seed in range(4):
        L, B = 40, 8
        cf = _random_conf(seed, p_delim=0.0, p_eos=0.0)
        S = sch.run(0, L, B, 0, cf, 500, tau=0.7, fallback_k=1, t_min=1)
        assert S.forks == 0
        assert [(ln.s, ln.b, ln.role) for ln in S.lanes] == [(k * B, min(B, L - k * B), 0)
                                                          for k in range((L + B - 1) // B)]
        assert not S.masked.any()
        assert S.collect() == [int(t) for t in S.tokens]
        assert S.nfe == 1 + S.iterations


def check_scheduler_structure(sch):
    """Random runs: forks come from generate lanes and split them in place
    (refine child at the parent's start, generate child right after it);
    successors start at s + v; refine lanes have no children; a filled
    position never changes afterwards; the output is a subsequence of the
    final tokens in position order with no EOS from a generate leaf."""
    for seed in range(6):
        L, B, window = 48, 8, (0, 8)[seed % 2]
        cf = _random_conf(seed)
        S = sch.Scheduler(2, L, B, window)
        seen = {}
        for it in range(300):
            order, _ = S.plan()
            if not order:
                break
            tk, mk = S.blocks(order)
            rows = np.flatnonzero(mk).astype(np.int32)
            conf, arg = cf(it, order, S.lanes, rows)
            ln = [S.lanes[x] for x in order]
            res = __import__("oracle").select.select_unmask(
                conf, arg, rows, tk, mk, S.W, np.array([x.role for x in ln], np.uint8),
                np.array([x.b for x in ln], np.int32), np.array([x.t + 1 for x in ln], np.int32),
                0, 0.8, 1, None, (0, 1), 2, 0.5, 2, tau_future=0.85 if window else None)
            S.commit(order, res["tokens"], res["is_masked"], res["lane_stats"])
            for pos in np.flatnonzero(S.masked == 0):
                assert seen.setdefault(int(pos), int(S.tokens[pos])) == int(S.tokens[pos])
        for ln in S.lanes:
            kids = [S.lanes[c] for c in ln.children]
            if ln.role == 1:
                assert not kids
            if ln.kind == "fork":
                assert ln.role == 0 and kids[0].role == 1 and kids[0].s == ln.s
                if len(kids) > 1:
                    assert kids[1].role == 0 and kids[1].s == ln.s + kids[0].b
            if ln.kind == "spawn":
                assert len(kids) == 1 and kids[0].s == ln.s + ln.v and ln.v > 0
            assert 0 <= ln.s and ln.s + ln.b <= L
        out = S.collect()
        it_tok = iter(int(t) for t in S.tokens)
        assert all(any(x == y for y in it_tok) for x in out)   # subsequence
        # NFE = 1 + sum over iterations of the prefix-state groups evaluated:
        # the two children of a fork share one state, every other lane has
        # its own (Section 3.4, shared-prefix lane batching).
        nfe = 1
        for order, _ in S.plans:
            keys = set()
            for x in order:
                par = S.lanes[x].parent
                keys.add(("fork", par) if par >= 0 and S.lanes[par].kind == "fork" else ("own", x))
            nfe += len(keys)
        assert S.nfe == nfe


SCHEDULER_CHECKS = [check_scheduler_golden, check_scheduler_blockwise, check_scheduler_structure]
