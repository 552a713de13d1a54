"""fp64 oracle: lane-batched bidirectional attention over a shared prefix.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed (paper Section 3.2, "Lane-local denoising", and Section 3.4,
"Shared-prefix lane batching"): every active lane l is a block of B query
tokens evaluated against its prefix state kappa_l plus its own block, with
bidirectional attention inside the block.  Lanes that share a prefix state are
evaluated in one batched call.  Readings fixed here (the paper leaves them
open):

* kappa_l = the shared cached prefix (P rows) followed by the blocks of l's
  proper ancestors in the lane tree (root first).  Siblings, cousins and
  descendants are invisible.  With one lane and no fork this is ordinary
  block-wise attention; along a chain it is block-causal attention.
* Masked positions are attended as ordinary keys (they carry the mask
  embedding); a lookahead window inside the B rows is an ordinary own-block
  row.
* scale = 1/sqrt(D); grouped-query heads map head h to K/V head h // (Hq/Hkv);
  no bias, soft-cap, window or positional term (rotary embedding is applied
  by the caller before the call).
* Compact cache refresh (Section 3.4, "Compact cache refresh and reuse"):
  refreshed prefix rows are rewritten in place first; lanes then attend over
  the updated prefix; refreshed rows' queries attend over the whole updated
  prefix only (a shared cache row cannot depend on one lane's block).

Shapes: q [L*B][Hq][D], k_lane/v_lane [L*B][Hkv][D], k_pre/v_pre [P][Hkv][D],
parent [L] with parent[i] in [-1, i).  Outputs are fp64.
"""
import math

import numpy as np


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def lane_ancestors(parent):
    """Proper ancestors of every lane, root first (walk of the parent links)."""
    out = []
    for i in range(len(parent)):
        chain = []
        j = int(parent[i])
        while j >= 0:
            chain.append(j)
            j = int(parent[j])
        out.append(chain[::-1])
    return out


def softmax_attend(q, k, v, scale):
    """Plain softmax attention of query rows q [M][D] over keys k, v [S][D].

    Returns (out [M][D], lse [M]) with lse = log sum_k exp(scale * q.k).
    Computed in the inputs' precision (fp64 for the oracle; the fp32 twin
    used only as a CPU timing baseline passes fp32 arrays)."""
    s = scale * (q @ k.T)
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    l = e.sum(axis=1, keepdims=True)
    p = e / l
    tol = 1e-12 if p.dtype == np.float64 else 1e-4
    assert np.all(np.abs(p.sum(axis=1) - 1.0) < tol), "softmax rows must sum to 1"
    return p @ v, (m + np.log(l))[:, 0]


def lane_attention_concat(q, k_lane, v_lane, k_pre, v_pre, parent, B, scale=None):
    """Form A: each lane run on its own explicitly concatenated context
    [prefix; ancestor blocks root->parent; own block]."""
    q, k_lane, v_lane, k_pre, v_pre = map(_f64, (q, k_lane, v_lane, k_pre, v_pre))
    LB, Hq, D = q.shape
    Hkv = k_lane.shape[1]
    g = Hq // Hkv
    L = len(parent)
    assert LB == L * B and Hq == g * Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    O = np.zeros((LB, Hq, D))
    LSE = np.zeros((LB, Hq))
    anc = lane_ancestors(parent)
    for i in range(L):
        blocks = anc[i] + [i]
        kc = np.concatenate([k_pre] + [k_lane[j * B:(j + 1) * B] for j in blocks], axis=0)
        vc = np.concatenate([v_pre] + [v_lane[j * B:(j + 1) * B] for j in blocks], axis=0)
        rows = slice(i * B, (i + 1) * B)
        for h in range(Hq):
            o, lse = softmax_attend(q[rows, h], kc[:, h // g], vc[:, h // g], scale)
            O[rows, h] = o
            LSE[rows, h] = lse
    return O, LSE


def ancestor_or_self(parent):
    """R[i][j] = True iff lane j is lane i or one of its ancestors.

    Built as the reflexive-transitive closure of the parent relation by
    repeated boolean products (independent of lane_ancestors)."""
    L = len(parent)
    adj = np.zeros((L, L), dtype=bool)
    for i in range(L):
        if parent[i] >= 0:
            adj[i, parent[i]] = True
    R = np.eye(L, dtype=bool)
    for _ in range(L):
        R = R | ((R.astype(np.int64) @ adj.astype(np.int64)) > 0)
    return R


def lane_attention_dense(q, k_lane, v_lane, k_pre, v_pre, parent, B, scale=None):
    """Form B: one dense [L*B] x [P + L*B] attention with a boolean visibility
    mask (every prefix row; lane-block rows of ancestor-or-self lanes)."""
    q, k_lane, v_lane, k_pre, v_pre = map(_f64, (q, k_lane, v_lane, k_pre, v_pre))
    LB, Hq, D = q.shape
    P, Hkv = k_pre.shape[0], k_pre.shape[1]
    g = Hq // Hkv
    L = len(parent)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    R = ancestor_or_self(parent)
    lane_of_row = np.arange(LB) // B
    vis = np.concatenate([np.ones((LB, P), dtype=bool),
                          R[lane_of_row][:, lane_of_row]], axis=1)
    k_all = np.concatenate([k_pre, k_lane], axis=0)
    v_all = np.concatenate([v_pre, v_lane], axis=0)
    O = np.zeros((LB, Hq, D))
    LSE = np.zeros((LB, Hq))
    for h in range(Hq):
        s = scale * (q[:, h] @ k_all[:, h // g].T)
        s = np.where(vis, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        e = np.exp(s - m)
        l = e.sum(axis=1, keepdims=True)
        O[:, h] = (e / l) @ v_all[:, h // g]
        LSE[:, h] = (m + np.log(l))[:, 0]
    return O, LSE


def refresh_scatter(k_pre, v_pre, refresh_idx, k_ref, v_ref):
    """Rewrite refreshed prefix rows: K_pre[idx[r]] <- K_ref[r], same for V.
    Returns updated copies (the inputs are not modified)."""
    k2 = np.array(k_pre, copy=True)
    v2 = np.array(v_pre, copy=True)
    for r, p in enumerate(np.asarray(refresh_idx)):
        k2[int(p)] = k_ref[r]
        v2[int(p)] = v_ref[r]
    return k2, v2


def refresh_attention(q_ref, k_pre, v_pre, scale=None):
    """Refreshed rows' queries over all P rows of the (updated) prefix."""
    q_ref, k_pre, v_pre = map(_f64, (q_ref, k_pre, v_pre))
    n, Hq, D = q_ref.shape
    Hkv = k_pre.shape[1]
    g = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    O = np.zeros((n, Hq, D))
    LSE = np.zeros((n, Hq))
    if n == 0:
        return O, LSE
    for h in range(Hq):
        o, lse = softmax_attend(q_ref[:, h], k_pre[:, h // g], v_pre[:, h // g], scale)
        O[:, h] = o
        LSE[:, h] = lse
    return O, LSE


def decode_attention(q, k_lane, v_lane, k_pre, v_pre, parent, B,
                     refresh_idx=None, q_ref=None, k_ref=None, v_ref=None,
                     scale=None, form="concat"):
    """The three attention steps of one decode call, in order:
    1. refreshed rows are written into the prefix;
    2. lanes attend over the updated prefix (form A or B);
    3. refreshed rows attend over the updated prefix.
    Returns dict(o, lse, o_ref, lse_ref, k_pre, v_pre)."""
    k_pre = _f64(k_pre)
    v_pre = _f64(v_pre)
    if refresh_idx is not None and len(refresh_idx):
        k_pre, v_pre = refresh_scatter(k_pre, v_pre, refresh_idx, _f64(k_ref), _f64(v_ref))
    fn = lane_attention_concat if form == "concat" else lane_attention_dense
    o, lse = fn(q, k_lane, v_lane, k_pre, v_pre, parent, B, scale)
    out = dict(o=o, lse=lse, k_pre=k_pre, v_pre=v_pre)
    if refresh_idx is not None and len(refresh_idx):
        out["o_ref"], out["lse_ref"] = refresh_attention(q_ref, k_pre, v_pre, scale)
    return out


def lane_attention_rows(q, k_lane, v_lane, k_pre, v_pre, parent, B, rows, heads=None,
                        scale=None, dtype=np.float64):
    """Outputs of selected query rows only, computed one row at a time on the
    row's own visible key set (for spot checks at full size).  dtype is the
    working precision: fp64 for the oracle; fp32 only for the CPU timing
    baseline's twin.
    Returns (O [len(rows)][len(heads)][D], LSE [len(rows)][len(heads)])."""
    LB, Hq, D = q.shape
    Hkv = k_lane.shape[1]
    g = Hq // Hkv
    heads = list(range(Hq)) if heads is None else list(heads)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    anc = lane_ancestors(parent)
    O = np.zeros((len(rows), len(heads), D), dtype=dtype)
    LSE = np.zeros((len(rows), len(heads)), dtype=dtype)
    cv = lambda x: np.asarray(x, dtype=dtype)
    for a, t in enumerate(rows):
        i = int(t) // B
        blocks = anc[i] + [i]
        for b, h in enumerate(heads):
            kv = h // g
            kc = np.concatenate([cv(k_pre[:, kv])] + [cv(k_lane[j * B:(j + 1) * B, kv]) for j in blocks])
            vc = np.concatenate([cv(v_pre[:, kv])] + [cv(v_lane[j * B:(j + 1) * B, kv]) for j in blocks])
            o, lse = softmax_attend(cv(q[t, h])[None, :], kc, vc, dtype(scale))
            O[a, b] = o[0]
            LSE[a, b] = lse[0]
    return O, LSE
