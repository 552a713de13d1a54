"""fp64 oracle: LM-head confidence and argmax over masked positions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed (paper Section 3.2, "Lane-local denoising"): the first b_l
outputs of a lane feed the block-wise sampler's confidence-based transfer
rule, where a position's confidence is the probability of its most likely
token.  For masked position n (hidden row row_idx[n]):

    z[n, v]   = sum_k H[row_idx[n], k] * W[v, k]          (W is [V][d])
    C_n       = all vocabulary ids, minus eos_id when suppress_eos[n]
                (refine lanes suppress EOS predictions, same section)
    m         = max_{v in C_n} z[n, v]
    argmax    = smallest v in C_n with z[n, v] = m
    lse       = m + log sum_{v in C_n} exp(z[n, v] - m)
    conf      = exp(m - lse)   (max softmax probability, temperature 0)

Reading: EOS is removed from both the softmax and the argmax of a
suppressed row.  ``gap`` (m minus the second-largest logit of C_n) is
reported so that near-ties can be excluded from index comparisons.
"""
import numpy as np


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def logits(hidden, row_idx, W, vocab_chunk=16384, dtype=np.float64):
    """z = H[row_idx] @ W^T in fp64 ([N][V]).  W is widened to fp64 a chunk
    of rows at a time only to bound memory.  (dtype=np.float32 is the fp32
    twin used only as a CPU timing baseline.)"""
    H = np.asarray(hidden, dtype=dtype)[np.asarray(row_idx, dtype=np.int64)]
    V = W.shape[0]
    z = np.empty((H.shape[0], V), dtype=dtype)
    for c0 in range(0, V, vocab_chunk):
        c1 = min(V, c0 + vocab_chunk)
        z[:, c0:c1] = H @ np.asarray(W[c0:c1], dtype=dtype).T
    return z


def _allowed(V, suppress, eos_id):
    allowed = np.ones(V, dtype=bool)
    if suppress and 0 <= eos_id < V:
        allowed[eos_id] = False
    return allowed


def confidence_from_logits(z, suppress_eos=None, eos_id=-1, dtype=np.float64):
    """Full-softmax form on given logits [N][V].
    Returns dict(conf, argmax, lse, logconf, gap, m)."""
    z = np.asarray(z, dtype=dtype)
    N, V = z.shape
    out = dict(conf=np.zeros(N), argmax=np.zeros(N, dtype=np.int64), lse=np.zeros(N),
               logconf=np.zeros(N), gap=np.full(N, np.inf), m=np.zeros(N))
    for n in range(N):
        sup = bool(suppress_eos[n]) if suppress_eos is not None else False
        ids = np.flatnonzero(_allowed(V, sup, eos_id))
        zn = z[n, ids]
        m = zn.max()
        out["m"][n] = m
        out["argmax"][n] = ids[np.flatnonzero(zn == m)[0]]
        lse = m + np.log(np.exp(zn - m).sum())
        out["lse"][n] = lse
        out["logconf"][n] = m - lse
        out["conf"][n] = np.exp(m - lse)
        if len(zn) > 1:
            top2 = np.sort(zn)[-2:]
            out["gap"][n] = top2[1] - top2[0]
    return out


def lmhead_confidence_full(hidden, row_idx, W, suppress_eos=None, eos_id=-1, dtype=np.float64):
    """Full-softmax form over explicit fp64 logits (dtype=np.float32: the
    fp32 twin, a CPU timing baseline only)."""
    return confidence_from_logits(logits(hidden, row_idx, W, dtype=dtype), suppress_eos, eos_id,
                                  dtype=dtype)


def lmhead_confidence_chunked(hidden, row_idx, W, suppress_eos=None, eos_id=-1,
                              chunk=256):
    """Online form: the vocabulary is visited in chunks in ascending order and
    each row keeps a running (max m, sum s = sum exp(z - m), first argmax).

    Merging a chunk (mc, sc, ic) into (m, s, i):
      mc > m  -> s = s * exp(m - mc) + sc, m = mc, i = ic
      mc == m -> s = s + sc              (i kept: it is the lower index)
      mc < m  -> s = s + sc * exp(mc - m)
    conf = 1 / s, lse = m + log s.  Returns dict(conf, argmax, lse, logconf)."""
    H = _f64(hidden)[np.asarray(row_idx, dtype=np.int64)]
    N = H.shape[0]
    V = W.shape[0]
    m = np.full(N, -np.inf)
    s = np.zeros(N)
    idx = np.full(N, -1, dtype=np.int64)
    sup = np.zeros(N, dtype=bool) if suppress_eos is None else np.asarray(suppress_eos, bool)
    for c0 in range(0, V, chunk):
        c1 = min(V, c0 + chunk)
        z = H @ _f64(W[c0:c1]).T
        for n in range(N):
            zn = z[n].copy()
            if sup[n] and c0 <= eos_id < c1:
                zn[eos_id - c0] = -np.inf
            mc = zn.max()
            if mc == -np.inf:
                continue
            ic = c0 + int(np.flatnonzero(zn == mc)[0])
            sc = np.exp(zn - mc).sum()
            if mc > m[n]:
                s[n] = s[n] * np.exp(m[n] - mc) + sc
                m[n] = mc
                idx[n] = ic
            elif mc == m[n]:
                s[n] = s[n] + sc
            else:
                s[n] = s[n] + sc * np.exp(mc - m[n])
    lse = m + np.log(s)
    return dict(conf=1.0 / s, argmax=idx, lse=lse, logconf=m - lse)
