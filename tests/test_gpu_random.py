"""Seeded random valid shapes for lane_attn_forward and both LM-head layouts
against the fp64 oracle, beyond the hand-picked sweeps: head layouts
(MHA and GQA up to 7 query heads per K/V head), D 64 / 128, blocks of
16-96 rows (several query tiles per lane), 1-19 lanes in every tree kind,
prefixes up to 2200 rows with refresh rows, and LM heads from 1 to 700
scored rows, d from 8 to 760, V from 1 to 70001 with EOS suppression, and
selection states with every option.  The comparison rules are those of
the attention, LM-head and selection tests."""
import numpy as np
import pytest

import oracle
import synth
import test_gpu_attention as TA
import test_gpu_lmhead as TL

pytestmark = pytest.mark.gpu


def _attn_cases(n, seed):
    rng = np.random.default_rng([seed, 5150])
    out = []
    for k in range(n):
        big = k % 3 == 2
        Hkv = int(rng.choice([4, 8] if big else [1, 2, 4]))
        g = int(rng.choice([1, 2, 4] if big else [1, 2, 4, 7]))
        L = int(rng.integers(4, 17) if big else rng.integers(1, 20))
        P = int(rng.integers(600, 2200) if big else rng.integers(0, 900))
        D = int(rng.choice([64, 128]))
        B = int(rng.choice([16, 32, 48, 64, 96]))
        tree = str(rng.choice(["linear", "fork", "random", "forest"]))
        rf = float(rng.choice([0.0, 0.0, 0.05, 0.2]))
        out.append((D, B, L, tree, Hkv * g, Hkv, P, rf, 100 + k + 1000 * seed))
    return out


def _lm_cases(n, seed):
    rng = np.random.default_rng([seed, 6160])
    out = []
    for k in range(n):
        N = int(rng.choice([1, 2, 31, 32, 33, 64, 77, 96, 97, 128, 129, 200, 224, 225, 300, 450,
                            614, 700]))
        n_rows = N + int(rng.integers(0, 40))
        d = int(8 * rng.integers(1, 96))
        V = int(rng.choice([1, 7, 100, 513, 4096, 9000, 40000, 70001]))
        while N * V * d > 3e9:
            V = max(1, V // 2)
        eos = int(rng.integers(-1, min(V, 50)))
        if V == 1 and eos == 0:   # an empty candidate set is rejected by the library
            eos = -1
        out.append((N, n_rows, d, V, eos, k + 1000 * seed))
    return out


ATTN = _attn_cases(16, 7)
LM = _lm_cases(24, 7)


@pytest.mark.parametrize("case", ATTN, ids=[str(c[:8]) for c in ATTN])
def test_attention_random_valid_shapes(case):
    D, B, L, tree, Hq, Hkv, P, rf, seed = case
    step = synth.make_step("tiny", seed, with_weight=False, D=D, B=B, L=L, tree=tree, Hq=Hq,
                           Hkv=Hkv, P=P, refresh_frac=rf, depth_max=5, V=64, d=64)
    TA._check_full(step, TA._run(step))


@pytest.mark.parametrize("case", LM, ids=[str(c[:5]) for c in LM])
def test_lmhead_random_valid_shapes(case):
    N, n_rows, d, V, eos, seed = case
    g = np.random.default_rng([seed, 77])
    scale = g.uniform(1, 6, n_rows).astype(np.float32)
    H = synth.f32_to_bf16_bits(g.standard_normal((n_rows, d), dtype=np.float32) * scale[:, None])
    W = synth.f32_to_bf16_bits(g.standard_normal((V, d), dtype=np.float32) / np.float32(np.sqrt(d)))
    row_idx = np.sort(g.choice(n_rows, N, replace=False)).astype(np.int32)
    sup = (g.random(N) < 0.5).astype(np.uint8)
    ref = oracle.lmhead.lmhead_confidence_full(TL.f32(H), row_idx, TL.f32(W), sup, eos)
    TL._compare(TL._run(H, W, row_idx, sup, eos), ref, f"plain {case[:5]}")
    TL._compare(TL._run_packed(H, W, row_idx, sup, eos), ref, f"packed {case[:5]}")


def test_select_random_states_with_id_sets():
    """Selection on seeded random states: both modes, lookahead thresholds,
    ValidBoundary digit / bracket id sets and delimiter sets, blocks of 1 to
    256 rows and up to 64 lanes; bit-exact against the oracle."""
    import test_gpu_select as TS
    rng = np.random.default_rng([7, 999])
    drafts = 0
    for trial in range(60):
        L = int(rng.integers(1, 65))
        B = int(rng.choice([1, 2, 3, 8, 16, 31, 32, 33, 64, 100, 128, 256]))
        if L * B > 8192:
            B = max(1, 8192 // L)
        LB = L * B
        is_masked = (rng.random(LB) < rng.uniform(0.0, 1.0)).astype(np.uint8)
        row_pos = np.flatnonzero(rng.random(LB) < rng.uniform(0.0, 1.0)).astype(np.int32)
        N = len(row_pos)
        conf = ((rng.integers(0, 9, N) / 8).astype(np.float32) if trial % 2
                else rng.random(N).astype(np.float32))
        arg = rng.integers(0, 12, N).astype(np.int32)
        tokens = rng.integers(0, 12, LB).astype(np.int32)
        b_len = rng.integers(0, B + 1, L).astype(np.int32)
        role = rng.integers(0, 2, L).astype(np.uint8)
        t_lane = rng.integers(0, 6, L).astype(np.int32)
        k_lane = rng.integers(0, 5, L).astype(np.int32)
        tau = float(rng.choice([0.0, 0.125, 0.5, 0.75, 1.0, 2.0]))
        rho = float(rng.choice([0.0, 0.25, 0.5, 0.6, 1.0]))
        tau_future = [None, 0.0, 0.5, 0.75, 1.0, 1.5][trial % 6]
        sets = [((), (), ()), ((3, 4), (6,), (7,)), ((3,), (), ()), ((), (6, 8), (7, 9))][trial % 4]
        delim = (0, 1, 5) if trial % 5 else (0,)
        ref = TS._run_both(conf, arg, row_pos, tokens, is_masked, L, B, role, b_len, t_lane,
                           int(trial % 3 == 0), tau, int(rng.integers(0, 3)), k_lane, delim, 2,
                           rho, int(rng.integers(0, 4)), tau_future, sets)
        drafts += int((ref["unmask_flag"] == 2).sum())
    assert drafts > 0
