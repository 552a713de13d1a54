"""select_unmask on the GPU against the oracle.

Fed the same fp32 confidences and token ids, selection is pure compare and
integer logic, so every output must match the oracle bit for bit with no
exclusions: unmask flags, written-back tokens and mask bits, ordered
compacted positions, counts, lane statistics and delimiter flags.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import dev

pytestmark = pytest.mark.gpu


def _run_both(conf, arg, row_pos, tokens, is_masked, L, B, role, b_len, t_lane, mode, tau, fb,
              k_lane, delim=(0, 1), eos=2, rho=0.5, tmin=2, tau_future=None, sets=((), (), ())):
    import paper_2606_08411_amd as al
    tok_d = dev(tokens)
    msk_d = dev(is_masked)
    out = al.select_unmask(dev(conf), dev(arg), dev(row_pos), tok_d, msk_d, L, B, role, b_len,
                           t_lane, mode, tau, fb, k_lane, delim, eos, rho, tmin, tau_future,
                           digit_ids=sets[0], open_ids=sets[1], close_ids=sets[2])
    torch.cuda.synchronize()
    ref = oracle.select.select_unmask(conf, arg, row_pos, tokens, is_masked, B, role,
                                      b_len if b_len is not None else np.full(L, B),
                                      t_lane if t_lane is not None else np.zeros(L, np.int32),
                                      mode, tau, fb, k_lane, delim, eos, rho, tmin,
                                      tau_future=tau_future, digit_ids=sets[0],
                                      open_ids=sets[1], close_ids=sets[2])
    N = len(row_pos)
    cu, cs = out["counts"].cpu().numpy()
    assert [cu, cs] == list(ref["counts"])
    assert np.array_equal(out["unmask_flag"].cpu().numpy()[:N], ref["unmask_flag"])
    assert np.array_equal(out["unmasked_pos"].cpu().numpy()[:cu], ref["unmasked_pos"])
    assert np.array_equal(out["still_masked_pos"].cpu().numpy()[:cs], ref["still_masked_pos"])
    assert np.array_equal(tok_d.cpu().numpy(), ref["tokens"])
    assert np.array_equal(msk_d.cpu().numpy(), ref["is_masked"])
    assert np.array_equal(out["lane_stats"].cpu().numpy(), ref["lane_stats"])
    assert np.array_equal(out["delim_flag"].cpu().numpy(), ref["delim_flag"])
    return ref


@pytest.mark.parametrize("name", ["tiny", "llada", "dream", "long", "wide"])
@pytest.mark.parametrize("ties", [0, 16])
def test_select_workloads(name, ties, step_cache):
    s = step_cache(name, 0, with_weight=False)
    conf, arg = synth.random_confidences(1, s.N, s.V, tie_levels=ties)
    arg[::7] = np.array([0, 1, 2])[np.arange(len(arg[::7])) % 3]   # delimiters and EOS
    for fb in (0, 1, 2):
        _run_both(conf, arg, s.row_pos, s.tokens, s.is_masked, s.L, s.B, s.role, s.b_len, s.t_lane,
                  0, s.tau, fb, None)
    k_lane = np.random.default_rng(3).integers(0, s.B + 1, s.L).astype(np.int32)
    _run_both(conf, arg, s.row_pos, s.tokens, s.is_masked, s.L, s.B, s.role, s.b_len, s.t_lane,
              1, s.tau, 0, k_lane)


def test_select_random_states():
    rng = np.random.default_rng(17)
    drafts = 0
    for trial in range(40):
        L = int(rng.integers(1, 65))
        B = int(rng.choice([1, 3, 8, 16, 32, 64, 100]))
        if L * B > 8192:
            B = 8192 // L
        LB = L * B
        is_masked = (rng.random(LB) < rng.uniform(0.1, 0.9)).astype(np.uint8)
        row_pos = np.flatnonzero(rng.random(LB) < 0.8).astype(np.int32)
        N = len(row_pos)
        conf = (rng.integers(0, 9, N) / 8).astype(np.float32) if trial % 2 else rng.random(N).astype(np.float32)
        arg = rng.integers(0, 6, N).astype(np.int32)
        tokens = rng.integers(0, 8, LB).astype(np.int32)
        b_len = rng.integers(0, B + 1, L).astype(np.int32)
        role = rng.integers(0, 2, L).astype(np.uint8)
        t_lane = rng.integers(0, 5, L).astype(np.int32)
        k_lane = rng.integers(0, 4, L).astype(np.int32)
        tau = float(rng.choice([0.0, 0.5, 0.75, 1.0, 2.0]))
        rho = float(rng.choice([0.0, 0.25, 0.5, 0.6, 1.0]))
        mode = trial % 3 == 0
        tau_future = [None, 0.0, 0.5, 0.75, 1.0, 1.5][trial % 6]
        ref = _run_both(conf, arg, row_pos, tokens, is_masked, L, B, role, b_len, t_lane, int(mode),
                        tau, int(rng.integers(0, 3)), k_lane, (0, 1, 5), 2, rho, 2, tau_future)
        drafts += int((ref["unmask_flag"] == 2).sum())
    assert drafts > 0   # the lookahead path was exercised


@pytest.mark.parametrize("name", ["tiny", "llada", "long", "wide"])
def test_select_lookahead_workloads(name, step_cache):
    """Generate lanes with a lookahead window: b_len drawn below B, so the
    rows of [b_len, B) are draft candidates (Section 3.2, "Advancement
    control")."""
    s = step_cache(name, 0, with_weight=False)
    rng = np.random.default_rng(5)
    b_len = rng.integers(s.B // 4, s.B + 1, s.L).astype(np.int32)
    conf, arg = synth.random_confidences(2, s.N, s.V, tie_levels=8)
    arg[::5] = 2   # EOS predictions are never drafted
    ref = None
    for tf in (0.9, 0.5, 0.0):
        ref = _run_both(conf, arg, s.row_pos, s.tokens, s.is_masked, s.L, s.B, s.role, b_len,
                        s.t_lane, 0, s.tau, 1, None, tau_future=tf)
    assert (ref["unmask_flag"] == 2).any()


def test_select_valid_boundary():
    """ValidBoundary id sets on random states, including lanes longer than
    one wavefront pass (B up to 200), so the bracket depth carries across
    passes."""
    rng = np.random.default_rng(41)
    sets_list = [((3, 4, 5), (), ()), ((), (6,), (7,)), ((3, 4), (6, 8), (7, 9)),
                 (tuple(range(10, 42)), tuple(range(42, 74)), tuple(range(74, 106)))]
    hits = 0
    for trial in range(24):
        L = int(rng.integers(1, 9))
        B = int(rng.choice([8, 32, 64, 65, 128, 200]))
        LB = L * B
        is_masked = (rng.random(LB) < 0.25).astype(np.uint8)
        row_pos = np.flatnonzero(rng.random(LB) < 0.5).astype(np.int32)
        N = len(row_pos)
        conf = rng.random(N).astype(np.float32)
        hi = 12 if trial % 4 != 3 else 110
        arg = rng.integers(0, hi, N).astype(np.int32)
        tokens = rng.integers(0, hi, LB).astype(np.int32)
        b_len = rng.integers(0, B + 1, L).astype(np.int32)
        role = np.zeros(L, np.uint8)
        t_lane = np.full(L, 3, np.int32)
        sets = sets_list[trial % 4]
        ref = _run_both(conf, arg, row_pos, tokens, is_masked, L, B, role, b_len, t_lane, 0, 0.7,
                        1, None, (0, 1), 2, 0.25, 2, None, sets)
        plain = oracle.select.select_unmask(conf, arg, row_pos, tokens, is_masked, B, role, b_len,
                                            t_lane, 0, 0.7, 1, None, (0, 1), 2, 0.25, 2)
        hits += int((ref["delim_flag"] != plain["delim_flag"]).sum())
    assert hits > 0   # the sets removed delimiters somewhere


def test_select_empty_and_full():
    L, B = 3, 16
    tokens = np.arange(L * B, dtype=np.int32) % 7
    masked = np.zeros(L * B, np.uint8)
    role = np.zeros(L, np.uint8)
    # N = 0: only statistics
    _run_both(np.zeros(0, np.float32), np.zeros(0, np.int32), np.zeros(0, np.int32), tokens, masked,
              L, B, role, None, None, 0, 0.9, 1, None)
    # every position masked and scored
    masked[:] = 1
    conf = np.linspace(0, 1, L * B).astype(np.float32)
    _run_both(conf, np.full(L * B, 1, np.int32), np.arange(L * B, dtype=np.int32), tokens, masked,
              L, B, role, None, np.full(L, 3, np.int32), 0, 0.0, 0, None)


@pytest.mark.parametrize("N", [1, 2, 63, 64, 65, 127, 128, 129, 255, 256, 257, 511, 512, 513,
                               1023, 1024, 1025, 2047, 2049, 4096, 8191, 8192])
def test_select_row_count_boundaries(N):
    """Row counts at every boundary of the kernel's work split (threads per
    ranked row 16 / 8 / 4 / 2 / 1 at 64 / 128 / 256 / 512 rows, then 1024
    rows per pass up to 8 passes): threshold with the top-k fallback, and
    top-k, on lanes long enough that ranking scans many rows; bit-exact."""
    rng = np.random.default_rng([N, 41])
    L = 8 if N <= 1024 else 32
    B = max(1, -(-N // L))
    LB = L * B
    assert LB <= 8192
    row_pos = np.sort(rng.choice(LB, N, replace=False)).astype(np.int32)
    is_masked = np.zeros(LB, np.uint8)
    is_masked[row_pos] = 1
    is_masked[rng.random(LB) < 0.05] = 1
    conf = (rng.integers(0, 33, N) / 32).astype(np.float32)   # many exact ties
    arg = rng.integers(0, 9, N).astype(np.int32)
    tokens = rng.integers(0, 9, LB).astype(np.int32)
    b_len = rng.integers(B // 2, B + 1, L).astype(np.int32)
    role = (np.arange(L) % 2).astype(np.uint8)
    t_lane = rng.integers(0, 5, L).astype(np.int32)
    k_lane = rng.integers(0, B + 1, L).astype(np.int32)
    for tau, fb in ((1.5, 3), (0.9, 1)):      # tau above every confidence: fallback on every lane
        _run_both(conf, arg, row_pos, tokens, is_masked, L, B, role, b_len, t_lane, 0, tau, fb,
                  None, tau_future=0.5)
    _run_both(conf, arg, row_pos, tokens, is_masked, L, B, role, b_len, t_lane, 1, 0.9, 0, k_lane)
