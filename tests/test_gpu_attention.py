"""lane_attn_forward on the GPU against the fp64 oracle.

Tolerance: outputs are bf16 and must be within 2e-2 max abs of the fp64
oracle on the same bf16 inputs; LSE (fp32) within 2e-3.  Full-size
workloads are compared element by element at seeds 0, 1 and 2 (and, as a
second path through the oracle, on sampled rows computed one row at a
time); small cases are compared element by element.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import dev, dev_bf16, f32, host_bf16_f32

pytestmark = pytest.mark.gpu
TOL_O = 2e-2
TOL_LSE = 2e-3


def _run(step, want_lse=True):
    import paper_2606_08411_amd as al
    kp = dev_bf16(step.k_pre)
    vp = dev_bf16(step.v_pre)
    n_ref = step.n_ref
    res = al.lane_attn_forward(
        dev_bf16(step.q), dev_bf16(step.k_lane), dev_bf16(step.v_lane), kp, vp, step.parent, step.B,
        refresh_idx=dev(step.refresh_idx) if n_ref else None,
        q_ref=dev_bf16(step.q_ref) if n_ref else None,
        k_ref=dev_bf16(step.k_ref) if n_ref else None,
        v_ref=dev_bf16(step.v_ref) if n_ref else None, want_lse=want_lse)
    torch.cuda.synchronize()
    o, lse, o_ref, lse_ref = res
    out = dict(o=host_bf16_f32(o), lse=None if lse is None else lse.cpu().numpy(),
               k_pre=host_bf16_f32(kp), v_pre=host_bf16_f32(vp))
    if n_ref:
        out["o_ref"] = host_bf16_f32(o_ref)
        out["lse_ref"] = lse_ref.cpu().numpy()
    return out


def _sample_rows(step):
    """Rows 0, B/2 and B-1 of every lane plus seeded extra rows (6 per lane
    up to 8 lanes, 4 up to 16, 3 beyond; the oracle computes each row on its
    own context)."""
    per_lane = 6 if step.L <= 8 else (4 if step.L <= 16 else 3)
    g = np.random.default_rng([step.seed, 41])
    rows = []
    for i in range(step.L):
        pick = {0, step.B // 2, step.B - 1}
        while len(pick) < min(per_lane, step.B):
            pick.add(int(g.integers(step.B)))
        rows += [i * step.B + a for a in sorted(pick)]
    return rows


def _check_full(step, out):
    ref = oracle.attention.decode_attention(
        f32(step.q), f32(step.k_lane), f32(step.v_lane), f32(step.k_pre), f32(step.v_pre),
        step.parent, step.B, step.refresh_idx, f32(step.q_ref), f32(step.k_ref), f32(step.v_ref))
    assert np.abs(out["o"] - ref["o"]).max() < TOL_O
    assert np.abs(out["lse"] - ref["lse"]).max() < TOL_LSE
    if step.n_ref:
        assert np.array_equal(out["k_pre"], ref["k_pre"]) and np.array_equal(out["v_pre"], ref["v_pre"])
        assert np.abs(out["o_ref"] - ref["o_ref"]).max() < TOL_O
        assert np.abs(out["lse_ref"] - ref["lse_ref"]).max() < TOL_LSE


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("name", ["tiny", "llada", "dream", "long", "wide"])
def test_attention_workloads(name, seed, step_cache):
    """Each seed draws its own inputs and (Dream, Long, Wide) its own lane
    tree (Section 3.3: the tree grows by forks, so every shape occurs)."""
    step = step_cache(name, seed, with_weight=False)
    out = _run(step)
    kp, vp = f32(step.k_pre), f32(step.v_pre)
    if step.n_ref:
        kp, vp = oracle.attention.refresh_scatter(kp, vp, step.refresh_idx, f32(step.k_ref), f32(step.v_ref))
        assert np.array_equal(out["k_pre"], kp) and np.array_equal(out["v_pre"], vp)
    if name == "tiny":
        _check_full(step, out)
        return
    rows = _sample_rows(step)
    o, lse = oracle.attention.lane_attention_rows(
        f32(step.q), f32(step.k_lane), f32(step.v_lane), kp, vp, step.parent, step.B, rows)
    assert np.abs(out["o"][rows] - o).max() < TOL_O
    assert np.abs(out["lse"][rows] - lse).max() < TOL_LSE
    if step.n_ref:
        rr = sorted({0, 1, step.n_ref // 2, step.n_ref - 1} |
                    set(np.random.default_rng([seed, 43]).choice(step.n_ref, 12, replace=False).tolist()))
        o_r, l_r = oracle.attention.refresh_attention(f32(step.q_ref)[rr], kp, vp)
        assert np.abs(out["o_ref"][rr] - o_r).max() < TOL_O
        assert np.abs(out["lse_ref"][rr] - l_r).max() < TOL_LSE


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("name", ["llada", "dream", "long", "wide"])
def test_attention_workloads_every_element(name, seed, step_cache):
    """Every output element at full size, each seed with its own lane tree:
    all lane rows and heads against oracle form A, and at Wide every refresh
    row and the rewritten prefix."""
    step = step_cache(name, seed, with_weight=False)
    out = _run(step)
    _check_full(step, out)


SWEEP = [
    # D, B, L, tree, Hq, Hkv, P, refresh_frac
    (64, 16, 1, "linear", 2, 2, 0, 0.0),
    (64, 32, 2, "fork", 4, 4, 128, 0.0),
    (128, 32, 3, "linear", 4, 1, 65, 0.0),
    (128, 64, 8, "random", 8, 2, 63, 0.1),
    (64, 48, 5, "forest", 7, 1, 200, 0.0),
    (128, 16, 33, "random", 4, 4, 100, 0.0),
    (64, 32, 64, "random", 2, 2, 31, 0.05),
    (128, 80, 4, "random", 8, 1, 1, 0.0),
    (64, 16, 12, "forest", 16, 2, 257, 0.3),
    (128, 32, 6, "linear", 28, 4, 130, 0.1),
    (64, 1024, 2, "fork", 16, 1, 64, 0.0),      # largest block, largest GQA group
    (128, 32, 64, "forest", 4, 1, 0, 0.0),      # no prefix, 64 roots: 256 workgroups of
                                                # the wavefront-split kernel, 64 units
    (128, 32, 64, "forest", 8, 2, 0, 0.0),      # the same on the 8-tile kernel: many key
                                                # splits hold no tile any wavefront of a
                                                # workgroup sees (empty-split path)
    (128, 48, 12, "random", 16, 2, 333, 0.2),   # 8-tile kernel (384 query tiles) with
                                                # 2 row tiles per lane; refresh rows on
                                                # the wavefront-split kernel
    (128, 16, 40, "random", 4, 2, 700, 0.0),    # wavefront-split kernel at its unit
                                                # limit (62 units), ragged prefix
]


@pytest.mark.parametrize("case", SWEEP, ids=[str(c) for c in SWEEP])
def test_attention_sweep(case):
    D, B, L, tree, Hq, Hkv, P, rf = case
    step = synth.make_step("tiny", 7, with_weight=False, D=D, B=B, L=L, tree=tree, Hq=Hq, Hkv=Hkv,
                           P=P, refresh_frac=rf, depth_max=4, V=64, d=64)
    out = _run(step)
    _check_full(step, out)


def _random_cases(n=10, seed=2606):
    """Seeded random valid shapes on both sides of the kernel choice (at
    most 256 query tiles x heads and 64 32-key units per tile take the
    wavefront-split kernel, larger ones the 8-tile kernel)."""
    rng = np.random.default_rng(seed)
    cases = []
    for k in range(n):
        big = k % 2 == 1          # long prefix or many heads: the 8-tile kernel
        Hkv = int(rng.choice([4, 8] if big else [1, 2, 4]))
        g = int(rng.choice([2, 4] if big else [1, 2, 4, 7]))
        L = int(rng.integers(6, 11) if big else rng.integers(1, 13))
        P = int(rng.integers(1000, 2200) if big else rng.integers(0, 700))
        cases.append((int(rng.choice([64, 128])), int(rng.choice([32, 48] if big else [16, 32, 48, 64])),
                      L, str(rng.choice(["linear", "fork", "random", "forest"])),
                      Hkv * g, Hkv, P, float(rng.choice([0.0, 0.0, 0.1]))))
    return cases


RANDOM = _random_cases(12)


@pytest.mark.parametrize("case", RANDOM, ids=[str(c) for c in RANDOM])
def test_attention_random_shapes(case):
    D, B, L, tree, Hq, Hkv, P, rf = case
    step = synth.make_step("tiny", 9, with_weight=False, D=D, B=B, L=L, tree=tree, Hq=Hq, Hkv=Hkv,
                           P=P, refresh_frac=rf, depth_max=4, V=64, d=64)
    out = _run(step)
    _check_full(step, out)


def test_attention_closed_forms():
    """V = 1 gives O = 1 exactly; K = 0 gives the mean of the visible V rows."""
    step = synth.make_step("tiny", 11, with_weight=False, L=5, tree="random", depth_max=3, P=70, B=32)
    one = np.full_like(step.v_lane, 0x3F80)
    step.v_lane = one
    step.v_pre = np.full_like(step.v_pre, 0x3F80)
    out = _run(step)
    assert np.all(out["o"] == 1.0)
    step = synth.make_step("tiny", 12, with_weight=False, L=4, tree="random", depth_max=3, P=70, B=32)
    step.k_lane = np.zeros_like(step.k_lane)
    step.k_pre = np.zeros_like(step.k_pre)
    out = _run(step)
    vall = np.concatenate([f32(step.v_pre), f32(step.v_lane)])
    for i in range(step.L):
        lanes = [i]
        j = int(step.parent[i])
        while j >= 0:
            lanes.append(j)
            j = int(step.parent[j])
        rows = list(range(step.P)) + [step.P + j * step.B + b for j in lanes for b in range(step.B)]
        mean = vall[rows].mean(axis=0)           # [Hkv][D]
        got = out["o"][i * step.B:(i + 1) * step.B]
        assert np.abs(got - mean[None]).max() < 1e-2


def test_attention_deterministic(step_cache):
    step = step_cache("dream", 0, with_weight=False)
    a = _run(step)
    b = _run(step)
    assert np.array_equal(a["o"], b["o"]) and np.array_equal(a["lse"], b["lse"])
