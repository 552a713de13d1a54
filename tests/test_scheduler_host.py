"""The library's host scheduler (al_sched_*) against the oracle scheduler.

The scheduler is host code, so this runs without a GPU: both schedulers are
driven by the oracle selection on the same confidences, and must produce the
same plans, lane trees, token states, outputs and counters, exactly.
"""
import json
import os

import numpy as np
import pytest

import oracle
import pins

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def al():
    import paper_2606_08411_amd as al
    try:
        al.library()
    except al.AsyncLaneError:
        pytest.skip("libasynclane.so not built")
    return al


class _LaneView:
    def __init__(self, s):
        self.s = s


def _drive_lib(al, P, L, B, window, conf_fn, max_iters, tau, fallback_k, tau_future, rho_min, t_min,
               max_lanes=64):
    S = al.AlSched(P, L, B, window, max_lanes)
    plans = []
    for it in range(max_iters):
        pl = S.plan()
        n = len(pl["lane_id"])
        if n == 0:
            break
        plans.append(([["gen" if r == 0 else "ref", int(s)] for r, s in zip(pl["role"], pl["start"])],
                      pl["call_parent"].tolist()))
        tk, mk = S.blocks()
        rows = np.flatnonzero(mk).astype(np.int32)
        lanes = {int(x): _LaneView(int(s)) for x, s in zip(pl["lane_id"], pl["start"])}
        conf, arg = conf_fn(it, [int(x) for x in pl["lane_id"]], lanes, rows)
        res = oracle.select.select_unmask(conf, arg, rows, tk, mk, S.W, pl["role"], pl["b_len"],
                                          pl["t_step"], 0, tau, fallback_k, None, (0, 1), 2,
                                          rho_min, t_min, tau_future=tau_future)
        S.commit(res["tokens"], res["is_masked"], res["lane_stats"])
    return S, plans


def test_golden_scenarios(al):
    G = json.load(open(os.path.join(HERE, "golden", "scheduler_scenarios.json")))
    for sc in G["scenarios"]:
        S, plans = _drive_lib(al, sc["P"], sc["L"], sc["B"], sc["window"], pins._script_conf(sc),
                              sc["max_iters"], sc["tau"], sc["fallback_k"], sc["tau_future"],
                              sc["rho_min"], sc["t_min"])
        ex = sc["expect"]
        tr = S.tree()
        kinds = {0: None, 1: "fork", 2: "spawn"}
        lanes = [["gen" if r == 0 else "ref", int(s), int(b), kinds[int(k)], None if v < 0 else int(v)]
                 for r, s, b, k, v in zip(tr["role"], tr["start"], tr["length"], tr["kind"], tr["v"])]
        assert lanes == ex["lanes"], lanes
        assert [[p, c] for p, c in plans] == ex["plans"]
        assert S.collect() == ex["output"]
        tk, mk = S.state()
        assert [int(t) if not m else -1 for t, m in zip(tk, mk)] == ex["tokens"]
        c = S.counters()
        assert [c[k] for k in ("iterations", "nfe", "forks", "spawns", "stops")] == \
            [ex[k] for k in ("iterations", "nfe", "forks", "spawns", "stops")]


@pytest.mark.parametrize("seed", range(8))
def test_random_runs_match_oracle(al, seed):
    L, B, window = [(64, 8, 0), (96, 16, 16), (40, 8, 8), (128, 32, 0)][seed % 4]
    max_lanes = 64 if seed < 6 else 2          # the plan cap truncates the depth-first order
    cf = pins._random_conf(110 + seed)
    tf = 0.85 if window else None
    S, plans = _drive_lib(al, 5, L, B, window, cf, 400, 0.8, 1, tf, 0.5, 2, max_lanes)
    R = oracle.scheduler.Scheduler(5, L, B, window, max_lanes)
    for it in range(400):
        order, _ = R.plan()
        if not order:
            break
        tk, mk = R.blocks(order)
        rows = np.flatnonzero(mk).astype(np.int32)
        conf, arg = cf(it, order, R.lanes, rows)
        ln = [R.lanes[x] for x in order]
        res = oracle.select.select_unmask(conf, arg, rows, tk, mk, R.W, np.array([x.role for x in ln], np.uint8),
                                          np.array([x.b for x in ln], np.int32),
                                          np.array([x.t + 1 for x in ln], np.int32), 0, 0.8, 1, None,
                                          (0, 1), 2, 0.5, 2, tau_future=tf)
        R.commit(order, res["tokens"], res["is_masked"], res["lane_stats"])
    ref_plans = [([["gen" if R.lanes[x].role == 0 else "ref", R.lanes[x].s] for x in o], cp)
                 for o, cp in R.plans if o]
    assert plans == ref_plans
    tr = S.tree()
    assert len(tr["role"]) == len(R.lanes)
    for i, ln in enumerate(R.lanes):
        assert (int(tr["role"][i]), int(tr["start"][i]), int(tr["length"][i]), int(tr["parent"][i])) == \
            (ln.role, ln.s, ln.b, ln.parent)
    tk, mk = S.state()
    assert np.array_equal(tk[mk == 0], R.tokens[R.masked == 0]) and np.array_equal(mk, R.masked)
    assert S.collect() == R.collect()
    c = S.counters()
    assert [c["iterations"], c["nfe"], c["forks"], c["spawns"], c["stops"]] == \
        [R.iterations, R.nfe, R.forks, R.spawns, R.stops]
    assert c["forks"] + c["spawns"] > 0


def test_bad_arguments(al):
    lib = al.library()
    assert not lib.al_sched_create(0, 0, 8, 0, 4, 3)
    assert not lib.al_sched_create(0, 16, 8, 0, 65, 3)
    S = al.AlSched(0, 16, 8)
    with pytest.raises(al.AsyncLaneError):
        S.plan(cap=0)


def test_commit_rejects_bad_statistics(al):
    """Lane statistics outside the lane's region are rejected and leave the
    scheduler state as it was."""
    S = al.AlSched(0, 16, 8)
    pl = S.plan()
    tk, mk = S.blocks()
    good = np.zeros((1, al.LANE_STATS), np.int32)
    for bad in ([9, 0, 0, 0, 0, 0], [0, -1, 0, 0, 0, 0], [0, 0, 9, 0, 0, 0], [0, 8, 8, 1, 0, 0]):
        with pytest.raises(al.AsyncLaneError):
            S.commit(tk, mk, np.array([bad], np.int32))
        assert S.counters()["iterations"] == 0
    assert S.commit(tk, mk, good) == 1
    assert S.counters()["iterations"] == 1
