"""Benchmark of one AsyncLane decode step's hot path on one MI355X.

A step = lane_attn_forward (with compact-refresh rows when the workload has
them) + lmhead_confidence over the masked positions + select_unmask, on
seeded synthetic inputs already resident in HBM.  Prints ONE JSON line.

value       (attention FLOPs + LM-head FLOPs) / step time, in TFLOP/s
roofline    the LM-head call (the step's dominant op: a streaming GEMM
            kernel + a small merge kernel) against HBM: algorithmic bytes
            per call / its measured average duration
cpu_baseline the fp64 oracle on a bounded sample of the same workload,
            timed on this host's cores
"""
import argparse
import hashlib
import re
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
WORKLOAD_NAMES = {
    "tiny": "tiny (4 heads, D 64, P 128, 2 lanes x 32, d 256, V 1024)",
    "llada": "LLaDA-8B-shaped layer + LM head (32/32 heads, D 128, P 512, 4 lanes x 32 "
             "linear tree, d 4096, V 126464, 60% masked)",
    "dream": "Dream-7B-shaped GQA layer + LM head (28/4 heads, D 128, P 1024, 8 lanes x 32, "
             "d 3584, V 152064, 50% masked)",
    "long": "long generation, LLaDA shape (P 2048, 16 lanes x 32 depth<=6, 40% masked)",
    "wide": "wide lane set + compact refresh (P 4096, 32 lanes x 64 depth<=8, 410 refresh "
            "rows, 30% masked)",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="llada", choices=list(WORKLOAD_NAMES))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kernel-reps", type=int, default=50)
    ap.add_argument("--w-layout", default="packed", choices=["packed", "plain"],
                    help="LM-head weight layout of the timed step: the one-time packed copy "
                         "(lmhead_pack_weight, made before timing, like a model load) or W as given")
    ap.add_argument("--quick", action="store_true",
                    help="skip the distribution, cold-input and graph passes (profiler runs)")
    ap.add_argument("--decode", action="store_true",
                    help="instead of the step benchmark, run whole synthetic decodes driven by "
                         "the library's active-lane scheduler and print their JSON line")
    ap.add_argument("--decode-len", type=int, default=256)
    ap.add_argument("--decode-runs", type=int, default=3)
    return ap.parse_args()


def depth_of(parent):
    out = []
    for i in range(len(parent)):
        dd, j = 0, int(parent[i])
        while j >= 0:
            dd, j = dd + 1, int(parent[j])
        out.append(dd)
    return out


def attention_flops(s):
    """Visible query-key pairs x 4 D (QK^T and PV), per query head."""
    pairs = sum(s.B * (s.P + s.B * (dd + 1)) for dd in depth_of(s.parent))
    f = 4.0 * s.Hq * s.D * pairs
    f += 4.0 * s.Hq * s.D * s.n_ref * s.P
    return f


def lmhead_flops(s):
    return 2.0 * s.N * s.d * s.V


def lmhead_bytes(s):
    """W once + the scored hidden rows + conf/argmax/lse per row."""
    return 2.0 * s.V * s.d + 2.0 * s.N * s.d + 12.0 * s.N


def _code_only(text):
    """C++ source without comments, trailing blanks and empty lines (the
    kernel sources hold no string literal containing a comment marker)."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return "\n".join(line.rstrip() for line in text.splitlines() if line.strip())


def kernel_source_hash():
    """Hash of the LM-head kernel code (comments excluded, so counters stay
    attached to the code they were taken on when only comments change)."""
    h = hashlib.sha256()
    for f in ("lmhead.hip", "common.h"):
        with open(os.path.join(ROOT, "paper_2606_08411_amd", "csrc", f)) as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(config, layout):
    """HBM bytes per LM-head call (both kernels) from the committed
    rocprofv3 counter summary, or None when it is missing, was taken on
    another version of the kernel source or on the other weight layout."""
    path = os.path.join(ROOT, "profiles", f"lmhead_confidence_{config}_pmc.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    if rec.get("w_layout", "plain") != layout:
        return None
    return rec.get("hbm_bytes_per_launch")


def device_info():
    """Name, compute-unit count and clock of the GPU the run used (boxes of
    the same model differ; the per-box context helps read the numbers)."""
    import torch
    pr = torch.cuda.get_device_properties(0)
    info = {"name": pr.name, "cus": pr.multi_processor_count}
    for key in ("gcnArchName", "clock_rate", "memory_clock_rate"):
        if hasattr(pr, key):
            info[key] = getattr(pr, key)
    return info


def host_cpu():
    """(CPUs this process may run on, CPU model string) of the host."""
    n = len(os.sched_getaffinity(0))
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return n, model


def cpu_baseline(s, min_seconds=8.0):
    """The oracle as it stands on a bounded sample of the workload, repeated
    until min_seconds have passed: every attention head of up to 256 lane
    query rows (all of them at the LLaDA shape; otherwise spread over the
    lanes), up to 128 masked rows of the LM head over the whole vocabulary
    (all 77 at the LLaDA shape) and the full selection step; the sampled
    parts are scaled to the whole step.  Timed twice: the fp64 oracle
    (`value`) and its fp32 twin (the same code at fp32).  Inputs are widened
    from bf16 before the clock starts (the GPU path also starts with its
    inputs resident).  BLAS runs on every CPU of the process's affinity
    set, capped by OMP_NUM_THREADS when that is set (the host's share)."""
    import numpy as np
    import oracle
    import synth
    affinity, model = host_cpu()
    threads = affinity
    if os.environ.get("OMP_NUM_THREADS", "").isdigit():
        threads = min(threads, int(os.environ["OMP_NUM_THREADS"]))
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        limiter = threadpool_limits(limits=threads)
        used = max([int(x.get("num_threads", 1)) for x in threadpool_info()] or [1])
    except Exception:
        limiter, used = None, threads
    f32 = synth.bf16_bits_to_f32
    LB = s.L * s.B
    if LB <= 256:
        rows = list(range(LB))
    else:
        per = max(1, 256 // s.L)
        rows = sorted({i * s.B + int(a) for i in range(s.L)
                       for a in np.linspace(0, s.B - 1, per).astype(int)})
    nlm = min(128, s.N)
    depth = depth_of(s.parent)
    f_attn = sum(4.0 * s.D * (s.P + s.B * (depth[r // s.B] + 1)) for r in rows) * s.Hq
    f_lm = 2.0 * nlm * s.d * s.V

    def run(dtype):
        q, kl, vl, kp, vp, H, W = (f32(x).astype(dtype) for x in
                                   (s.q, s.k_lane, s.v_lane, s.k_pre, s.v_pre, s.hidden, s.W))
        t_attn = t_lm = t_sel = 0.0
        reps = 0
        t_start = time.perf_counter()
        while reps == 0 or time.perf_counter() - t_start < min_seconds:
            t0 = time.perf_counter()
            oracle.attention.lane_attention_rows(q, kl, vl, kp, vp, s.parent, s.B, rows, dtype=dtype)
            t1 = time.perf_counter()
            ref = oracle.lmhead.lmhead_confidence_full(H, s.row_pos[:nlm], W, s.suppress_eos[:nlm],
                                                       s.eos_id, dtype=dtype)
            t2 = time.perf_counter()
            conf = np.zeros(s.N)
            arg = np.zeros(s.N, dtype=np.int64)
            conf[:nlm], arg[:nlm] = ref["conf"], ref["argmax"]
            oracle.select.select_unmask(conf, arg, s.row_pos, s.tokens, s.is_masked, s.B, s.role,
                                        s.b_len, s.t_lane, 0, s.tau, s.fallback_k)
            t3 = time.perf_counter()
            t_attn, t_lm, t_sel = t_attn + t1 - t0, t_lm + t2 - t1, t_sel + t3 - t2
            reps += 1
        # Each part scaled to the whole step's work, seconds per call.
        per_call = {"lane_attn_forward": t_attn / reps * attention_flops(s) / f_attn,
                    "lmhead_confidence": t_lm / reps * lmhead_flops(s) / f_lm,
                    "select_unmask": t_sel / reps}
        t_step = sum(per_call.values())
        return ((attention_flops(s) + lmhead_flops(s)) / t_step / 1e12,
                {k: round(v, 4) for k, v in per_call.items()}, reps, t_attn + t_lm + t_sel)

    v64, pc64, reps64, sec64 = run(np.float64)
    v32, pc32, reps32, sec32 = run(np.float32)
    if limiter is not None:
        limiter.restore_original_limits()
    return {
        "value": v64,
        "unit": "TFLOP/s",
        "cores": used,
        "kind": "oracle",
        "sample": f"fp64 oracle: all {s.Hq} heads of {len(rows)} of {LB} lane query rows, "
                  f"{nlm} of {s.N} masked LM-head rows over all {s.V} vocab ids, full selection; "
                  f"{reps64} repetitions in {sec64:.1f} s, scaled to one step",
        "cpu_model": model,
        "affinity_cpus": affinity,
        "blas_threads": used,
        "seconds_per_call": pc64,
        "fp32_twin": {"value": v32, "unit": "TFLOP/s", "seconds_per_call": pc32,
                      "sample": f"the same sample in fp32; {reps32} repetitions in {sec32:.1f} s"},
    }


def decode_bench(args):
    """Whole decodes: the library scheduler (AlSched) plans each iteration,
    one lane_attn_forward runs per prefix-state group, lmhead_confidence
    scores the masked block rows, select_unmask transfers / drafts and
    computes the lane statistics, and the scheduler commits (one host round
    trip per iteration).  Synthetic model: seeded Q/K/V pools and hidden
    rows; the workload's W with the delimiter rows scaled by 2.5 and the
    EOS row by 1.8, so forks and cascade stops occur."""
    import numpy as np
    import torch

    import paper_2606_08411_amd as al
    import synth

    s = synth.make_step(args.config, args.seed)
    dev = torch.device("cuda:0")
    rng = np.random.default_rng([args.seed, 77])
    L, B, window = args.decode_len, s.B, s.B
    Wb = B + window

    def bf(a):
        return torch.from_numpy(synth.f32_to_bf16_bits(np.asarray(a, np.float32)).view(np.int16)) \
            .view(torch.bfloat16).to(dev)

    W = torch.from_numpy(np.ascontiguousarray(s.W).view(np.int16)).view(torch.bfloat16).to(dev)
    W[0:2] *= 2.5
    W[2] *= 1.8
    W_packed = al.lmhead_pack_weight(W) if args.w_layout == "packed" else None
    H = bf(rng.standard_normal((4 * L, s.d)) * rng.uniform(1, 6, (4 * L, 1)))
    pool = lambda n, h: bf(rng.standard_normal((n, h, s.D)))
    q, kl, vl = pool(64 * Wb, s.Hq), pool(64 * Wb, s.Hkv), pool(64 * Wb, s.Hkv)
    kp, vp = pool(s.P + L, s.Hkv), pool(s.P + L, s.Hkv)

    # Host <-> device traffic per iteration goes through one pinned staging
    # buffer: one upload (row ids, rows, suppress flags, tokens, masks) and
    # one download (tokens, masks and lane statistics, adjacent sections the
    # selection updates in place), waited for once.  Separate synchronous
    # copies from pageable memory cost ~140 us per iteration.
    cap = 64 * Wb
    sec = [0]
    def section(nbytes):
        off = sec[0]
        sec[0] += -(-nbytes // 256) * 256
        return off
    o_ridx, o_rows, o_sup = section(4 * cap), section(4 * cap), section(cap)
    o_tok, o_msk, o_st = section(4 * cap), section(cap), section(4 * 64 * al.LANE_STATS)
    up_h = torch.empty(sec[0], dtype=torch.uint8, pin_memory=True)
    up_d = torch.empty(sec[0], dtype=torch.uint8, device=dev)
    up_np = up_h.numpy()
    down_h = torch.empty(sec[0] - o_tok, dtype=torch.uint8, pin_memory=True)
    down_np = down_h.numpy()
    # Device outputs allocated once (capacity-sized; each call uses a prefix).
    conf_d = torch.empty(cap, dtype=torch.float32, device=dev)
    arg_d = torch.empty(cap, dtype=torch.int32, device=dev)
    sel_out = dict(unmask_flag=torch.empty(cap, dtype=torch.uint8, device=dev),
                   unmasked_pos=torch.empty(cap, dtype=torch.int32, device=dev),
                   still_masked_pos=torch.empty(cap, dtype=torch.int32, device=dev),
                   counts=torch.empty(2, dtype=torch.int32, device=dev),
                   lane_stats=up_d[o_st:].view(torch.int32).view(64, al.LANE_STATS),
                   delim_flag=None)

    def one_decode():
        S = al.AlSched(s.P, L, B, window, 64)
        attn_calls = 0
        for it in range(100000):
            pl = S.plan()
            n = len(pl["lane_id"])
            if n == 0:
                break
            tk, mk = S.blocks()
            for grp in sorted(set(pl["group"].tolist())):
                idx = [k for k in range(n) if pl["group"][k] == grp]
                parent = [idx.index(pl["call_parent"][k]) if pl["call_parent"][k] >= 0 else -1
                          for k in idx]
                Pg = s.P + int(min(pl["start"][k] for k in idx))
                m = len(idx) * Wb
                al.lane_attn_forward(q[:m], kl[:m], vl[:m], kp[:Pg], vp[:Pg], parent, Wb,
                                     want_lse=False)
                attn_calls += 1
            rows = np.flatnonzero(mk).astype(np.int32)
            nr, nb = len(rows), n * Wb
            up_np[o_ridx:o_ridx + 4 * nr].view(np.int32)[:] = \
                (it % 4) * L + pl["start"][rows // Wb] + rows % Wb
            up_np[o_rows:o_rows + 4 * nr].view(np.int32)[:] = rows
            up_np[o_tok:o_tok + 4 * nb].view(np.int32)[:] = tk
            up_np[o_sup:o_sup + nr] = pl["role"][rows // Wb] == al.ROLE_REF
            up_np[o_msk:o_msk + nb] = mk
            up_d[:o_st].copy_(up_h[:o_st], non_blocking=True)
            row_idx = up_d[o_ridx:o_ridx + 4 * nr].view(torch.int32)
            rows_d = up_d[o_rows:o_rows + 4 * nr].view(torch.int32)
            tok_d = up_d[o_tok:o_tok + 4 * nb].view(torch.int32)
            sup = up_d[o_sup:o_sup + nr]
            msk_d = up_d[o_msk:o_msk + nb]
            if W_packed is not None:
                conf, arg, _ = al.lmhead_confidence_packed(H, W_packed, s.V, row_idx=row_idx,
                                                           suppress_eos=sup, eos_id=s.eos_id,
                                                           conf=conf_d, argmax=arg_d, want_lse=False)
            else:
                conf, arg, _ = al.lmhead_confidence(H, W, row_idx=row_idx, suppress_eos=sup,
                                                    eos_id=s.eos_id, conf=conf_d, argmax=arg_d,
                                                    want_lse=False)
            al.select_unmask(conf, arg, rows_d, tok_d, msk_d, n, Wb,
                             pl["role"], pl["b_len"], pl["t_step"], al.MODE_THRESHOLD, s.tau,
                             1, None, s.delim_ids, s.eos_id, s.rho_min, s.t_min,
                             tau_future=s.tau, with_delim_flag=False, out=sel_out)
            down_h.copy_(up_d[o_tok:], non_blocking=True)
            torch.cuda.current_stream().synchronize()
            S.commit(down_np[:4 * nb].view(np.int32), down_np[o_msk - o_tok:o_msk - o_tok + nb],
                     down_np[o_st - o_tok:o_st - o_tok + 4 * n * al.LANE_STATS].view(np.int32))
        return S, attn_calls

    one_decode()   # warm-up
    torch.cuda.synchronize()
    runs = []
    for _ in range(args.decode_runs):
        t0 = time.perf_counter()
        S, calls = one_decode()
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        runs.append((dt, S, calls))
    dt = sorted(r[0] for r in runs)[len(runs) // 2]
    S = runs[0][1]
    c = S.counters()
    n_out = len(S.collect(s.eos_id))
    print(json.dumps({
        "metric": "synthetic active-lane decode, committed tokens/s (scheduler + 3 device calls)",
        "value": round(n_out / dt, 1), "unit": "tokens/s", "n_gpus": 1,
        "higher_is_better": True, "data": "synthetic",
        "config": {"workload": WORKLOAD_NAMES[args.config] + f"; decode of {L} positions, block "
                   f"{B}, lookahead window {window}, delimiter rows of W x2.5, EOS row x1.8, "
                   f"{args.w_layout} LM-head weight",
                   "name": args.config, "seed": args.seed, "L_gen": L, "B": B, "window": window},
        "ms_per_decode": round(dt * 1000, 3), "runs": args.decode_runs,
        "iterations": c["iterations"], "nfe": c["nfe"], "forks": c["forks"],
        "spawns": c["spawns"], "stops": c["stops"], "lanes": c["lanes"],
        "committed_tokens": n_out, "ms_per_iteration": round(dt * 1000 / c["iterations"], 3),
    }))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); "
              "this build has no multi-GPU path", file=sys.stderr)
        sys.exit(2)
    if args.decode:
        decode_bench(args)
        return
    import numpy as np
    import torch

    import paper_2606_08411_amd as al
    import synth

    s = synth.make_step(args.config, args.seed)
    dev = torch.device("cuda:0")

    def bf(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

    q, kl, vl = bf(s.q), bf(s.k_lane), bf(s.v_lane)
    kp, vp = bf(s.k_pre), bf(s.v_pre)
    hidden, W = bf(s.hidden), bf(s.W)
    row_pos = torch.from_numpy(s.row_pos).to(dev)
    sup = torch.from_numpy(s.suppress_eos).to(dev)
    n_ref = s.n_ref
    ref_args = {}
    if n_ref:
        ref_args = dict(refresh_idx=torch.from_numpy(s.refresh_idx).to(dev), q_ref=bf(s.q_ref),
                        k_ref=bf(s.k_ref), v_ref=bf(s.v_ref))
    o = torch.empty_like(q)
    lse = torch.empty((q.shape[0], s.Hq), dtype=torch.float32, device=dev)
    o_ref = torch.empty_like(ref_args["q_ref"]) if n_ref else None
    lse_ref = torch.empty((n_ref, s.Hq), dtype=torch.float32, device=dev) if n_ref else None
    conf = torch.empty(s.N, dtype=torch.float32, device=dev)
    arg = torch.empty(s.N, dtype=torch.int32, device=dev)
    lm_lse = torch.empty(s.N, dtype=torch.float32, device=dev)
    nsteps = args.warmup + args.steps
    # One fresh (tokens, is_masked) pair per step of the main loop and of
    # the per-step distribution pass, so every step selects on the same state.
    toks = [torch.from_numpy(s.tokens).to(dev) for _ in range(nsteps + args.steps)]
    msks = [torch.from_numpy(s.is_masked).to(dev) for _ in range(nsteps + args.steps)]
    sel_out = None

    ws_attn = torch.empty(max(16, al.lane_attn_workspace_size(s.L, s.B, s.P, s.Hq, s.Hkv, s.D,
                                                              n_ref)), dtype=torch.uint8, device=dev)
    ws_lm = torch.empty(max(16, al.lmhead_confidence_workspace_size(s.N, s.d, s.V)),
                        dtype=torch.uint8, device=dev)

    def attn():
        al.lane_attn_forward(q, kl, vl, kp, vp, s.parent, s.B, o=o, lse=lse, o_ref=o_ref,
                             lse_ref=lse_ref, workspace=ws_attn, **ref_args)

    # The packed weight is made once, outside the timed region: weights do
    # not change between decode steps.
    W_packed = al.lmhead_pack_weight(W) if args.w_layout == "packed" else None

    def lm_plain():
        al.lmhead_confidence(hidden, W, row_idx=row_pos, suppress_eos=sup, eos_id=s.eos_id,
                             conf=conf, argmax=arg, lse=lm_lse, workspace=ws_lm)

    def lm_packed():
        al.lmhead_confidence_packed(hidden, W_packed, s.V, row_idx=row_pos, suppress_eos=sup,
                                    eos_id=s.eos_id, conf=conf, argmax=arg, lse=lm_lse,
                                    workspace=ws_lm)

    lm = lm_packed if W_packed is not None else lm_plain

    def select(i):
        nonlocal sel_out
        sel_out = al.select_unmask(conf, arg, row_pos, toks[i], msks[i], s.L, s.B, s.role, s.b_len,
                                   s.t_lane, al.MODE_THRESHOLD, s.tau, s.fallback_k,
                                   delim_ids=s.delim_ids, eos_id=s.eos_id, rho_min=s.rho_min,
                                   t_min=s.t_min, out=sel_out)

    def step(i):
        attn()
        lm()
        select(i)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(args.warmup, nsteps):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps

    # Per-call averages (each call enqueues on torch's current stream; the
    # LM head is a single kernel launch).
    def timed(fn, reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    reps = args.kernel_reps
    t_attn = timed(attn, reps)
    t_lm = timed(lm, reps)
    t_lm_other = timed(lm_plain, reps) if W_packed is not None else None
    t_sel = timed(lambda: select(nsteps - 1), reps)

    def pct(xs):
        xs = sorted(xs)
        return [round(xs[int(q * (len(xs) - 1) + 0.5)], 4) for q in (0.1, 0.5, 0.9)]

    def per_rep(fn, n):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(n)]
        torch.cuda.synchronize()
        for k, (a, b) in enumerate(evs):
            a.record(stream)
            fn(k)
            b.record(stream)
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in evs]

    def extra_passes():
        # Distributions: whole steps (fresh selection state each), LM-head calls.
        step_p = pct(per_rep(lambda k: step(nsteps + k), args.steps))
        lm_p = pct(per_rep(lambda k: lm(), reps))
        # The selection outcome of one step on fresh state (committed tokens).
        n_commit = int(sel_out["counts"][0].item())

        # Cold attention: rotate over copies of the attention inputs whose total
        # exceeds the 256 MB last-level cache, so no call finds its K/V cached.
        set_bytes = sum(t.numel() * t.element_size() for t in (q, kl, vl, kp, vp))
        n_sets = max(4, -(-512 * 2**20 // set_bytes))
        sets = [tuple(t.clone() for t in (q, kl, vl, kp, vp)) for _ in range(n_sets)]

        def attn_set(k):
            qq, kk, vv, kpp, vpp = sets[k % n_sets]
            al.lane_attn_forward(qq, kk, vv, kpp, vpp, s.parent, s.B, o=o, lse=lse, o_ref=o_ref,
                                 lse_ref=lse_ref, workspace=ws_attn, **ref_args)

        for k in range(n_sets):
            attn_set(k)
        it = iter(range(10**9))
        t_attn_cold = timed(lambda: attn_set(next(it)), max(reps, 2 * n_sets))
        del sets

        # HIP-graph replays (no host launch cost): the whole step, and each call
        # captured 20 times in one graph.  The captured selection works on one
        # (tokens, is_masked) pair, so later replays select on the evolving state.
        graph = None
        try:
            tk_g, mk_g = toks[0].clone(), msks[0].clone()
            sel_g = al.select_unmask(conf, arg, row_pos, tk_g, mk_g, s.L, s.B, s.role, s.b_len,
                                     s.t_lane, al.MODE_THRESHOLD, s.tau, s.fallback_k,
                                     delim_ids=s.delim_ids, eos_id=s.eos_id, rho_min=s.rho_min,
                                     t_min=s.t_min)

            def select_g():
                al.select_unmask(conf, arg, row_pos, tk_g, mk_g, s.L, s.B, s.role, s.b_len,
                                 s.t_lane, al.MODE_THRESHOLD, s.tau, s.fallback_k,
                                 delim_ids=s.delim_ids, eos_id=s.eos_id, rho_min=s.rho_min,
                                 t_min=s.t_min, out=sel_g)

            def graph_ms(body, calls, n_rep):
                g = torch.cuda.CUDAGraph()
                torch.cuda.synchronize()
                with torch.cuda.graph(g):
                    for _ in range(calls):
                        body()
                for _ in range(3):
                    g.replay()
                torch.cuda.synchronize()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                for _ in range(n_rep):
                    g.replay()
                b.record()
                torch.cuda.synchronize()
                return a.elapsed_time(b) / (n_rep * calls)

            graph = {
                "ms_per_step": round(graph_ms(lambda: (attn(), lm(), select_g()), 1, args.steps), 4),
                "per_call_ms": {"lane_attn_forward": round(graph_ms(attn, 20, 10), 4),
                                "lmhead_confidence": round(graph_ms(lm, 5, 10), 4),
                                "select_unmask": round(graph_ms(select_g, 20, 10), 4)},
            }
        except Exception as e:   # reported, never silent
            graph = {"error": f"{type(e).__name__}: {e}"}
        # The box's plain HBM copy rate (torch copy of 1 GiB: 2 GiB moved),
        # context for the LM-head fraction; boxes of one model differ.
        src = torch.empty(2**30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        copy_ms = timed(lambda: dst.copy_(src), 5)
        del src, dst
        return {
            "hbm_copy_gbs": round(2 * 2**30 / (copy_ms * 1e-3) / 1e9, 1),
            "step_ms_p10_p50_p90": step_p,
            "lmhead_ms_p10_p50_p90": lm_p,
            "attention_cold_ms": round(t_attn_cold, 4),
            "attention_cold_sets": n_sets,
            "committed_tokens_per_step": n_commit,
            "committed_tokens_per_s": round(n_commit / (ms_step * 1e-3), 1),
            "graph": graph,
        }

    extras = extra_passes() if not args.quick else {}

    f_attn, f_lm = attention_flops(s), lmhead_flops(s)
    value = (f_attn + f_lm) / (ms_step * 1e-3) / 1e12
    lm_gbs = lmhead_bytes(s) / (t_lm * 1e-3) / 1e9
    traffic = measured_traffic(args.config, args.w_layout)
    out = {
        "metric": "lane-attn + fused LM-head TFLOP/s (MFMA util %), masked positions scored/s",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "device": device_info(),
        "config": {"workload": WORKLOAD_NAMES[args.config], "name": args.config, "seed": args.seed,
                   "L": s.L, "B": s.B, "P": s.P, "Hq": s.Hq, "Hkv": s.Hkv, "D": s.D, "d": s.d,
                   "V": s.V, "N_masked": s.N, "n_refresh": n_ref},
        "mfma_util_pct": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "masked_positions_per_s": round(s.N / (ms_step * 1e-3), 1),
        "lane_tokens_per_s": round(s.L * s.B / (ms_step * 1e-3), 1),
        "per_call_ms": {"lane_attn_forward": round(t_attn, 4), "lmhead_confidence": round(t_lm, 4),
                        "select_unmask": round(t_sel, 4)},
        "lm_weight_layout": args.w_layout,
        "lmhead_plain_weight_ms": None if t_lm_other is None else round(t_lm_other, 4),
        **extras,
        "attention_tflops": round(f_attn / (t_attn * 1e-3) / 1e12, 2),
        "lmhead_tflops": round(f_lm / (t_lm * 1e-3) / 1e12, 2),
        "roofline": {
            "kernel": ("lmhead_confidence_packed" if W_packed is not None else "lmhead_confidence")
                      + " (lmhead_partial_kernel + lmhead_merge_kernel)",
            "bound": "hbm",
            "achieved": round(lm_gbs, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(lm_gbs / PEAK_HBM_GBS, 4),
            "traffic": traffic,
        },
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(s)
        out["cpu_baseline"]["gpu_over_oracle"] = round(value / out["cpu_baseline"]["value"], 1)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
