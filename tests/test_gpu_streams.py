"""Calls on two streams at once, with the binding's default workspaces.

The binding keeps one default workspace per (kind, device, stream), so
lane_attn_forward (key-split pass, partials in the workspace) and
lmhead_confidence (per-vocab-tile partials) enqueued on two ordinary
streams concurrently must reproduce the serial results bit for bit.
"""
import numpy as np
import pytest
import torch

import synth
from gpu_util import dev, dev_bf16

pytestmark = pytest.mark.gpu


def _problem(seed):
    s = synth.make_step("long", seed, with_weight=False)   # shared-staging kernel with key splits
    g = np.random.default_rng([seed, 3])
    N, d, V = 205, 1024, 70000
    H = synth.f32_to_bf16_bits(g.standard_normal((300, d), dtype=np.float32) *
                               g.uniform(1, 6, (300, 1)).astype(np.float32))
    W = synth.f32_to_bf16_bits(g.standard_normal((V, d), dtype=np.float32) / np.float32(32))
    t = dict(q=dev_bf16(s.q), kl=dev_bf16(s.k_lane), vl=dev_bf16(s.v_lane), kp=dev_bf16(s.k_pre),
             vp=dev_bf16(s.v_pre), H=dev_bf16(H), W=dev_bf16(W),
             ridx=dev(np.sort(g.choice(300, N, replace=False)).astype(np.int32)))
    out = dict(o=torch.empty_like(t["q"]), lse=torch.empty(s.L * s.B, s.Hq, device="cuda"),
               conf=torch.empty(N, device="cuda"), arg=torch.empty(N, dtype=torch.int32, device="cuda"),
               lm_lse=torch.empty(N, device="cuda"))
    return s, t, out


def _run(s, t, out):
    import paper_2606_08411_amd as al
    al.lane_attn_forward(t["q"], t["kl"], t["vl"], t["kp"], t["vp"], s.parent, s.B, o=out["o"],
                         lse=out["lse"])
    al.lmhead_confidence(t["H"], t["W"], row_idx=t["ridx"], eos_id=-1, conf=out["conf"],
                         argmax=out["arg"], lse=out["lm_lse"])


def test_two_streams_match_serial():
    import paper_2606_08411_amd as al
    assert al.lane_attn_workspace_size(16, 32, 2048, 32, 32, 128, 0) > 0   # the split pass
    probs = [_problem(1), _problem(2)]
    for p in probs:
        _run(*p)
    torch.cuda.synchronize()
    want = [{k: v.clone() for k, v in p[2].items()} for p in probs]
    for p in probs:
        for v in p[2].values():
            v.zero_()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for _ in range(6):
        for st, p in zip(streams, probs):
            with torch.cuda.stream(st):
                _run(*p)
    torch.cuda.synchronize()
    for p, w in zip(probs, want):
        for k, v in p[2].items():
            assert torch.equal(v, w[k]), f"{k} differs from the serial result"
