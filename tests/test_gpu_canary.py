"""Unwritten outputs and out-of-bounds writes (canaries and guard bands).

Every output buffer is the front part of a larger allocation: the part the
call owns is prefilled with a canary (NaN bits for bf16 / fp32, an
impossible value for integers) and the guard band after it with a second
pattern.  After the call no canary may remain where the call defines a
value, and every guard band (outputs, in/out buffers, explicit workspaces)
must be untouched.  Each call also runs twice on the same inputs, which
must give bitwise identical outputs.  Cases: the five workloads and the
edges of the supported shapes (B = 1024, L = 64, P = 0, N = 0 and 1).
"""
import numpy as np
import pytest
import torch

import synth
from gpu_util import dev, dev_bf16

pytestmark = pytest.mark.gpu
GUARD = 4096          # elements after every buffer
GUARD_BYTE = 0x5A


class Guarded:
    """A buffer of n elements followed by GUARD guard elements."""

    def __init__(self, n, dtype, canary):
        self.n = int(n)
        self.full = torch.empty(self.n + GUARD, dtype=dtype, device="cuda")
        raw = self.full.view(torch.uint8)
        raw.fill_(GUARD_BYTE)
        self.full[:self.n].view(torch.uint8).fill_(canary)
        self.guard_ref = raw[self.n * self.full.element_size():].clone()

    def view(self, *shape):
        return self.full[:self.n].view(*shape) if shape else self.full[:self.n]

    def guard_ok(self):
        return torch.equal(self.full.view(torch.uint8)[self.n * self.full.element_size():],
                           self.guard_ref)


def guarded_copy(t):
    """An input/output tensor copied into a guarded buffer."""
    g = Guarded(t.numel(), t.dtype, 0)
    g.view().copy_(t.reshape(-1))
    return g


def _attn_case(step):
    import paper_2606_08411_amd as al
    LB, Hq, Hkv, D, P, n_ref = step.L * step.B, step.Hq, step.Hkv, step.D, step.P, step.n_ref
    kp = guarded_copy(dev_bf16(step.k_pre))
    vp = guarded_copy(dev_bf16(step.v_pre))
    o = Guarded(LB * Hq * D, torch.bfloat16, 0xFF)
    lse = Guarded(LB * Hq, torch.float32, 0xFF)
    ref = {}
    bufs = [o, lse, kp, vp]
    if n_ref:
        o_r = Guarded(n_ref * Hq * D, torch.bfloat16, 0xFF)
        lse_r = Guarded(n_ref * Hq, torch.float32, 0xFF)
        bufs += [o_r, lse_r]
        ref = dict(refresh_idx=dev(step.refresh_idx), q_ref=dev_bf16(step.q_ref),
                   k_ref=dev_bf16(step.k_ref), v_ref=dev_bf16(step.v_ref),
                   o_ref=o_r.view(n_ref, Hq, D), lse_ref=lse_r.view(n_ref, Hq))
    need = al.lane_attn_workspace_size(step.L, step.B, P, Hq, Hkv, D, n_ref)
    ws = Guarded(max(need, 16), torch.uint8, 0xFF)
    bufs.append(ws)
    al.lane_attn_forward(dev_bf16(step.q), dev_bf16(step.k_lane), dev_bf16(step.v_lane),
                         kp.view(P, Hkv, D), vp.view(P, Hkv, D), step.parent, step.B,
                         o=o.view(LB, Hq, D), lse=lse.view(LB, Hq), workspace=ws.view(), **ref)
    torch.cuda.synchronize()
    assert all(b.guard_ok() for b in bufs), "a guard band was written"
    outs = [o.view(), lse.view()] + ([ref["o_ref"], ref["lse_ref"]] if n_ref else [])
    for t in outs:
        assert not torch.isnan(t.float()).any(), "an output element was left unwritten"
    return [t.clone() for t in outs] + [kp.view().clone(), vp.view().clone()]


ATTN_EDGES = [  # D, B, L, tree, Hq, Hkv, P, refresh_frac
    (64, 1024, 2, "fork", 16, 1, 64, 0.0),     # largest block
    (128, 32, 64, "random", 8, 2, 96, 0.1),    # most lanes, with refresh rows
    (64, 16, 64, "forest", 4, 4, 31, 0.0),     # most lanes, wavefront-split kernel
    (128, 32, 3, "linear", 4, 1, 0, 0.0),      # no prefix
]


@pytest.mark.parametrize("case", ["tiny", "llada", "dream", "long", "wide"] + ATTN_EDGES,
                         ids=str)
def test_attention_canaries(case, step_cache):
    if isinstance(case, str):
        step = step_cache(case, 0, with_weight=False)
    else:
        D, B, L, tree, Hq, Hkv, P, rf = case
        step = synth.make_step("tiny", 5, with_weight=False, D=D, B=B, L=L, tree=tree, Hq=Hq,
                               Hkv=Hkv, P=P, refresh_frac=rf, depth_max=4, V=64, d=64)
    a = _attn_case(step)
    b = _attn_case(step)
    for x, y in zip(a, b):
        assert torch.equal(x, y), "two runs differ"


def _lm_case(H, W, ridx, sup, eos, Wp=None):
    import paper_2606_08411_amd as al
    N = ridx.shape[0]
    conf = Guarded(N, torch.float32, 0xFF)
    arg = Guarded(N, torch.int32, 0xFF)        # -1: not a token id
    lse = Guarded(N, torch.float32, 0xFF)
    need = al.lmhead_confidence_workspace_size(N, H.shape[1], W.shape[0])
    ws = Guarded(max(need, 16), torch.uint8, 0xFF)
    outs = dict(row_idx=ridx, suppress_eos=sup, eos_id=eos, conf=conf.view(), argmax=arg.view(),
                lse=lse.view(), workspace=ws.view())
    if Wp is None:
        al.lmhead_confidence(H, W, **outs)
    else:
        al.lmhead_confidence_packed(H, Wp, W.shape[0], **outs)
    torch.cuda.synchronize()
    assert all(b.guard_ok() for b in (conf, arg, lse, ws)), "a guard band was written"
    assert not torch.isnan(conf.view()).any() and not torch.isnan(lse.view()).any()
    assert ((arg.view() >= 0) & (arg.view() < W.shape[0])).all()
    return [conf.view().clone(), arg.view().clone(), lse.view().clone()]


@pytest.mark.parametrize("case", ["tiny", "llada", "dream", "long", "wide",
                                  (1, 5, 264, 4097, 2), (0, 5, 264, 4097, 2),
                                  (225, 300, 64, 70000, 1)], ids=str)
def test_lmhead_canaries(case, step_cache):
    if isinstance(case, str):
        s = step_cache(case, 0)
        H, W, ridx, sup, eos = (dev_bf16(s.hidden), dev_bf16(s.W), dev(s.row_pos),
                                dev(s.suppress_eos), s.eos_id)
    else:
        N, n_rows, d, V, eos = case
        g = np.random.default_rng([N, d, V])
        H = dev_bf16(synth.f32_to_bf16_bits(g.standard_normal((n_rows, d), dtype=np.float32)))
        W = dev_bf16(synth.f32_to_bf16_bits(g.standard_normal((V, d), dtype=np.float32) * 0.1))
        ridx = dev(np.arange(N, dtype=np.int32))
        sup = dev((g.random(N) < 0.5).astype(np.uint8))
    a = _lm_case(H, W, ridx, sup, eos)
    b = _lm_case(H, W, ridx, sup, eos)
    for x, y in zip(a, b):
        assert torch.equal(x, y), "two runs differ"
    # the packed weight: its copy written into a guarded buffer, then the call
    import paper_2606_08411_amd as al
    wp = Guarded(al.lmhead_packed_weight_size(W.shape[1], W.shape[0]) // 2, torch.bfloat16, 0xFF)
    al.lmhead_pack_weight(W, out=wp.view())
    torch.cuda.synchronize()
    assert wp.guard_ok(), "the packed copy overran its buffer"
    assert not torch.isnan(wp.view().float()).any(), "part of the packed copy was left unwritten"
    a = _lm_case(H, W, ridx, sup, eos, Wp=wp.view())
    b = _lm_case(H, W, ridx, sup, eos, Wp=wp.view())
    for x, y in zip(a, b):
        assert torch.equal(x, y), "two runs differ (packed)"


def _sel_case(s, conf, arg, L, B, row_pos, tokens, masked):
    import paper_2606_08411_amd as al
    N, LB = len(row_pos), L * B
    tok = guarded_copy(dev(tokens))
    msk = guarded_copy(dev(masked))
    out = dict(unmask_flag=Guarded(N, torch.uint8, 0xFF), unmasked_pos=Guarded(N, torch.int32, 0xFF),
               still_masked_pos=Guarded(N, torch.int32, 0xFF), counts=Guarded(2, torch.int32, 0xFF),
               lane_stats=Guarded(L * 6, torch.int32, 0xFF), delim_flag=Guarded(LB, torch.uint8, 0xFF))
    views = {k: (v.view(L, 6) if k == "lane_stats" else v.view()) for k, v in out.items()}
    al.select_unmask(dev(conf), dev(arg), dev(row_pos), tok.view(), msk.view(), L, B,
                     np.zeros(L, np.uint8), None, np.full(L, 3, np.int32), al.MODE_THRESHOLD, 0.6, 1,
                     tau_future=0.5, out=views)
    torch.cuda.synchronize()
    assert all(b.guard_ok() for b in list(out.values()) + [tok, msk]), "a guard band was written"
    cu, cs = (int(x) for x in views["counts"].cpu())
    assert 0 <= cu <= N and 0 <= cs <= N and cu + cs <= N
    flags = views["unmask_flag"].cpu().numpy()
    assert np.isin(flags, [0, 1, 2]).all()
    assert np.isin(views["delim_flag"].cpu().numpy(), [0, 1]).all()
    assert (views["lane_stats"].cpu().numpy() != -1).all()
    assert (views["unmasked_pos"][:cu].cpu().numpy() >= 0).all()
    assert (views["still_masked_pos"][:cs].cpu().numpy() >= 0).all()
    res = [views[k].clone() for k in ("unmask_flag", "counts", "lane_stats", "delim_flag")]
    res += [views["unmasked_pos"][:cu].clone(), views["still_masked_pos"][:cs].clone(),
            tok.view().clone(), msk.view().clone()]
    return res


@pytest.mark.parametrize("case", ["tiny", "llada", "dream", "long", "wide",
                                  (64, 128, 0.5), (64, 32, 0.0), (1, 1, 1.0), (8, 100, 0.02)],
                         ids=str)
def test_select_canaries(case, step_cache):
    if isinstance(case, str):
        s = step_cache(case, 0, with_weight=False)
        L, B, row_pos, tokens, masked = s.L, s.B, s.row_pos, s.tokens, s.is_masked
    else:
        L, B, frac = case
        g = np.random.default_rng([L, B])
        masked = (g.random(L * B) < frac).astype(np.uint8)
        row_pos = np.flatnonzero(masked).astype(np.int32)
        tokens = g.integers(0, 6, L * B).astype(np.int32)
        s = None
    conf, arg = synth.random_confidences(4, len(row_pos), 50, tie_levels=8)
    a = _sel_case(s, conf, arg, L, B, row_pos, tokens, masked)
    b = _sel_case(s, conf, arg, L, B, row_pos, tokens, masked)
    for x, y in zip(a, b):
        assert torch.equal(x, y), "two runs differ"
