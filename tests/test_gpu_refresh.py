"""Compact cache refresh (Section 3.4, "Compact cache refresh and reuse") on
the GPU against the oracle.

The refresh forward is a refresh-only lane_attn_forward over the window
[0, L_refresh) with every window row refreshed: the cache rows of the
window are rewritten (bit-exact) and every refreshed query attends over the
whole window (bf16 outputs within 2e-2 of fp64, LSE within 2e-3).  The
refresh logits of the window's masked generation rows then drive the next
transfer without another LM-head pass; that selection must match the
oracle's bit for bit when both are fed the same (conf, argmax).
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


def _bf16(rng, shape, scale=1.0):
    return synth.f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


@pytest.mark.parametrize("Hq,Hkv,D", [(8, 4, 64), (28, 4, 128), (32, 32, 128)])
def test_refresh_window_forward(Hq, Hkv, D):
    import paper_2606_08411_amd as al
    rng = np.random.default_rng(Hq * 7 + D)
    P_prompt, L_gen, B = 300, 256, 32
    cap = P_prompt + L_gen                      # cache rows allocated
    starts = np.arange(0, L_gen, B)[:6]
    valid = np.array([B, B, 20, 7, 0, 0], np.int32)
    Lr = al.al_refresh_window(P_prompt, L_gen, starts, valid, 8)
    # frontier max(s + v) = 160 + 0 -> 300 + 160 + 8 = 468 (< P + L = 556)
    assert Lr == oracle.refresh.refresh_window_len(P_prompt, L_gen, starts, valid, 8) == 468
    k_cache = _bf16(rng, (cap, Hkv, D))
    v_cache = _bf16(rng, (cap, Hkv, D))
    q_ref = _bf16(rng, (Lr, Hq, D))
    k_ref = _bf16(rng, (Lr, Hkv, D))
    v_ref = _bf16(rng, (Lr, Hkv, D))
    kc, vc = dev_bf16(k_cache), dev_bf16(v_cache)
    idx = dev(np.arange(Lr, dtype=np.int32))
    _, _, o_ref, lse_ref = al.lane_attn_forward(None, None, None, kc[:Lr], vc[:Lr], [], 16,
                                                refresh_idx=idx, q_ref=dev_bf16(q_ref),
                                                k_ref=dev_bf16(k_ref), v_ref=dev_bf16(v_ref))
    torch.cuda.synchronize()
    kc_h, vc_h = host_bf16_f32(kc), host_bf16_f32(vc)
    assert np.array_equal(kc_h[:Lr], f32(k_ref)) and np.array_equal(vc_h[:Lr], f32(v_ref))
    assert np.array_equal(kc_h[Lr:], f32(k_cache)[Lr:]) and np.array_equal(vc_h[Lr:], f32(v_cache)[Lr:])
    o, lse = oracle.attention.refresh_attention(f32(q_ref), f32(k_ref), f32(v_ref))
    assert np.abs(host_bf16_f32(o_ref) - o).max() < TOL_O
    assert np.abs(lse_ref.cpu().numpy() - lse).max() < TOL_LSE


def test_refresh_logit_reuse():
    """Refresh logits of the window's masked generation rows drive the next
    transfer (and lookahead drafts) without a new LM-head pass."""
    import paper_2606_08411_amd as al
    rng = np.random.default_rng(9)
    P_prompt, L, B, d, V = 64, 4, 32, 256, 1024
    L_gen = L * B
    starts = np.arange(L) * B
    tokens = rng.integers(3, V, L_gen).astype(np.int32)
    masked = (rng.random(L_gen) < 0.6).astype(np.uint8)
    b_len = np.array([32, 32, 24, 16], np.int32)
    role = np.array([1, 1, 0, 0], np.uint8)
    valid = np.array([int(np.argmax(masked[l * B:l * B + b_len[l]])) if masked[l * B:l * B + b_len[l]].any()
                      else int(b_len[l]) for l in range(L)], np.int32)
    Lr = al.al_refresh_window(P_prompt, L_gen, starts, valid, 40)
    assert Lr == oracle.refresh.refresh_window_len(P_prompt, L_gen, starts, valid, 40)
    # window rows of masked generation positions, ascending
    pos = np.flatnonzero(masked)
    pos = pos[P_prompt + pos < Lr].astype(np.int32)
    row_idx = (P_prompt + pos).astype(np.int32)
    hidden = synth.f32_to_bf16_bits((rng.standard_normal((Lr, d)) *
                                     rng.uniform(1, 6, (Lr, 1))).astype(np.float32))
    W = synth.f32_to_bf16_bits((rng.standard_normal((V, d)) / np.sqrt(d)).astype(np.float32))
    sup = role[pos // B].astype(np.uint8)      # refine-lane rows suppress EOS
    conf, arg, _ = al.lmhead_confidence(dev_bf16(hidden), dev_bf16(W), row_idx=dev(row_idx),
                                        suppress_eos=dev(sup), eos_id=2)
    torch.cuda.synchronize()
    ref_lm = oracle.lmhead.lmhead_confidence_full(f32(hidden), row_idx, f32(W), sup, 2)
    assert np.abs(conf.cpu().numpy() - ref_lm["conf"]).max() < 2e-2
    c_h, a_h = conf.cpu().numpy(), arg.cpu().numpy()
    # next iteration: the cached (conf, argmax) feed the transfer and drafts
    tok_d, msk_d = dev(tokens), dev(masked)
    out = al.select_unmask(conf, arg, dev(pos), tok_d, msk_d, L, B, role, b_len, np.full(L, 3, np.int32),
                           al.MODE_THRESHOLD, 0.9, 1, None, (0, 1), 2, 0.5, 2, tau_future=0.5)
    torch.cuda.synchronize()
    ref = oracle.select.select_unmask(c_h, a_h, pos, tokens, masked, B, role, b_len,
                                      np.full(L, 3, np.int32), 0, 0.9, 1, None, (0, 1), 2, 0.5, 2,
                                      tau_future=0.5)
    cu, cs = out["counts"].cpu().numpy()
    assert [cu, cs] == list(ref["counts"])
    assert np.array_equal(out["unmask_flag"].cpu().numpy()[:len(pos)], ref["unmask_flag"])
    assert np.array_equal(tok_d.cpu().numpy(), ref["tokens"])
    assert np.array_equal(out["lane_stats"].cpu().numpy(), ref["lane_stats"])
