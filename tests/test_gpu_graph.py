"""The three calls captured in one HIP graph and replayed: every replay must
reproduce the eager results bit for bit (the kernels are deterministic and
the graph holds the same launches).

Between replays the test runs eager work of its own (a fresh eager step on
other buffers) and synchronises; the selection state is reset by an eager
copy before each replay, so every replay selects on the same input state.
The Wide workload includes the compact-refresh scatter, which rewrites the
same prefix rows with the same values on every replay.  The graph holds
kernel launches only (no memset nodes).
"""
import numpy as np
import pytest
import torch

import synth
from gpu_util import dev, dev_bf16

pytestmark = pytest.mark.gpu


def _inputs(name, seed):
    s = synth.make_step(name, seed)
    t = dict(q=dev_bf16(s.q), kl=dev_bf16(s.k_lane), vl=dev_bf16(s.v_lane),
             kp=dev_bf16(s.k_pre), vp=dev_bf16(s.v_pre), hidden=dev_bf16(s.hidden),
             W=dev_bf16(s.W), row_pos=dev(s.row_pos), sup=dev(s.suppress_eos),
             tok0=dev(s.tokens), msk0=dev(s.is_masked))
    if s.n_ref:
        t.update(ridx=dev(s.refresh_idx), q_ref=dev_bf16(s.q_ref), k_ref=dev_bf16(s.k_ref),
                 v_ref=dev_bf16(s.v_ref))
    return s, t


class _Step:
    """Preallocated outputs and one step (attention, LM head, selection)."""

    def __init__(self, s, t):
        import paper_2606_08411_amd as al
        self.al, self.s, self.t = al, s, t
        LB = s.L * s.B
        self.o = torch.empty_like(t["q"])
        self.lse = torch.empty((LB, s.Hq), dtype=torch.float32, device="cuda")
        self.o_ref = torch.empty_like(t["q_ref"]) if s.n_ref else None
        self.lse_ref = (torch.empty((s.n_ref, s.Hq), dtype=torch.float32, device="cuda")
                        if s.n_ref else None)
        self.conf = torch.empty(s.N, dtype=torch.float32, device="cuda")
        self.arg = torch.empty(s.N, dtype=torch.int32, device="cuda")
        self.lm_lse = torch.empty(s.N, dtype=torch.float32, device="cuda")
        self.tok = t["tok0"].clone()
        self.msk = t["msk0"].clone()
        self.sel = None
        # explicit workspaces: the binding refuses its default ones while a
        # graph is being captured
        ws = al.lane_attn_workspace_size(s.L, s.B, s.P, s.Hq, s.Hkv, s.D, s.n_ref)
        self.ws_attn = torch.empty(max(ws, 16), dtype=torch.uint8, device="cuda")
        self.ws_lm = torch.empty(al.lmhead_confidence_workspace_size(s.N, s.d, s.V),
                                 dtype=torch.uint8, device="cuda")

    def __call__(self):
        al, s, t = self.al, self.s, self.t
        ref = {}
        if s.n_ref:
            ref = dict(refresh_idx=t["ridx"], q_ref=t["q_ref"], k_ref=t["k_ref"], v_ref=t["v_ref"],
                       o_ref=self.o_ref, lse_ref=self.lse_ref)
        al.lane_attn_forward(t["q"], t["kl"], t["vl"], t["kp"], t["vp"], s.parent, s.B,
                             o=self.o, lse=self.lse, workspace=self.ws_attn, **ref)
        al.lmhead_confidence(t["hidden"], t["W"], row_idx=t["row_pos"], suppress_eos=t["sup"],
                             eos_id=s.eos_id, conf=self.conf, argmax=self.arg, lse=self.lm_lse,
                             workspace=self.ws_lm)
        self.sel = al.select_unmask(self.conf, self.arg, t["row_pos"], self.tok, self.msk, s.L,
                                    s.B, s.role, s.b_len, s.t_lane, al.MODE_THRESHOLD, s.tau,
                                    s.fallback_k, delim_ids=s.delim_ids, eos_id=s.eos_id,
                                    rho_min=s.rho_min, t_min=s.t_min, out=self.sel)

    def reset(self):
        self.tok.copy_(self.t["tok0"])
        self.msk.copy_(self.t["msk0"])

    def snapshot(self):
        out = [self.o, self.lse, self.conf, self.arg, self.lm_lse, self.tok, self.msk]
        out += [v for k, v in sorted(self.sel.items()) if v is not None]
        if self.o_ref is not None:
            out += [self.o_ref, self.lse_ref]
        return [x.clone() for x in out]


@pytest.mark.parametrize("name", ["tiny", "llada", "wide"])
def test_graph_replays_match_eager(name):
    s, t = _inputs(name, 0)
    st = _Step(s, t)
    st()                      # eager reference
    torch.cuda.synchronize()
    st.reset()
    st()
    torch.cuda.synchronize()
    want = st.snapshot()

    other = _Step(*_inputs(name, 1))   # eager work between replays
    other()

    g = torch.cuda.CUDAGraph()
    st.reset()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        st()
    torch.cuda.synchronize()
    for rep in range(3):
        st.reset()
        other.reset()
        other()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = st.snapshot()
        assert len(got) == len(want)
        for a, b in zip(got, want):
            assert torch.equal(a, b), f"replay {rep} differs from the eager step"
