"""The Python binding rejects wrong dtypes, shapes and devices before
anything reaches the library (CPU tensors: no launch can happen here).

Each call first gets one wrong argument and must name it; a call whose
arguments are all well-formed but live on the host fails on the device
check, also before any launch.
"""
import pytest
import torch

import paper_2606_08411_amd as al
from paper_2606_08411_amd import AsyncLaneError

bf16 = torch.bfloat16


def _attn_args(L=2, B=16, P=32, Hq=4, Hkv=2, D=64):
    return dict(q=torch.zeros(L * B, Hq, D, dtype=bf16), k_lane=torch.zeros(L * B, Hkv, D, dtype=bf16),
                v_lane=torch.zeros(L * B, Hkv, D, dtype=bf16),
                k_prefix=torch.zeros(P, Hkv, D, dtype=bf16), v_prefix=torch.zeros(P, Hkv, D, dtype=bf16),
                parent=[-1, 0], B=B)


@pytest.mark.parametrize("key,bad,msg", [
    ("q", torch.zeros(32, 4, 64, dtype=torch.float32), "q: dtype"),
    ("q", torch.zeros(31, 4, 64, dtype=bf16), "q:"),
    ("q", torch.zeros(32, 4, 128, dtype=bf16), "q:"),
    ("k_lane", torch.zeros(32, 4, 64, dtype=bf16), "k_lane: shape"),
    ("v_lane", torch.zeros(32, 2, 64, dtype=torch.float16), "v_lane: dtype"),
    ("v_prefix", torch.zeros(33, 2, 64, dtype=bf16), "v_prefix: shape"),
    ("k_prefix", torch.zeros(32, 128, dtype=bf16), "k_prefix:"),
    ("o", torch.zeros(32, 4, 64, dtype=torch.float32), "o: dtype"),
    ("lse", torch.zeros(32, 3, dtype=torch.float32), "lse: shape"),
    ("workspace", "not a tensor", "device tensor expected|workspace"),
])
def test_attention_rejects(key, bad, msg):
    a = _attn_args()
    a[key] = bad
    with pytest.raises(AsyncLaneError, match=msg):
        al.lane_attn_forward(**a)


def test_attention_refresh_rejects():
    a = _attn_args()
    ref = dict(refresh_idx=torch.zeros(3, dtype=torch.int64), q_ref=torch.zeros(3, 4, 64, dtype=bf16),
               k_ref=torch.zeros(3, 2, 64, dtype=bf16), v_ref=torch.zeros(3, 2, 64, dtype=bf16))
    with pytest.raises(AsyncLaneError, match="refresh_idx: dtype"):
        al.lane_attn_forward(**a, **ref)
    ref["refresh_idx"] = torch.zeros(3, dtype=torch.int32)
    ref["k_ref"] = torch.zeros(3, 4, 64, dtype=bf16)
    with pytest.raises(AsyncLaneError, match="k_ref: shape"):
        al.lane_attn_forward(**a, **ref)


def test_attention_host_tensors_rejected():
    with pytest.raises(AsyncLaneError, match="device tensor expected"):
        al.lane_attn_forward(**_attn_args())


def _lm_args(n=8, d=64, V=100):
    return dict(hidden=torch.zeros(n, d, dtype=bf16), W=torch.zeros(V, d, dtype=bf16),
                row_idx=torch.arange(n, dtype=torch.int32))


@pytest.mark.parametrize("fn", [al.lmhead_confidence, al.lmhead_confidence_noalloc])
@pytest.mark.parametrize("key,bad,msg", [
    ("hidden", torch.zeros(8, 64, dtype=torch.float32), "hidden: dtype"),
    ("hidden", torch.zeros(8, 64, 1, dtype=bf16), "hidden:"),
    ("W", torch.zeros(100, 32, dtype=bf16), "W:"),
    ("row_idx", torch.arange(8, dtype=torch.int64), "row_idx: dtype"),
    ("row_idx", torch.zeros(2, 4, dtype=torch.int32), "row_idx: 1-D"),
    ("suppress_eos", torch.zeros(8, dtype=torch.bool), "suppress_eos: dtype"),
    ("suppress_eos", torch.zeros(7, dtype=torch.uint8), "suppress_eos:"),
    ("conf", torch.zeros(7, dtype=torch.float32), "conf:"),
    ("argmax", torch.zeros(8, dtype=torch.int64), "argmax: dtype"),
    ("lse", torch.zeros(8, dtype=torch.float64), "lse: dtype"),
])
def test_lmhead_rejects(fn, key, bad, msg):
    a = _lm_args()
    a[key] = bad
    with pytest.raises(AsyncLaneError, match=msg):
        fn(**a)


def test_lmhead_host_tensors_rejected():
    with pytest.raises(AsyncLaneError, match="device tensor expected"):
        al.lmhead_confidence(**_lm_args())
    with pytest.raises(AsyncLaneError, match="device tensor expected"):
        al.lmhead_confidence_noalloc(**_lm_args())


def _sel_args(L=2, B=8, N=5):
    return dict(conf=torch.zeros(N), argmax=torch.zeros(N, dtype=torch.int32),
                row_pos=torch.arange(N, dtype=torch.int32), tokens=torch.zeros(L * B, dtype=torch.int32),
                is_masked=torch.ones(L * B, dtype=torch.uint8), L=L, B=B, role=[0, 0])


@pytest.mark.parametrize("key,bad,msg", [
    ("conf", torch.zeros(5, dtype=torch.float64), "conf: dtype"),
    ("conf", torch.zeros(4), "conf:"),
    ("argmax", torch.zeros(5, dtype=torch.int64), "argmax: dtype"),
    ("row_pos", torch.arange(5, dtype=torch.int64), "row_pos: dtype"),
    ("tokens", torch.zeros(15, dtype=torch.int32), "tokens:"),
    ("tokens", torch.zeros(16, dtype=torch.int64), "tokens: dtype"),
    ("is_masked", torch.ones(16, dtype=torch.bool), "is_masked: dtype"),
    ("role", [0], "role"),
])
def test_select_rejects(key, bad, msg):
    a = _sel_args()
    a[key] = bad
    with pytest.raises(AsyncLaneError, match=msg):
        al.select_unmask(**a)


def test_select_out_buffers_checked():
    out = dict(unmask_flag=torch.zeros(5, dtype=torch.uint8), unmasked_pos=torch.zeros(5, dtype=torch.int32),
               still_masked_pos=torch.zeros(5, dtype=torch.int32), counts=torch.zeros(2, dtype=torch.int32),
               lane_stats=torch.zeros(1, al.LANE_STATS, dtype=torch.int32), delim_flag=None)
    with pytest.raises(AsyncLaneError, match="lane_stats:"):
        al.select_unmask(**_sel_args(), out=out)
    out["lane_stats"] = torch.zeros(2, al.LANE_STATS, dtype=torch.int32)
    out["unmasked_pos"] = torch.zeros(5, dtype=torch.int64)
    with pytest.raises(AsyncLaneError, match="unmasked_pos: dtype"):
        al.select_unmask(**_sel_args(), out=out)
    del out["counts"]
    out["unmasked_pos"] = torch.zeros(5, dtype=torch.int32)
    with pytest.raises(AsyncLaneError, match="missing 'counts'"):
        al.select_unmask(**_sel_args(), out=out)


def test_lmhead_packed_rejects():
    a = _lm_args()
    Wp = torch.zeros(al.lmhead_packed_weight_size(64, 100) // 2, dtype=bf16)
    with pytest.raises(AsyncLaneError, match="W_packed:"):
        al.lmhead_confidence_packed(a["hidden"], Wp[:-1], 100, row_idx=a["row_idx"])
    with pytest.raises(AsyncLaneError, match="W_packed: dtype"):
        al.lmhead_confidence_packed(a["hidden"], Wp.float(), 100, row_idx=a["row_idx"])
    with pytest.raises(AsyncLaneError, match="W_packed: no packed layout"):
        al.lmhead_confidence_packed(torch.zeros(8, 12, dtype=bf16), Wp, 100)
    with pytest.raises(AsyncLaneError, match="device tensor expected"):
        al.lmhead_confidence_packed(a["hidden"], Wp, 100, row_idx=a["row_idx"])
    with pytest.raises(AsyncLaneError, match="W: dtype"):
        al.lmhead_pack_weight(torch.zeros(100, 64))


def test_call_makes_the_tensor_device_current(monkeypatch):
    """The library takes pointers of the current device, so the binding makes
    the tensors' device current around the call when it is another one."""
    from paper_2606_08411_amd import _lib
    seen = []

    class Dev:
        def __init__(self, index):
            self.index = index

    class T:
        def __init__(self, index):
            self.device = Dev(index)

    class Guard:
        def __init__(self, idx):
            self.idx = idx

        def __enter__(self):
            seen.append(("enter", self.idx))

        def __exit__(self, *a):
            seen.append(("exit", self.idx))

    monkeypatch.setattr(torch.cuda, "current_device", lambda: 0)
    monkeypatch.setattr(torch.cuda, "device", Guard)
    assert _lib._call(lambda *a: ("ran", a), T(0), 1, 2) == ("ran", (1, 2))
    assert seen == []
    assert _lib._call(lambda *a: ("ran", a), T(1), 3) == ("ran", (3,))
    assert seen == [("enter", 1), ("exit", 1)]
