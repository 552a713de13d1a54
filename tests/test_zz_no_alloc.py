"""lmhead_confidence_noalloc (partials in the library's fixed device array,
no workspace) through the C ABI, against lmhead_confidence with a caller
workspace: the same kernels run, so the outputs must agree bit for bit.
Two calls in a row, the second with a smaller input (the array keeps the
first call's partials, which must not leak into the second), then the
first shape again."""
import ctypes

import numpy as np
import pytest
import torch

import synth
from gpu_util import dev, dev_bf16

pytestmark = pytest.mark.gpu


def _inputs(N, n_rows, d, V, seed):
    g = np.random.default_rng([seed, N, d, V])
    scale = g.uniform(1, 6, n_rows).astype(np.float32)
    H = synth.f32_to_bf16_bits(g.standard_normal((n_rows, d), dtype=np.float32) * scale[:, None])
    W = synth.f32_to_bf16_bits(g.standard_normal((V, d), dtype=np.float32) / np.float32(np.sqrt(d)))
    row_idx = np.sort(g.choice(n_rows, N, replace=False)).astype(np.int32)
    sup = (g.random(N) < 0.5).astype(np.uint8)
    return dev_bf16(H), dev_bf16(W), dev(row_idx), dev(sup)


def _outputs(N):
    return (torch.full((N,), float("nan"), device="cuda"),
            torch.full((N,), -1, dtype=torch.int32, device="cuda"),
            torch.full((N,), float("nan"), device="cuda"))


def _call(lib, fn, H, W, ridx, sup, eos, outs, ws=None):
    n_rows, d = H.shape
    V = W.shape[0]
    N = ridx.shape[0]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    args = [p(H), n_rows, p(ridx), N, p(W), d, V, p(sup), eos, p(outs[0]), p(outs[1]), p(outs[2])]
    if ws is not None:
        args += [p(ws), ws.numel()]
    st = getattr(lib, fn)(*args, stream)
    assert st == 0, f"{fn} returned {st}"


def test_noalloc_matches_workspace_entry():
    import paper_2606_08411_amd as al
    lib = al.library()
    shapes = [(614, 640, 1024, 70000, 2), (77, 90, 512, 30001, 5), (614, 640, 1024, 70000, 2)]
    for k, (N, n_rows, d, V, eos) in enumerate(shapes):
        H, W, ridx, sup = _inputs(N, n_rows, d, V, seed=k % 2)
        need = al.lmhead_confidence_workspace_size(N, d, V)
        assert 0 < need <= 8 << 20
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        want, got = _outputs(N), _outputs(N)
        _call(lib, "lmhead_confidence", H, W, ridx, sup, eos, want, ws)
        _call(lib, "lmhead_confidence_noalloc", H, W, ridx, sup, eos, got)
        torch.cuda.synchronize()
        for a, b, name in zip(got, want, ("conf", "argmax", "lse")):
            assert torch.equal(a, b), f"call {k} ({N} rows): {name} differs"
        assert not torch.isnan(got[0]).any() and (got[1] >= 0).all()
