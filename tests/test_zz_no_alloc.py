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


def test_noalloc_in_graph_capture():
    """The use it exists for: captured into a HIP graph (no allocation
    during capture), replayed several times with eager work of another
    shape in between; every replay equals the eager call."""
    import paper_2606_08411_amd as al
    H, W, ridx, sup = _inputs(200, 256, 512, 40000, seed=3)
    H2, W2, ridx2, sup2 = _inputs(50, 64, 256, 9000, seed=4)
    want = _outputs(200)
    al.lmhead_confidence_noalloc(H, W, row_idx=ridx, suppress_eos=sup, eos_id=2, conf=want[0],
                                 argmax=want[1], lse=want[2])
    got = _outputs(200)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        al.lmhead_confidence_noalloc(H, W, row_idx=ridx, suppress_eos=sup, eos_id=2, conf=got[0],
                                     argmax=got[1], lse=got[2])
    torch.cuda.synchronize()
    other = _outputs(50)
    for rep in range(3):
        for t in got:
            t.fill_(0)
        al.lmhead_confidence_noalloc(H2, W2, row_idx=ridx2, suppress_eos=sup2, eos_id=1,
                                     conf=other[0], argmax=other[1], lse=other[2])
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b, name in zip(got, want, ("conf", "argmax", "lse")):
            assert torch.equal(a, b), f"replay {rep}: {name} differs from the eager call"
