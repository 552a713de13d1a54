"""ctypes binding of libasynclane.so (the C ABI in include/asynclane.h).

Argument marshalling only: every step of the decode-step hot path runs in the
library's HIP kernels.  PyTorch supplies device memory and the current HIP
stream.  There is no fallback: when the library is missing or a call fails,
an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
import threading

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libasynclane.so")

AL_OK = 0
STATUS = {0: "AL_OK", -1: "AL_ERR_NULL", -2: "AL_ERR_SHAPE", -3: "AL_ERR_TREE",
          -4: "AL_ERR_WORKSPACE", -5: "AL_ERR_ALIGN", -6: "AL_ERR_UNSUPPORTED",
          -7: "AL_ERR_HIP"}
ROLE_GEN, ROLE_REF = 0, 1
MODE_THRESHOLD, MODE_TOPK = 0, 1
LANE_STATS = 6
MAX_SELECT_POSITIONS = 8192

_vp = ctypes.c_void_p
_i = ctypes.c_int
_f = ctypes.c_float
_sz = ctypes.c_size_t

_SIGNATURES = {
    "al_status_string": (ctypes.c_char_p, [_i]),
    "lane_attn_workspace_size": (_sz, [_i] * 7),
    "lane_attn_forward": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _f,
                               _vp, _i, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "lmhead_confidence_workspace_size": (_sz, [_i, _i, _i]),
    "al_refresh_window": (_i, [_i, _i, _vp, _vp, _i, _i]),
    "al_sched_create": (_vp, [_i, _i, _i, _i, _i, _i]),
    "al_sched_destroy": (None, [_vp]),
    "al_sched_plan": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i]),
    "al_sched_blocks": (_i, [_vp, _vp, _vp]),
    "al_sched_commit": (_i, [_vp, _vp, _vp, _vp]),
    "al_sched_collect": (_i, [_vp, _i, _vp, _i]),
    "al_sched_counters": (_i, [_vp, _vp]),
    "al_sched_tree": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i]),
    "al_sched_state": (_i, [_vp, _vp, _vp]),
    "lmhead_confidence": (_i, [_vp, _i, _vp, _i, _vp, _i, _i, _vp, _i, _vp, _vp, _vp, _vp,
                               _sz, _vp]),
    "lmhead_packed_weight_size": (_sz, [_i, _i]),
    "lmhead_pack_weight": (_i, [_vp, _i, _i, _vp, _sz, _vp]),
    "lmhead_confidence_packed": (_i, [_vp, _i, _vp, _i, _vp, _i, _i, _vp, _i, _vp, _vp, _vp, _vp,
                                      _sz, _vp]),
    "lmhead_confidence_noalloc": (_i, [_vp, _i, _vp, _i, _vp, _i, _i, _vp, _i, _vp, _vp, _vp,
                                       _vp]),
    "select_unmask": (_i, [_vp, _vp, _vp, _i, _vp, _vp, _i, _i, _vp, _vp, _vp, _i, _f, _i,
                           _vp, _vp, _i, _vp, _i, _vp, _i, _vp, _i, _i, _f, _i, _f,
                           _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
}

_lib = None
_lock = threading.Lock()


class AsyncLaneError(RuntimeError):
    pass


def library() -> ctypes.CDLL:
    """Load libasynclane.so (raises when it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise AsyncLaneError(
                    f"{LIB_PATH} is missing: build it with "
                    "`python -m paper_2606_08411_amd.build` (hipcc, gfx950)")
            lib = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in _SIGNATURES.items():
                fn = getattr(lib, name)
                fn.restype = res
                fn.argtypes = args
            _lib = lib
    return _lib


def _check(status: int, what: str):
    if status != AL_OK:
        msg = library().al_status_string(status).decode()
        raise AsyncLaneError(f"{what} failed: {STATUS.get(status, status)} ({msg})")


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise AsyncLaneError("device tensor expected")
    if not t.is_contiguous():
        raise AsyncLaneError("contiguous tensor expected")
    return t.data_ptr()


def _tensor(t, name, dtype, shape=None, min_numel=None, optional=False):
    """Check a tensor argument before anything reaches the library: its
    dtype, then its exact shape (shape) or at least min_numel elements (an
    output buffer of which the call writes a prefix).  Device and layout are
    checked by _ptr."""
    if t is None:
        if optional:
            return None
        raise AsyncLaneError(f"{name}: a tensor is required")
    if not isinstance(t, torch.Tensor):
        raise AsyncLaneError(f"{name}: torch.Tensor expected, got {type(t).__name__}")
    if t.dtype != dtype:
        raise AsyncLaneError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(int(x) for x in shape):
        raise AsyncLaneError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if min_numel is not None and t.numel() < min_numel:
        raise AsyncLaneError(f"{name}: {t.numel()} elements, at least {min_numel} expected")
    return t


def _same_device(*ts):
    """Every tensor given is a device tensor, all on one device."""
    ts = [t for t in ts if t is not None]
    if any(not t.is_cuda for t in ts):
        raise AsyncLaneError("device tensor expected")
    devs = {t.device for t in ts}
    if len(devs) > 1:
        raise AsyncLaneError(f"tensors on different devices: {sorted(str(d) for d in devs)}")


def _call(fn, t, *args):
    """Call library function fn with t's device current: the ABI takes device
    pointers (and the stream) of the current HIP device, and the library's
    per-device state (compute-unit count, the no-alloc array's address) is
    looked up on the current device."""
    idx = t.device.index
    if idx is not None and idx != torch.cuda.current_device():
        with torch.cuda.device(idx):
            return fn(*args)
    return fn(*args)


# torch's raw-handle accessor costs ~0.1 us against ~3 us for
# torch.cuda.current_stream(); both name the same stream.
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(t=None):
    """Handle of torch's current stream on t's device (else the current device)."""
    idx = t.device.index if t is not None else torch.cuda.current_device()
    if _raw_stream is not None:
        return _raw_stream(idx)
    return torch.cuda.current_stream(idx).cuda_stream


def _host_i32(x, n, name):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.int32))
    if a.shape != (n,):
        raise AsyncLaneError(f"{name}: expected {n} entries")
    return a


def _host_u8(x, n, name):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.uint8))
    if a.shape != (n,):
        raise AsyncLaneError(f"{name}: expected {n} entries")
    return a


def _np_ptr(a):
    return None if a is None else a.ctypes.data


_id_sets: dict = {}


def _host_ids(x):
    """int32 array of a token-id set; tuples and lists are converted once."""
    if isinstance(x, (tuple, list)):
        key = tuple(int(v) for v in x)
        a = _id_sets.get(key)
        if a is None:
            if len(_id_sets) >= 64:   # a few fixed sets in practice; stay bounded
                _id_sets.clear()
            a = _id_sets[key] = np.asarray(key, dtype=np.int32)
        return a
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


# ------------------------------------------------------------ workspaces
# Default workspaces, one per (kind, device, stream): calls on different
# streams never share one.  A buffer that has to grow is replaced by one at
# least twice its size and the old one is kept alive (never returned to the
# allocator), because a launch still in flight may still write to it.  While
# a HIP graph is being captured the caller must pass its own workspace, so
# no two graphs (or a graph and eager calls) share one by default.
_ws_cache: dict = {}
_ws_retired: list = []


def _workspace(kind: str, nbytes: int, device, stream: int):
    if nbytes == 0:
        return None, 0
    if torch.cuda.is_current_stream_capturing():
        raise AsyncLaneError(
            f"{kind}: pass workspace= while a HIP graph is being captured (the call needs "
            f"{nbytes} bytes of workspace)")
    key = (kind, device.index, int(stream))
    buf = _ws_cache.get(key)
    if buf is None or buf.numel() < nbytes:
        grow = 0 if buf is None else 2 * buf.numel()
        new = torch.empty(max(nbytes, 256, grow), dtype=torch.uint8, device=device)
        if buf is not None:
            _ws_retired.append(buf)
        _ws_cache[key] = buf = new
    return buf, buf.numel()


def _explicit_workspace(ws, device):
    if not isinstance(ws, torch.Tensor):
        raise AsyncLaneError("workspace: torch.Tensor expected")
    if ws.device != device:
        raise AsyncLaneError(f"workspace on {ws.device}, expected {device}")
    return ws, ws.numel() * ws.element_size()


# ------------------------------------------------------------ entry points
def lane_attn_workspace_size(L, B, P, Hq, Hkv, D, n_refresh=0) -> int:
    return int(library().lane_attn_workspace_size(L, B, P, Hq, Hkv, D, n_refresh))


def lane_attn_forward(q, k_lane, v_lane, k_prefix, v_prefix, parent, B, scale=0.0,
                      refresh_idx=None, q_ref=None, k_ref=None, v_ref=None,
                      o=None, lse=None, o_ref=None, lse_ref=None, want_lse=True,
                      workspace=None):
    """Shared-prefix lane-batched attention (+ compact-refresh rows).

    q [L*B][Hq][D], k_lane/v_lane [L*B][Hkv][D], k_prefix/v_prefix
    [P][Hkv][D] are bf16 device tensors; parent is a host sequence of L ints.
    k_prefix / v_prefix are updated in place when refresh rows are given.
    A refresh-only call (compact cache refresh) passes q = k_lane = v_lane
    = None and parent = [] with refresh rows.  Returns (o, lse, o_ref,
    lse_ref).  Every tensor's dtype and shape is checked before the call."""
    lib = library()
    bf16, f32 = torch.bfloat16, torch.float32
    _tensor(k_prefix, "k_prefix", bf16)
    if k_prefix.dim() != 3:
        raise AsyncLaneError(f"k_prefix: [P][Hkv][D] expected, got shape {tuple(k_prefix.shape)}")
    P, Hkv, D = k_prefix.shape
    _tensor(v_prefix, "v_prefix", bf16, (P, Hkv, D))
    L = len(parent)
    par = _host_i32(parent, L, "parent")
    n_ref = 0 if refresh_idx is None else int(refresh_idx.shape[0])
    dev = k_prefix.device
    if L > 0:
        B = int(B)
        _tensor(q, "q", bf16)
        if q.dim() != 3 or q.shape[0] != L * B or q.shape[2] != D:
            raise AsyncLaneError(f"q: [L*B={L * B}][Hq][D={D}] expected, got {tuple(q.shape)}")
        Hq = int(q.shape[1])
        LB = L * B
        _tensor(k_lane, "k_lane", bf16, (LB, Hkv, D))
        _tensor(v_lane, "v_lane", bf16, (LB, Hkv, D))
        if o is None:
            o = torch.empty_like(q)
        if lse is None and want_lse:
            lse = torch.empty((LB, Hq), dtype=f32, device=dev)
        _tensor(o, "o", bf16, (LB, Hq, D))
        _tensor(lse, "lse", f32, (LB, Hq), optional=True)
    else:
        if n_ref == 0:
            raise AsyncLaneError("lane_attn_forward: no lanes and no refresh rows")
        _tensor(q_ref, "q_ref", bf16)
        if q_ref.dim() != 3:
            raise AsyncLaneError(f"q_ref: [n_refresh][Hq][D] expected, got {tuple(q_ref.shape)}")
        Hq = int(q_ref.shape[1])
        B = 16
    if n_ref:
        _tensor(refresh_idx, "refresh_idx", torch.int32, (n_ref,))
        _tensor(q_ref, "q_ref", bf16, (n_ref, Hq, D))
        _tensor(k_ref, "k_ref", bf16, (n_ref, Hkv, D))
        _tensor(v_ref, "v_ref", bf16, (n_ref, Hkv, D))
        if o_ref is None:
            o_ref = torch.empty_like(q_ref)
        if lse_ref is None and want_lse:
            lse_ref = torch.empty((n_ref, Hq), dtype=f32, device=dev)
        _tensor(o_ref, "o_ref", bf16, (n_ref, Hq, D))
        _tensor(lse_ref, "lse_ref", f32, (n_ref, Hq), optional=True)
    _same_device(q, k_lane, v_lane, k_prefix, v_prefix, o, lse, refresh_idx, q_ref, k_ref,
                 v_ref, o_ref, lse_ref)
    need = int(lib.lane_attn_workspace_size(L, B, P, Hq, Hkv, D, n_ref))
    if workspace is not None:
        ws, ws_bytes = _explicit_workspace(workspace, dev)
    stream = _stream(k_prefix)
    if workspace is None:
        ws, ws_bytes = _workspace("attn", need, dev, stream)
    st = _call(
        lib.lane_attn_forward, k_prefix,
        _ptr(q), _ptr(k_lane), _ptr(v_lane), _ptr(k_prefix), _ptr(v_prefix),
        _np_ptr(par) if L else None,
        L, B, P, Hq, Hkv, D, float(scale),
        _ptr(refresh_idx) if n_ref else None, n_ref,
        _ptr(q_ref) if n_ref else None, _ptr(k_ref) if n_ref else None,
        _ptr(v_ref) if n_ref else None, _ptr(o_ref) if n_ref else None,
        _ptr(lse_ref) if n_ref else None, _ptr(o), _ptr(lse), _ptr(ws), ws_bytes, stream)
    _check(st, "lane_attn_forward")
    return o, lse, o_ref, lse_ref


def al_refresh_window(P, L_gen, lane_start, valid_len, margin) -> int:
    """Compact refresh window length L_refresh (host computation)."""
    n = len(lane_start)
    s = _host_i32(lane_start, n, "lane_start")
    v = _host_i32(valid_len, n, "valid_len")
    r = int(library().al_refresh_window(int(P), int(L_gen), _np_ptr(s) if n else None,
                                        _np_ptr(v) if n else None, n, int(margin)))
    if r < 0:
        _check(r, "al_refresh_window")
    return r


def lmhead_confidence_workspace_size(N, d, V) -> int:
    return int(library().lmhead_confidence_workspace_size(N, d, V))


def _lmhead_args(hidden, W, row_idx, suppress_eos, conf, argmax, lse, want_lse, V=None):
    """Checks and output allocation shared by the LM-head calls.  W is the
    [V][d] weight, or (V given) the flat packed copy of a [V][d] weight."""
    bf16 = torch.bfloat16
    _tensor(hidden, "hidden", bf16)
    if hidden.dim() != 2:
        raise AsyncLaneError(f"hidden: [n_rows][d] expected, got shape {tuple(hidden.shape)}")
    n_rows, d = hidden.shape
    if V is None:
        _tensor(W, "W", bf16)
        if W.dim() != 2 or W.shape[1] != d:
            raise AsyncLaneError(f"W: [V][d={d}] expected, got shape {tuple(W.shape)}")
        V = int(W.shape[0])
    else:
        nbytes = int(library().lmhead_packed_weight_size(int(d), int(V)))
        if nbytes == 0:
            raise AsyncLaneError(f"W_packed: no packed layout for d={d}, V={V}")
        _tensor(W, "W_packed", bf16, min_numel=nbytes // 2)
    N = n_rows
    if row_idx is not None:
        _tensor(row_idx, "row_idx", torch.int32)
        if row_idx.dim() != 1:
            raise AsyncLaneError(f"row_idx: 1-D expected, got shape {tuple(row_idx.shape)}")
        N = int(row_idx.shape[0])
    _tensor(suppress_eos, "suppress_eos", torch.uint8, min_numel=N, optional=True)
    dev = hidden.device
    if conf is None:
        conf = torch.empty(N, dtype=torch.float32, device=dev)
    if argmax is None:
        argmax = torch.empty(N, dtype=torch.int32, device=dev)
    if lse is None and want_lse:
        lse = torch.empty(N, dtype=torch.float32, device=dev)
    _tensor(conf, "conf", torch.float32, min_numel=N)
    _tensor(argmax, "argmax", torch.int32, min_numel=N)
    _tensor(lse, "lse", torch.float32, min_numel=N, optional=True)
    _same_device(hidden, W, row_idx, suppress_eos, conf, argmax, lse)
    return n_rows, d, int(V), N, conf, argmax, lse


def lmhead_confidence(hidden, W, row_idx=None, suppress_eos=None, eos_id=-1,
                      conf=None, argmax=None, lse=None, want_lse=True, workspace=None):
    """Per scored row: max softmax probability, its token id and the
    log-sum-exp over the vocabulary (EOS excluded for suppressed rows).
    hidden [n_rows][d] and W [V][d] are bf16 device tensors; row_idx is an
    int32 device tensor (None = every row).  Output buffers passed in need
    at least N entries (the first N are written).  Returns (conf, argmax,
    lse)."""
    lib = library()
    n_rows, d, V, N, conf, argmax, lse = _lmhead_args(hidden, W, row_idx, suppress_eos, conf,
                                                      argmax, lse, want_lse)
    if N == 0:
        return conf, argmax, lse
    dev = hidden.device
    need = int(lib.lmhead_confidence_workspace_size(N, d, V))
    if workspace is not None:
        ws, ws_bytes = _explicit_workspace(workspace, dev)
    stream = _stream(hidden)
    if workspace is None:
        ws, ws_bytes = _workspace("lmhead", need, dev, stream)
    st = _call(lib.lmhead_confidence, hidden,
               _ptr(hidden), n_rows, _ptr(row_idx), N, _ptr(W), d, V,
               _ptr(suppress_eos), int(eos_id), _ptr(conf), _ptr(argmax),
               _ptr(lse), _ptr(ws), ws_bytes, stream)
    _check(st, "lmhead_confidence")
    return conf, argmax, lse


def lmhead_packed_weight_size(d, V) -> int:
    return int(library().lmhead_packed_weight_size(int(d), int(V)))


def lmhead_pack_weight(W, out=None):
    """One-time repack of the LM-head weight W [V][d] (bf16, device) into
    the layout lmhead_confidence_packed streams.  Returns a flat bf16 device
    tensor (or fills `out`)."""
    lib = library()
    _tensor(W, "W", torch.bfloat16)
    if W.dim() != 2:
        raise AsyncLaneError(f"W: [V][d] expected, got shape {tuple(W.shape)}")
    V, d = (int(x) for x in W.shape)
    nbytes = int(lib.lmhead_packed_weight_size(d, V))
    if nbytes == 0:
        raise AsyncLaneError(f"W: unsupported shape {tuple(W.shape)}")
    if out is None:
        out = torch.empty(nbytes // 2, dtype=torch.bfloat16, device=W.device)
    _tensor(out, "out", torch.bfloat16, min_numel=nbytes // 2)
    _same_device(W, out)
    st = _call(lib.lmhead_pack_weight, W, _ptr(W), d, V, _ptr(out), out.numel() * 2, _stream(W))
    _check(st, "lmhead_pack_weight")
    return out


def lmhead_confidence_packed(hidden, W_packed, V, row_idx=None, suppress_eos=None, eos_id=-1,
                             conf=None, argmax=None, lse=None, want_lse=True, workspace=None):
    """lmhead_confidence reading the weight from lmhead_pack_weight's copy
    (V = vocabulary size of the original W; d is hidden's width)."""
    lib = library()
    n_rows, d, V, N, conf, argmax, lse = _lmhead_args(hidden, W_packed, row_idx, suppress_eos, conf,
                                                      argmax, lse, want_lse, V=int(V))
    if N == 0:
        return conf, argmax, lse
    dev = hidden.device
    need = int(lib.lmhead_confidence_workspace_size(N, d, V))
    if workspace is not None:
        ws, ws_bytes = _explicit_workspace(workspace, dev)
    stream = _stream(hidden)
    if workspace is None:
        ws, ws_bytes = _workspace("lmhead", need, dev, stream)
    st = _call(lib.lmhead_confidence_packed, hidden,
               _ptr(hidden), n_rows, _ptr(row_idx), N, _ptr(W_packed), d, V,
               _ptr(suppress_eos), int(eos_id), _ptr(conf), _ptr(argmax),
               _ptr(lse), _ptr(ws), ws_bytes, stream)
    _check(st, "lmhead_confidence_packed")
    return conf, argmax, lse


def lmhead_confidence_noalloc(hidden, W, row_idx=None, suppress_eos=None, eos_id=-1,
                              conf=None, argmax=None, lse=None, want_lse=True):
    """lmhead_confidence without a workspace: the library keeps the partials
    in a fixed device array of its own (calls that overlap on one GPU race).
    Pass conf / argmax (/ lse) to allocate nothing at all."""
    lib = library()
    n_rows, d, V, N, conf, argmax, lse = _lmhead_args(hidden, W, row_idx, suppress_eos, conf,
                                                      argmax, lse, want_lse)
    if N == 0:
        return conf, argmax, lse
    st = _call(lib.lmhead_confidence_noalloc, hidden,
               _ptr(hidden), n_rows, _ptr(row_idx), N, _ptr(W), d, V,
               _ptr(suppress_eos), int(eos_id), _ptr(conf),
               _ptr(argmax), _ptr(lse), _stream(hidden))
    _check(st, "lmhead_confidence_noalloc")
    return conf, argmax, lse


def select_unmask(conf, argmax, row_pos, tokens, is_masked, L, B, role, b_len=None,
                  t_lane=None, mode=MODE_THRESHOLD, tau=0.9, fallback_k=0, k_lane=None,
                  delim_ids=(0, 1), eos_id=2, rho_min=0.5, t_min=2, tau_future=None,
                  with_delim_flag=True, out=None, digit_ids=(), open_ids=(), close_ids=()):
    """Per-lane transfer, lookahead drafts (tau_future None = off) and
    write-back (tokens / is_masked updated in place), ordered compaction and
    lane statistics with ValidBoundary id sets (digit_ids, open_ids,
    close_ids; empty = every delimiter counts).  Returns a dict of device
    tensors: unmask_flag, unmasked_pos, still_masked_pos, counts,
    lane_stats, delim_flag."""
    lib = library()
    L, B = int(L), int(B)
    _tensor(row_pos, "row_pos", torch.int32)
    if row_pos.dim() != 1:
        raise AsyncLaneError(f"row_pos: 1-D expected, got shape {tuple(row_pos.shape)}")
    N = int(row_pos.shape[0])
    _tensor(conf, "conf", torch.float32, min_numel=N)
    _tensor(argmax, "argmax", torch.int32, min_numel=N)
    for t, name, dt in ((tokens, "tokens", torch.int32), (is_masked, "is_masked", torch.uint8)):
        _tensor(t, name, dt)
        if t.numel() != L * B:
            raise AsyncLaneError(f"{name}: {t.numel()} elements, L*B = {L * B} expected")
    dev = tokens.device
    role_h = _host_u8(role, L, "role")
    b_len_h = None if b_len is None else _host_i32(b_len, L, "b_len")
    t_lane_h = None if t_lane is None else _host_i32(t_lane, L, "t_lane")
    k_lane_h = None if k_lane is None else _host_i32(k_lane, L, "k_lane")
    delim_h = _host_ids(delim_ids)
    sets = [_host_ids(x) for x in (digit_ids, open_ids, close_ids)]
    if out is None:
        out = dict(
            unmask_flag=torch.empty(max(N, 1), dtype=torch.uint8, device=dev),
            unmasked_pos=torch.empty(max(N, 1), dtype=torch.int32, device=dev),
            still_masked_pos=torch.empty(max(N, 1), dtype=torch.int32, device=dev),
            counts=torch.empty(2, dtype=torch.int32, device=dev),
            lane_stats=torch.empty((L, LANE_STATS), dtype=torch.int32, device=dev),
            delim_flag=torch.empty(L * B, dtype=torch.uint8, device=dev) if with_delim_flag else None)
    for name, dt, n in (("unmask_flag", torch.uint8, N), ("unmasked_pos", torch.int32, N),
                        ("still_masked_pos", torch.int32, N), ("counts", torch.int32, 2),
                        ("lane_stats", torch.int32, L * LANE_STATS)):
        if name not in out:
            raise AsyncLaneError(f"out: missing '{name}'")
        _tensor(out[name], name, dt, min_numel=n)
    _tensor(out.get("delim_flag"), "delim_flag", torch.uint8, min_numel=L * B, optional=True)
    _same_device(conf, argmax, row_pos, tokens, is_masked, *out.values())
    st = _call(
        lib.select_unmask, conf,
        _ptr(conf) if N else None, _ptr(argmax) if N else None, _ptr(row_pos) if N else None, N,
        _ptr(tokens), _ptr(is_masked), L, B, _np_ptr(role_h), _np_ptr(b_len_h), _np_ptr(t_lane_h),
        int(mode), float(tau), int(fallback_k), _np_ptr(k_lane_h),
        _np_ptr(delim_h) if len(delim_h) else None, len(delim_h),
        _np_ptr(sets[0]) if len(sets[0]) else None, len(sets[0]),
        _np_ptr(sets[1]) if len(sets[1]) else None, len(sets[1]),
        _np_ptr(sets[2]) if len(sets[2]) else None, len(sets[2]), int(eos_id), float(rho_min),
        int(t_min), float("inf") if tau_future is None else float(tau_future),
        _ptr(out["unmask_flag"]), _ptr(out["unmasked_pos"]),
        _ptr(out["still_masked_pos"]), _ptr(out["counts"]), _ptr(out["lane_stats"]),
        _ptr(out["delim_flag"]), _stream(tokens))
    _check(st, "select_unmask")
    return out


# ------------------------------------------------------------------ scheduler
class AlSched:
    """Host active-lane scheduler (al_sched_* in include/asynclane.h); every
    method is one call into the library.  Arrays are host numpy arrays."""

    def __init__(self, P, L_gen, B, window=0, max_lanes=64, pad_id=3):
        self._lib = library()
        self.L, self.B, self.W = int(L_gen), int(B), int(B) + int(window)
        self._h = self._lib.al_sched_create(int(P), int(L_gen), int(B), int(window),
                                            int(max_lanes), int(pad_id))
        if not self._h:
            raise AsyncLaneError("al_sched_create: bad arguments")
        self._n = 0
        # Output buffers reused across calls, with their addresses cached
        # (numpy's pointer lookup costs ~1 us per array).
        self._plan_bufs = {}
        nb = max(int(max_lanes), 1) * self.W
        self._blk = (np.zeros(nb, np.int32), np.zeros(nb, np.uint8))
        self._blk_ptr = tuple(x.ctypes.data for x in self._blk)

    def __del__(self):
        if getattr(self, "_h", None):
            self._lib.al_sched_destroy(self._h)
            self._h = None

    _PLAN_KEYS = ("lane_id", "role", "start", "b_len", "t_step", "group", "call_parent")

    def plan(self, cap=64):
        """Returns dict of [n] arrays: lane_id, role, start, b_len, t_step,
        group, call_parent."""
        bufs = self._plan_bufs.get(cap)
        if bufs is None:
            arrs = [np.zeros(cap, np.uint8 if k == "role" else np.int32) for k in self._PLAN_KEYS]
            bufs = self._plan_bufs[cap] = (arrs, [x.ctypes.data for x in arrs])
        arrs, ptrs = bufs
        n = self._lib.al_sched_plan(self._h, *ptrs, cap)
        if n < 0:
            _check(n, "al_sched_plan")
        self._n = n
        return {k: x[:n].copy() for k, x in zip(self._PLAN_KEYS, arrs)}

    def blocks(self):
        """Tokens and mask flags of the planned lanes' blocks, [n * (B + window)]."""
        r = self._lib.al_sched_blocks(self._h, *self._blk_ptr)
        if r < 0:
            _check(r, "al_sched_blocks")
        m = self._n * self.W
        return self._blk[0][:m].copy(), self._blk[1][:m].copy()

    def commit(self, tokens, masked, lane_stats):
        tk = np.ascontiguousarray(tokens, np.int32)
        mk = np.ascontiguousarray(masked, np.uint8)
        st = np.ascontiguousarray(lane_stats, np.int32)
        r = self._lib.al_sched_commit(self._h, _np_ptr(tk), _np_ptr(mk), _np_ptr(st))
        if r < 0:
            _check(r, "al_sched_commit")
        return r

    def collect(self, eos_id=2):
        out = np.zeros(self.L, np.int32)
        n = self._lib.al_sched_collect(self._h, int(eos_id), _np_ptr(out), self.L)
        if n < 0:
            _check(n, "al_sched_collect")
        return out[:n].tolist()

    def counters(self):
        out = np.zeros(6, np.int32)
        _check(self._lib.al_sched_counters(self._h, _np_ptr(out)), "al_sched_counters")
        return dict(zip(("iterations", "nfe", "forks", "spawns", "stops", "lanes"), out.tolist()))

    def tree(self, cap=100000):
        a = [np.zeros(cap, np.uint8)] + [np.zeros(cap, np.int32) for _ in range(5)]
        n = self._lib.al_sched_tree(self._h, *[_np_ptr(x) for x in a], cap)
        if n < 0:
            _check(n, "al_sched_tree")
        return dict(zip(("role", "start", "length", "parent", "kind", "v"), [x[:n].copy() for x in a]))

    def state(self):
        tk = np.zeros(self.L, np.int32)
        mk = np.zeros(self.L, np.uint8)
        r = self._lib.al_sched_state(self._h, _np_ptr(tk), _np_ptr(mk))
        if r < 0:
            _check(r, "al_sched_state")
        return tk, mk
