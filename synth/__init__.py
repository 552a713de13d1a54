"""Seeded synthetic inputs for the AsyncLane decode-step hot path.

This module is the only code shared by the CPU oracle and the HIP path.  It
draws random tensors and integer structure (lane trees, mask patterns, token
ids) and stores floating-point tensors as bfloat16 bit patterns (``uint16``).
It holds none of the method's arithmetic: no attention, no softmax, no
selection rule.

Workload shapes follow the backbones the paper evaluates (LLaDA-8B and
Dream-7B, Section 4.1) at the lane counts and prefix lengths of the five
synthetic decode steps listed in ``CONFIGS``.  The paper's datasets, weights
and tokenizer are not used: every value here is random and seeded.

RNG discipline: every tensor has its own sub-stream
``np.random.default_rng([seed, stream_id(, chunk)])`` so adding a tensor never
shifts another one.  Floats are drawn in fp32 and rounded to bf16 with
round-to-nearest-even on the fp32 bit pattern.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

ROLE_GEN = 0
ROLE_REF = 1
MODE_THRESHOLD = 0
MODE_TOPK = 1

# Stream ids (one per tensor / structure).
_S_Q, _S_KL, _S_VL, _S_KP, _S_VP = 1, 2, 3, 4, 5
_S_H, _S_HSCALE, _S_W = 6, 7, 8
_S_TREE, _S_MASK, _S_TOK, _S_TLANE, _S_DELIM = 9, 10, 11, 12, 13
_S_REFIDX, _S_QREF, _S_KREF, _S_VREF = 14, 15, 16, 17

# The five decode-step workloads.  L = active lanes, B = query tokens per
# lane, P = shared cached prefix rows, d = hidden size, V = vocabulary.
CONFIGS: dict[str, dict] = {
    "tiny": dict(Hq=4, Hkv=4, D=64, P=128, L=2, B=32, tree="fork", depth_max=1,
                 d=256, V=1024, mask_frac=0.5, tau=0.9, fallback_k=0,
                 delim_frac=0.0, refresh_frac=0.0),
    "llada": dict(Hq=32, Hkv=32, D=128, P=512, L=4, B=32, tree="linear", depth_max=3,
                  d=4096, V=126464, mask_frac=0.6, tau=0.9, fallback_k=1,
                  delim_frac=0.0, refresh_frac=0.0),
    "dream": dict(Hq=28, Hkv=4, D=128, P=1024, L=8, B=32, tree="random", depth_max=3,
                  d=3584, V=152064, mask_frac=0.5, tau=0.9, fallback_k=0,
                  delim_frac=0.0, refresh_frac=0.0),
    "long": dict(Hq=32, Hkv=32, D=128, P=2048, L=16, B=32, tree="random", depth_max=6,
                 d=4096, V=126464, mask_frac=0.4, tau=0.9, fallback_k=0,
                 delim_frac=0.05, refresh_frac=0.0),
    "wide": dict(Hq=32, Hkv=32, D=128, P=4096, L=32, B=64, tree="random", depth_max=8,
                 d=4096, V=126464, mask_frac=0.3, tau=0.9, fallback_k=0,
                 delim_frac=0.0, refresh_frac=0.1),
}

DELIM_IDS = (0, 1)
EOS_ID = 2
FIRST_ORDINARY_ID = 3
RHO_MIN = 0.5
T_MIN = 2


# ---------------------------------------------------------------- bf16 bits
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest-even) and return the uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).copy()
    t = u >> 16
    t &= 1
    t += 0x7FFF
    u += t
    u >>= 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _normal_bf16(seed, stream, shape, std=1.0) -> np.ndarray:
    g = np.random.default_rng([seed, stream])
    x = g.standard_normal(int(np.prod(shape)), dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return f32_to_bf16_bits(x).reshape(shape)


def lm_head_weight(seed: int, V: int, d: int, rows_per_chunk: int = 512,
                   threads: int | None = None) -> np.ndarray:
    """W [V][d] ~ N(0, 1/d) as bf16 bits, generated in fixed row chunks.

    Chunk c uses sub-stream [seed, W, c]; the result does not depend on the
    number of threads.
    """
    out = np.empty((V, d), dtype=np.uint16)
    std = np.float32(1.0 / math.sqrt(d))
    nch = (V + rows_per_chunk - 1) // rows_per_chunk

    def work(c):
        r0 = c * rows_per_chunk
        r1 = min(V, r0 + rows_per_chunk)
        g = np.random.default_rng([seed, _S_W, c])
        x = g.standard_normal((r1 - r0) * d, dtype=np.float32)
        x *= std
        out[r0:r1] = f32_to_bf16_bits(x).reshape(r1 - r0, d)

    if threads is None:
        try:
            threads = min(16, len(os.sched_getaffinity(0)))
        except AttributeError:  # pragma: no cover
            threads = 4
    if nch == 1 or threads <= 1:
        for c in range(nch):
            work(c)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(work, range(nch)))
    return out


# ---------------------------------------------------------------- structure
def lane_tree(kind: str, L: int, seed: int, depth_max: int) -> np.ndarray:
    """parent[L] int32 with parent[i] in [-1, i).

    fork: root + forks off the root; linear: chain; random: parent[i] uniform
    over earlier lanes whose depth (edges to the root) is below depth_max;
    forest: every lane is a root.
    """
    parent = np.full(L, -1, dtype=np.int32)
    if kind == "fork":
        parent[1:] = 0
    elif kind == "linear":
        parent[1:] = np.arange(L - 1)
    elif kind == "forest":
        pass
    elif kind == "random":
        g = np.random.default_rng([seed, _S_TREE])
        depth = np.zeros(L, dtype=np.int64)
        for i in range(1, L):
            ok = np.nonzero(depth[:i] < depth_max)[0]
            j = int(ok[g.integers(len(ok))])
            parent[i] = j
            depth[i] = depth[j] + 1
    else:
        raise ValueError(kind)
    return parent


def lane_roles(parent: np.ndarray) -> np.ndarray:
    """Leaves are generate lanes, lanes with children are refine lanes."""
    L = len(parent)
    role = np.full(L, ROLE_GEN, dtype=np.uint8)
    for i in range(L):
        if parent[i] >= 0:
            role[parent[i]] = ROLE_REF
    return role


@dataclass
class DecodeStep:
    """All inputs of one synthetic decode step (bf16 tensors as uint16 bits)."""
    name: str
    seed: int
    Hq: int
    Hkv: int
    D: int
    P: int
    L: int
    B: int
    d: int
    V: int
    parent: np.ndarray
    role: np.ndarray
    b_len: np.ndarray
    t_lane: np.ndarray
    q: np.ndarray          # [L*B][Hq][D]
    k_lane: np.ndarray     # [L*B][Hkv][D]
    v_lane: np.ndarray
    k_pre: np.ndarray      # [P][Hkv][D]
    v_pre: np.ndarray
    refresh_idx: np.ndarray  # [n_ref] int32, sorted unique
    q_ref: np.ndarray      # [n_ref][Hq][D]
    k_ref: np.ndarray      # [n_ref][Hkv][D]
    v_ref: np.ndarray
    hidden: np.ndarray     # [L*B][d]
    W: np.ndarray | None   # [V][d]
    tokens: np.ndarray     # [L*B] int32 (-1 at masked positions)
    is_masked: np.ndarray  # [L*B] uint8
    row_pos: np.ndarray    # [N] int32 ascending masked positions
    suppress_eos: np.ndarray  # [N] uint8 (rows of refine lanes)
    tau: float
    fallback_k: int
    topk_k: np.ndarray | None = None  # per-lane k for top-k mode
    delim_ids: tuple = DELIM_IDS
    eos_id: int = EOS_ID
    rho_min: float = RHO_MIN
    t_min: int = T_MIN
    extra: dict = field(default_factory=dict)

    @property
    def N(self) -> int:
        return int(len(self.row_pos))

    @property
    def n_ref(self) -> int:
        return int(len(self.refresh_idx))


def make_step(name: str = "tiny", seed: int = 0, with_weight: bool = True,
              **over) -> DecodeStep:
    """Build one synthetic decode step.  ``over`` overrides config fields
    (any of CONFIGS' keys, plus ``parent`` to force a lane tree)."""
    cfg = dict(CONFIGS[name])
    forced_parent = over.pop("parent", None)
    cfg.update(over)
    Hq, Hkv, D, P, L, B = (cfg[k] for k in ("Hq", "Hkv", "D", "P", "L", "B"))
    d, V = cfg["d"], cfg["V"]
    LB = L * B

    if forced_parent is not None:
        parent = np.asarray(forced_parent, dtype=np.int32)
        assert len(parent) == L
    else:
        parent = lane_tree(cfg["tree"], L, seed, cfg["depth_max"])
    role = lane_roles(parent)
    b_len = np.full(L, B, dtype=np.int32)
    t_lane = np.random.default_rng([seed, _S_TLANE]).integers(0, 8, L).astype(np.int32)

    q = _normal_bf16(seed, _S_Q, (LB, Hq, D))
    k_lane = _normal_bf16(seed, _S_KL, (LB, Hkv, D))
    v_lane = _normal_bf16(seed, _S_VL, (LB, Hkv, D))
    k_pre = _normal_bf16(seed, _S_KP, (P, Hkv, D))
    v_pre = _normal_bf16(seed, _S_VP, (P, Hkv, D))

    n_ref = int(round(cfg["refresh_frac"] * P))
    if n_ref:
        g = np.random.default_rng([seed, _S_REFIDX])
        refresh_idx = np.sort(g.choice(P, n_ref, replace=False)).astype(np.int32)
    else:
        refresh_idx = np.zeros(0, dtype=np.int32)
    q_ref = _normal_bf16(seed, _S_QREF, (n_ref, Hq, D))
    k_ref = _normal_bf16(seed, _S_KREF, (n_ref, Hkv, D))
    v_ref = _normal_bf16(seed, _S_VREF, (n_ref, Hkv, D))

    g = np.random.default_rng([seed, _S_H])
    h = g.standard_normal((LB, d), dtype=np.float32)
    s_row = np.random.default_rng([seed, _S_HSCALE]).uniform(1.0, 6.0, LB).astype(np.float32)
    hidden = f32_to_bf16_bits(h * s_row[:, None])
    W = lm_head_weight(seed, V, d) if with_weight else None

    n_mask = int(round(cfg["mask_frac"] * LB))
    gm = np.random.default_rng([seed, _S_MASK])
    row_pos = np.sort(gm.choice(LB, n_mask, replace=False)).astype(np.int32)
    is_masked = np.zeros(LB, dtype=np.uint8)
    is_masked[row_pos] = 1
    gt = np.random.default_rng([seed, _S_TOK])
    tokens = gt.integers(FIRST_ORDINARY_ID, max(V, FIRST_ORDINARY_ID + 1), LB).astype(np.int32)
    if cfg["delim_frac"] > 0:
        gd = np.random.default_rng([seed, _S_DELIM])
        committed = np.nonzero(is_masked == 0)[0]
        nd = int(round(cfg["delim_frac"] * len(committed)))
        pick = gd.choice(committed, nd, replace=False)
        tokens[pick] = gd.choice(np.asarray(DELIM_IDS), nd)
    tokens[is_masked == 1] = -1
    suppress_eos = (role[row_pos // B] == ROLE_REF).astype(np.uint8)

    return DecodeStep(
        name=name, seed=seed, Hq=Hq, Hkv=Hkv, D=D, P=P, L=L, B=B, d=d, V=V,
        parent=parent, role=role, b_len=b_len, t_lane=t_lane,
        q=q, k_lane=k_lane, v_lane=v_lane, k_pre=k_pre, v_pre=v_pre,
        refresh_idx=refresh_idx, q_ref=q_ref, k_ref=k_ref, v_ref=v_ref,
        hidden=hidden, W=W, tokens=tokens, is_masked=is_masked,
        row_pos=row_pos, suppress_eos=suppress_eos,
        tau=float(cfg["tau"]), fallback_k=int(cfg["fallback_k"]),
    )


def random_confidences(seed: int, N: int, V: int, tie_levels: int = 0):
    """Random (conf, argmax) pairs for exercising selection alone.

    With tie_levels > 0, conf takes values k/tie_levels so exact ties occur.
    """
    g = np.random.default_rng([seed, 21])
    if tie_levels:
        conf = (g.integers(0, tie_levels + 1, N) / tie_levels).astype(np.float32)
    else:
        conf = g.uniform(0.0, 1.0, N).astype(np.float32)
    argmax = g.integers(0, V, N).astype(np.int32)
    return conf, argmax
