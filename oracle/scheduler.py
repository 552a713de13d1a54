"""Active-lane scheduler (Algorithm "AsyncLane active-lane decoding"), plain
Python.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 3.2 (fork operator eq. fork_operator, "Advancement control") and
Section 3.3 (active-lane scheduling, output reconstruction), Section 3.4
(model-call NFE accounting).  Readings (the paper leaves them open):

* Generation coordinates 0..L-1.  A lane has a role (gen/ref), a start s, a
  length b (its valid update region [s, s+b)), a prefix-state group, a
  local step count t and an ordered child list.  The root is a generate
  lane at s = 0, b = min(B, L), group 0.
* Each iteration evaluates the active lanes (in depth-first tree order,
  refine children before generate children; at most max_lanes of them).
  Lane i's block is positions [s, s+W), W = B + window (the lookahead
  window of eq. lane_input); positions past L are filled padding.  The
  transfer, drafts and lane statistics are select_unmask's
  (``select.select_unmask``), fed one (conf, argmax) per masked block row,
  rows in lane order then position order.
* The step condition of eq. fork_condition sees the lane's step count
  including the current step (t + 1).
* Write-back: first every lane's update region, then window drafts into
  positions still masked.  Every evaluated lane's t grows by one.
* Transitions, in plan order, from the lane statistics:
  - generate lane with fork_ok: fork at p = split (eq. fork_operator):
    refine child (s, p) and, when s + p < L, generate child
    (s + p, min(B, L - s - p)), both in a new group; the lane is done;
  - otherwise a lane whose region is filled (n_filled = b) is completed:
    a refine lane is done; a generate lane with valid length v = 0, or
    s + v >= L, stops advancing (done); else it is done and spawns a
    successor generate lane (s + v, min(B, L - s - v)) in a new group.
* The call for an iteration is one batched model call per prefix-state
  group (NFE_t = |G_t|); NFE = 1 (prompt) + sum of |G_t| (no refresh here).
* Output (CollectDFS): a forked lane emits its refine child, then its
  generate child; a lane that spawned a successor emits [s, s+v) then the
  successor; a leaf emits [s, s+b) cut before its first mask, and a
  generate leaf also before its first EOS (EOS itself is not emitted).
"""
import numpy as np

from . import select as sel

GEN, REF = sel.ROLE_GEN, sel.ROLE_REF


class Lane:
    def __init__(self, lid, role, s, b, parent, group):
        self.id, self.role, self.s, self.b = lid, role, s, b
        self.parent, self.group = parent, group
        self.done = False
        self.t = 0
        self.children = []   # ids, creation order
        self.kind = None     # "fork" | "spawn" | None (how children were made)
        self.v = None        # valid length when a successor was spawned


class Scheduler:
    def __init__(self, P, L, B, window=0, max_lanes=64, pad_id=3):
        self.P, self.L, self.B, self.window, self.max_lanes = P, L, B, window, max_lanes
        self.pad_id = pad_id
        self.W = B + window
        self.tokens = np.full(L, -1, np.int32)
        self.masked = np.ones(L, np.uint8)
        self.lanes = [Lane(0, GEN, 0, min(B, L), -1, 0)]
        self.next_group = 1
        self.iterations = 0
        self.nfe = 1
        self.forks = self.spawns = self.stops = 0
        self.plans = []      # per plan() call: (lane ids in order, call parents)

    # ---------------------------------------------------------------- plan
    def _dfs(self, lid, out):
        ln = self.lanes[lid]
        if not ln.done:
            out.append(lid)
        for c in ln.children:
            self._dfs(c, out)

    def plan(self):
        order = []
        self._dfs(0, order)
        order = order[:self.max_lanes]
        call_parent = []
        for k, lid in enumerate(order):
            ln = self.lanes[lid]
            cp = -1
            if ln.role == GEN and ln.parent >= 0 and self.lanes[ln.parent].kind == "fork":
                sib = self.lanes[ln.parent].children[0]     # the refine sibling
                if sib in order[:k] and self.lanes[sib].group == ln.group:
                    cp = order.index(sib)
            call_parent.append(cp)
        self.plans.append((list(order), list(call_parent)))
        return order, call_parent

    def blocks(self, order):
        n, W = len(order), self.W
        tk = np.full(n * W, self.pad_id, np.int32)   # padding past L: filled
        mk = np.zeros(n * W, np.uint8)
        for i, lid in enumerate(order):
            s = self.lanes[lid].s
            for a in range(W):
                if s + a < self.L:
                    tk[i * W + a] = self.tokens[s + a]
                    mk[i * W + a] = self.masked[s + a]
        return tk, mk

    # -------------------------------------------------------------- commit
    def commit(self, order, blk_tok, blk_msk, stats):
        W, L = self.W, self.L
        for phase in ("region", "window"):
            for i, lid in enumerate(order):
                ln = self.lanes[lid]
                rng = range(0, ln.b) if phase == "region" else range(ln.b, W)
                for a in rng:
                    pos = ln.s + a
                    if pos < L and self.masked[pos] and not blk_msk[i * W + a]:
                        self.tokens[pos] = blk_tok[i * W + a]
                        self.masked[pos] = 0
        groups = set(self.lanes[lid].group for lid in order)
        self.nfe += len(groups)
        self.iterations += 1
        for lid in order:
            self.lanes[lid].t += 1
        for i, lid in enumerate(order):
            ln = self.lanes[lid]
            st = stats[i]
            if ln.role == GEN and st[sel.STAT_FORK]:
                p = int(st[sel.STAT_SPLIT])
                g = self.next_group
                self.next_group += 1
                self._add(lid, REF, ln.s, p, g)
                if ln.s + p < L:
                    self._add(lid, GEN, ln.s + p, min(self.B, L - ln.s - p), g)
                ln.kind = "fork"
                ln.done = True
                self.forks += 1
            elif int(st[sel.STAT_FILLED]) == ln.b:
                ln.done = True
                if ln.role == GEN:
                    v = int(st[sel.STAT_VALID])
                    if v == 0 or ln.s + v >= L:
                        self.stops += 1
                    else:
                        g = self.next_group
                        self.next_group += 1
                        self._add(lid, GEN, ln.s + v, min(self.B, L - ln.s - v), g)
                        ln.kind = "spawn"
                        ln.v = v
                        self.spawns += 1
        return sum(1 for x in self.lanes if not x.done)

    def _add(self, parent, role, s, b, group):
        lid = len(self.lanes)
        self.lanes.append(Lane(lid, role, s, b, parent, group))
        self.lanes[parent].children.append(lid)

    # ------------------------------------------------------------- collect
    def collect(self, eos_id=2):
        out = []

        def emit(lid):
            ln = self.lanes[lid]
            if ln.kind == "fork":
                for c in ln.children:
                    emit(c)
            elif ln.kind == "spawn":
                out.extend(int(x) for x in self.tokens[ln.s:ln.s + ln.v])
                emit(ln.children[0])
            else:
                for a in range(ln.b):
                    pos = ln.s + a
                    if self.masked[pos] or (ln.role == GEN and self.tokens[pos] == eos_id):
                        break
                    out.append(int(self.tokens[pos]))
        emit(0)
        return out


def run(P, L, B, window, conf_fn, max_iters, max_lanes=64, mode=sel.MODE_THRESHOLD, tau=0.9,
        fallback_k=1, tau_future=None, delim_ids=(0, 1), eos_id=2, rho_min=0.5, t_min=2):
    """Drive the scheduler with the oracle selection.  conf_fn(iteration,
    order, lanes, positions) returns (conf, argmax) for the masked block rows
    (flat block positions, ascending).  Returns the scheduler."""
    s = Scheduler(P, L, B, window, max_lanes)
    for it in range(max_iters):
        order, _ = s.plan()
        if not order:
            break
        tk, mk = s.blocks(order)
        rows = np.flatnonzero(mk).astype(np.int32)
        conf, arg = conf_fn(it, order, s.lanes, rows)
        ln = [s.lanes[x] for x in order]
        res = sel.select_unmask(conf, arg, rows, tk, mk, s.W, np.array([x.role for x in ln], np.uint8),
                                np.array([x.b for x in ln], np.int32), np.array([x.t + 1 for x in ln], np.int32),
                                mode, tau, fallback_k, None, delim_ids, eos_id, rho_min, t_min,
                                tau_future=tau_future)
        s.commit(order, res["tokens"], res["is_masked"], res["lane_stats"])
    return s
