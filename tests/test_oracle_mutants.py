"""Plant plausible mistakes in copies of the oracle (on the CPU) and check
that the pins catch every one of them.

Each mutant is a textual edit of one oracle module's source; the edited
source is executed as a fresh module and every pin of that module is run
against it.  At least one pin must fail, otherwise the pins would not have
noticed that mistake in the oracle itself.
"""
import importlib.util
import os
import types

import pytest

import pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    "attention": [
        ("drop softmax scale", "s = scale * (q @ k.T)", "s = (q @ k.T)"),
        ("modular GQA head map (form A)", "kc[:, h // g], vc[:, h // g]", "kc[:, h % Hkv], vc[:, h % Hkv]"),
        ("modular GQA head map (form B)", "k_all[:, h // g].T", "k_all[:, h % Hkv].T"),
        ("ancestors dropped", "blocks = anc[i] + [i]", "blocks = [i]"),
        ("own block dropped", "blocks = anc[i] + [i]", "blocks = anc[i] if anc[i] else [i]"),
        ("parent only, no deeper ancestors", "for _ in range(L):\n        R = R |", "for _ in range(1):\n        R = R |"),
        ("siblings visible", "adj[i, parent[i]] = True", "adj[i, parent[i]] = True\n            adj[i, [x for x in range(L) if parent[x] == parent[i]]] = True"),
        ("softmax not normalised", "return p @ v, (m + np.log(l))[:, 0]", "return e @ v, (m + np.log(l))[:, 0]"),
        ("value operand swapped", "return p @ v, (m", "return p @ k, (m"),
        ("lse without max", "return p @ v, (m + np.log(l))[:, 0]", "return p @ v, np.log(l)[:, 0]"),
        ("row form skips ancestors", "        blocks = anc[i] + [i]\n        for b, h in enumerate(heads):",
         "        blocks = [i]\n        for b, h in enumerate(heads):"),
        ("row form modular GQA", "            kv = h // g\n", "            kv = h % Hkv\n"),
        ("refresh writes wrong row", "k2[int(p)] = k_ref[r]", "k2[r] = k_ref[r]"),
        ("refresh rows see their own row only", "o, lse = softmax_attend(q_ref[:, h], k_pre[:, h // g], v_pre[:, h // g], scale)",
         "o, lse = softmax_attend(q_ref[:, h], k_pre[:n, h // g], v_pre[:n, h // g], scale)"),
    ],
    "lmhead": [
        ("last index on ties", "ids[np.flatnonzero(zn == m)[0]]", "ids[np.flatnonzero(zn == m)[-1]]"),
        ("EOS never suppressed", "allowed[eos_id] = False", "pass"),
        ("conf without max", "out[\"conf\"][n] = np.exp(m - lse)", "out[\"conf\"][n] = np.exp(-lse)"),
        ("chunk merge forgets rescale", "s[n] = s[n] * np.exp(m[n] - mc) + sc", "s[n] = s[n] + sc"),
        ("chunk merge takes later index on ties", "elif mc == m[n]:\n                s[n] = s[n] + sc",
         "elif mc == m[n]:\n                s[n] = s[n] + sc\n                idx[n] = ic"),
        ("chunk merge wrong sign", "s[n] = s[n] + sc * np.exp(mc - m[n])", "s[n] = s[n] + sc * np.exp(m[n] - mc)"),
        ("chunked EOS never suppressed", "zn[eos_id - c0] = -np.inf", "pass"),
        ("gathered rows ignored",
         "H = np.asarray(hidden, dtype=dtype)[np.asarray(row_idx, dtype=np.int64)]\n    V = W.shape[0]\n    z",
         "H = np.asarray(hidden, dtype=dtype)[:len(row_idx)]\n    V = W.shape[0]\n    z"),
        ("lse drops log", "lse = m + np.log(np.exp(zn - m).sum())", "lse = m + np.exp(zn - m).sum()"),
    ],
    "select": [
        ("strict threshold", "if conf32[n] >= tau32]", "if conf32[n] > tau32]"),
        ("ties broken by later position", "(-float(conf32[n]), int(row_pos[n]))", "(-float(conf32[n]), -int(row_pos[n]))"),
        ("ascending confidence order", "(-float(conf32[n]), int(row_pos[n]))", "(float(conf32[n]), int(row_pos[n]))"),
        ("fallback always added", "if not chosen and fallback_k > 0:", "if fallback_k > 0:"),
        ("b_len boundary inclusive", "row_pos[n] % B < b_len[lane]", "row_pos[n] % B <= b_len[lane]"),
        ("unmasked rows also candidates", "and is_masked[row_pos[n]]]", "]"),
        ("split without +1", "split = i + 1", "split = i"),
        ("valid length off by one", "valid = i\n", "valid = i + 1\n"),
        ("EOS does not end the valid prefix", "(masked or tok == eos_id)", "(masked)"),
        ("masked delimiters counted", "if not masked:\n                filled += 1\n                if tok in dset and",
         "if True:\n                filled += not masked\n                if tok in dset and"),
        ("strict fill ratio", "np.float32(filled) >= np.float32(rho_min)", "np.float32(filled) > np.float32(rho_min)"),
        ("fill ratio in fp64", "np.float32(filled) >= np.float32(rho_min) * np.float32(n)", "filled >= rho_min * n"),
        ("refine lanes fork", "int(role[lane]) == ROLE_GEN and", "True and"),
        ("step condition ignored", "and int(t_lane[lane]) >= int(t_min))", ")"),
        ("top-k takes k+1", "chosen = order[:max(0, min(int(k_lane[lane]), len(cand)))]",
         "chosen = order[:max(0, min(int(k_lane[lane]) + 1, len(cand)))]"),
        ("refine lanes draft", "if (int(role[lane]) == ROLE_GEN and i >= int(b_len[lane])",
         "if (True and i >= int(b_len[lane])"),
        ("window starts after b_len", "and i >= int(b_len[lane]) and is_masked[pos]",
         "and i > int(b_len[lane]) and is_masked[pos]"),
        ("strict draft threshold", "and conf32[n] >= tf32 and", "and conf32[n] > tf32 and"),
        ("EOS drafted", "and int(argmax[n]) != int(eos_id)):", "):"),
        ("unmasked window rows drafted", "and is_masked[pos]\n                    and conf32", "\n                    and conf32"),
        ("drafts counted as transfers", "elif flag[n] == 2:\n            stats[row_pos[n] // B, STAT_NDRAFT] += 1",
         "elif flag[n] == 2:\n            stats[row_pos[n] // B, STAT_NSEL] += 1"),
        ("drafts left out of unmasked_pos", "unmasked_pos = row_pos[flag != 0]", "unmasked_pos = row_pos[flag == 1]"),
        ("digit test reads the next position", "int(tokens[start + i - 1]) in set(digit_ids)",
         "start + i + 1 < len(tokens) and int(tokens[start + i + 1]) in set(digit_ids)"),
        ("digit test ignores the mask", "if i > 0 and not is_masked[start + i - 1] and", "if i > 0 and"),
        ("strictly negative depth required", "return depth <= 0", "return depth < 0"),
        ("masked brackets counted", "        if is_masked[start + j]:\n            continue\n", ""),
        ("close brackets ignored", "depth -= 1", "depth -= 0"),
        ("ValidBoundary ignored", "if tok in dset and valid_boundary(", "if tok in dset and True or valid_boundary("),
    ],
    "refresh": [
        ("margin dropped", "int(P) + l_eff + int(margin))", "int(P) + l_eff)"),
        ("no clip at the sequence end", "return min(int(P) + int(L), int(P) + l_eff + int(margin))",
         "return int(P) + l_eff + int(margin)"),
        ("frontier without the lane start", "l_eff = max(l_eff, int(s) + int(v))", "l_eff = max(l_eff, int(v))"),
        ("first lane only", "l_eff = max(l_eff, int(s) + int(v))", "l_eff = l_eff or int(s) + int(v)"),
        ("prompt left out", "int(P) + l_eff + int(margin))", "l_eff + int(margin))"),
    ],
    "scheduler": [
        ("generate child before refine child", "        self._dfs(0, order)\n",
         "        self._dfs(0, order)\n        order = sorted(order, key=lambda x: self.lanes[x].role)\n"),
        ("step count without the current step", "np.array([x.t + 1 for x in ln], np.int32)",
         "np.array([x.t for x in ln], np.int32)"),
        ("successor after the whole lane", "self._add(lid, GEN, ln.s + v, min(self.B, L - ln.s - v), g)",
         "self._add(lid, GEN, ln.s + ln.b, min(self.B, L - ln.s - ln.b), g) if ln.s + ln.b < L else None"),
        ("no cascade stop", "if v == 0 or ln.s + v >= L:", "if ln.s + v >= L:"),
        ("EOS emitted", "if self.masked[pos] or (ln.role == GEN and self.tokens[pos] == eos_id):",
         "if self.masked[pos]:"),
        ("NFE counts lanes", "self.nfe += len(groups)", "self.nfe += len(order)"),
        ("fork children share the parent group", "                g = self.next_group\n                self.next_group += 1\n                self._add(lid, REF",
         "                g = ln.group\n                self._add(lid, REF"),
        ("refine lanes spawn", "                if ln.role == GEN:\n                    v = int(st[sel.STAT_VALID])",
         "                if True:\n                    v = int(st[sel.STAT_VALID])"),
    ],
}

CHECKS = {"attention": pins.ATTENTION_CHECKS, "lmhead": pins.LMHEAD_CHECKS,
          "select": pins.SELECT_CHECKS, "refresh": pins.REFRESH_CHECKS,
          "scheduler": pins.SCHEDULER_CHECKS}


def _mutated(module, old, new):
    path = os.path.join(ROOT, "oracle", module + ".py")
    src = open(path).read()
    assert old in src, f"mutation anchor not found in oracle/{module}.py: {old!r}"
    mod = types.ModuleType(f"oracle_mutant_{module}")
    mod.__file__ = path
    mod.__package__ = "oracle"      # relative imports resolve to the real oracle modules
    exec(compile(src.replace(old, new), path, "exec"), mod.__dict__)
    return mod


CASES = [(m, name, old, new) for m, lst in MUTANTS.items() for (name, old, new) in lst]


@pytest.mark.parametrize("module,name,old,new", CASES, ids=[f"{c[0]}:{c[1]}" for c in CASES])
def test_pins_catch_mutant(module, name, old, new):
    mod = _mutated(module, old, new)
    caught = []
    for check in CHECKS[module]:
        try:
            check(mod)
        except Exception as e:  # any failure (assertion or crash) counts
            caught.append((check.__name__, type(e).__name__))
    assert caught, f"no pin caught mutant '{name}' of oracle/{module}.py"
