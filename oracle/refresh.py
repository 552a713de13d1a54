"""Compact cache refresh window (fp64/int oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 3.4, "Compact cache refresh and reuse": instead of the whole
prompt-plus-generation sequence, a refresh re-encodes only the meaningful
prefix plus a small margin,

    L_refresh = min(P + L, P + L_eff + m),   L_eff = max over lanes (s + v),

with P the prompt length, L the generation length, s a lane's start and v
its valid prefix length (generation coordinates), m the margin.  With no
lanes L_eff is taken as 0.  The refresh forward is bidirectional over the
window: every row of [0, L_refresh) attends to every row of the window
(``attention.decode_attention`` / ``refresh_attention`` on a prefix cut to
L_refresh rows with every row refreshed), and its logits for the window's
generation rows are reused by the next iteration's transfer and lookahead
drafts instead of a new LM-head pass.
"""


def refresh_window_len(P, L, lane_start, valid_len, margin):
    """L_refresh of the equation above (integers)."""
    assert len(lane_start) == len(valid_len)
    l_eff = 0
    for s, v in zip(lane_start, valid_len):
        l_eff = max(l_eff, int(s) + int(v))
    return min(int(P) + int(L), int(P) + l_eff + int(margin))
