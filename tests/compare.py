"""Comparators between the HIP path's results and the oracle's (test helpers).

Mask rule: a GPU row G and an oracle row O (sets of kv-block ids) agree when
they are equal; otherwise every id in G \\ O must pair one-to-one, in score
order, with an id in O \\ G whose float64 oracle score is within 1e-6
relative (a near-tie where either choice is correct), and |G| may differ from
|O| by one only when the oracle's cumulative mass at the top-p boundary is
within 1e-6 of top_p (a near-tie of the stopping rule).
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from oracle import mask as om

TIE_REL = 1e-6
BOUNDARY = 1e-6


@dataclass
class MaskReport:
    exact: int = 0
    excused: int = 0
    failing: list = field(default_factory=list)

    @property
    def ok(self) -> bool:
        return not self.failing


def compare_row(g_row, o_row, scores, top_p: float, min_top_k: float):
    """Returns 'exact', 'excused' or a failure description."""
    G, O = set(int(x) for x in g_row), set(int(x) for x in o_row)
    if len(g_row) != len(G) or list(g_row) != sorted(G):
        return "gpu row not strictly ascending"
    if G == O:
        return "exact"
    n = scores.shape[0]
    if len(G) != len(O):
        if abs(len(G) - len(O)) != 1:
            return f"count {len(G)} vs {len(O)}"
        order = om.row_order(scores)
        c = np.cumsum(om.row_mass(scores)[order])
        kp = om.top_p_count(om.row_mass(scores)[order], top_p)
        near = [c[k - 1] for k in (kp - 1, kp) if 1 <= k <= n]
        if not any(abs(x - top_p) <= BOUNDARY for x in near):
            return f"count {len(G)} vs {len(O)} away from the top-p boundary"
    extra = sorted(G - O, key=lambda j: (-scores[j], j))
    missing = sorted(O - G, key=lambda j: (-scores[j], j))
    for a, b in zip(extra, missing):
        sa, sb = scores[a], scores[b]
        if abs(sa - sb) > TIE_REL * max(abs(sa), abs(sb)):
            return f"block {a} (s={sa!r}) vs {b} (s={sb!r}) not a near-tie"
    if abs(len(extra) - len(missing)) > 1:
        return "unpaired differences"
    return "excused"


def compare_masks(g_rp, g_ci, o_mask, rows, top_p, min_top_k) -> MaskReport:
    rep = MaskReport()
    for r in rows:
        g_row = g_ci[g_rp[r]:g_rp[r + 1]]
        res = compare_row(g_row, o_mask.row(r), o_mask.scores[r], top_p, min_top_k)
        if res == "exact":
            rep.exact += 1
        elif res == "excused":
            rep.excused += 1
        else:
            rep.failing.append((r, res))
    return rep


def max_abs_err(a, b) -> float:
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))
