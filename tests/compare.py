"""Comparators between the HIP path's results and the oracle's (test helpers).

Mask rule (per row; G = the GPU's kv ids, O = the oracle's, both sets):

* G = O: the row is exact.
* Otherwise G must be a prefix of the oracle's own order (score descending,
  index ascending) up to near-ties: with P = the first |G| ids of that order,
  the ids of G \\ P and of P \\ G, each taken in score order, pair one to one
  and every pair is a near-tie (scores within ``TIE_REL`` relative, where
  either choice is correct).  An id of G that is not in P and not a near-tie
  of the id it displaces fails the row, whatever the counts.
* |G| may differ from |O| by exactly one, and only where the top-p rule set
  the count: the smaller count is at least the floor max(k_min, 1) (so the
  floor did not fix both), and the oracle's cumulative mass after that many
  blocks is within ``BOUNDARY`` of top_p (the stopping test could go either
  way).

The tolerances default to the builder's (float64 scores on both sides);
selection from GPU block masses passes looser ones derived from the mass
error bound (``tie=`` and ``boundary=``).
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from oracle import mask as om

TIE_REL = 1e-6
BOUNDARY = 1e-6


def rel_tie(sa: float, sb: float) -> bool:
    return abs(sa - sb) <= TIE_REL * max(abs(sa), abs(sb))


@dataclass
class MaskReport:
    exact: int = 0
    excused: int = 0
    failing: list = field(default_factory=list)

    @property
    def ok(self) -> bool:
        return not self.failing


def compare_row(g_row, o_row, scores, top_p: float, min_top_k: float, tie=rel_tie,
                boundary: float = BOUNDARY):
    """Returns 'exact', 'excused' or a failure description.

    ``scores`` are the oracle's float64 scores of the row (for selection from
    block masses: log-masses, whose softmax is the mass share); ``tie(sa, sb)``
    decides whether two scores are a near-tie."""
    G = set(int(x) for x in g_row)
    O = set(int(x) for x in o_row)
    if len(g_row) != len(G) or list(int(x) for x in g_row) != sorted(G):
        return "gpu row not strictly ascending"
    if G == O:
        return "exact"
    n = scores.shape[0]
    if any(j < 0 or j >= n for j in G):
        return "gpu id out of range"
    kg, ko = len(G), len(O)
    order = om.row_order(scores)
    if kg != ko:
        if abs(kg - ko) != 1:
            return f"count {kg} vs {ko}"
        k_lo = min(kg, ko)
        k_floor = max(om.floor_count(min_top_k, n), 1)
        if k_lo < k_floor:
            return f"count {kg} vs {ko} where the floor {k_floor} sets the count"
        c = np.cumsum(om.row_mass(scores)[order])
        if abs(c[k_lo - 1] - top_p) > boundary:
            return f"count {kg} vs {ko} away from the top-p boundary (C={c[k_lo - 1]!r})"
    P = set(int(j) for j in order[:kg])
    key = lambda j: (-scores[j], j)
    extra = sorted(G - P, key=key)
    missing = sorted(P - G, key=key)
    for a, b in zip(extra, missing):
        if not tie(scores[a], scores[b]):
            return f"block {a} (s={scores[a]!r}) in place of {b} (s={scores[b]!r}): not a near-tie"
    return "excused"


def compare_masks(g_rp, g_ci, o_mask, rows, top_p, min_top_k, tie=rel_tie,
                  boundary: float = BOUNDARY) -> MaskReport:
    rep = MaskReport()
    for r in rows:
        g_row = g_ci[g_rp[r]:g_rp[r + 1]]
        res = compare_row(g_row, o_mask.row(r), o_mask.scores[r], top_p, min_top_k, tie, boundary)
        if res == "exact":
            rep.exact += 1
        elif res == "excused":
            rep.excused += 1
        else:
            rep.failing.append((r, res))
    return rep


def max_abs_err(a, b) -> float:
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))
