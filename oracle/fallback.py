"""Oracle: block-pair visit refreshing, the first safeguard of the safety
fallback (float-free set logic, plain NumPy booleans).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Sec. 3.2 "Safety fallback against information loss", (1) block-pair visit
refreshing: a binary map V[h, q, k] records, for the current request, which
(head, q-block, kv-block) pairs the sparse masks of the current layer group
have activated.  Layers are grouped N at a time (``layer_flash``, N = 8 in
Sec. 4.1).  Inside a group V is updated layer by layer; at the group's last
layer every pair still unvisited is forced into that layer's mask, so every
pair is touched at least once per group; V is cleared when the next group
starts.  Written out for one group of masks M_1 .. M_N (sets of pairs):

    V_0 = {}
    V_l = V_{l-1} | M_l                 for l < N   (masks used as given)
    M_N' = M_N | (all pairs - V_{N-1})  (the last layer's mask after refresh)

so V_{N-1} | M_N' covers every pair.  (2) the minimum top-k guarantee is the
floor of the selection rule (``mask.select_row``).
"""

from __future__ import annotations

import numpy as np


def dense_of(row_ptr, col_idx, rows: int, n: int) -> np.ndarray:
    """Boolean [rows, n] view of a CSR mask."""
    D = np.zeros((rows, n), dtype=bool)
    for r in range(rows):
        D[r, col_idx[row_ptr[r]:row_ptr[r + 1]]] = True
    return D


def csr_of(D: np.ndarray):
    """CSR (ascending ids) of a boolean [rows, n] map."""
    rows, n = D.shape
    counts = D.sum(axis=1).astype(np.int64)
    row_ptr = np.zeros(rows + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    col_idx = np.concatenate([np.nonzero(D[r])[0] for r in range(rows)]).astype(np.int64) \
        if counts.sum() else np.zeros(0, np.int64)
    return row_ptr, col_idx


def visit_update(V: np.ndarray, mask_dense: np.ndarray) -> np.ndarray:
    """V_l = V_{l-1} | M_l."""
    return V | mask_dense


def visit_refresh(V: np.ndarray, mask_dense: np.ndarray) -> np.ndarray:
    """The group's last layer: M_N | (all pairs not visited by the layers before it)."""
    return mask_dense | ~V


def run_group(masks, n: int):
    """Masks of one layer group (boolean [rows, n] each) -> the masks the
    layers actually use (all but the last unchanged) and the final map."""
    V = np.zeros_like(masks[0])
    used = []
    for l, M in enumerate(masks):
        if l + 1 < len(masks):
            used.append(M)
            V = visit_update(V, M)
        else:
            last = visit_refresh(V, M)
            used.append(last)
            V = visit_update(V, last)
    return used, V
