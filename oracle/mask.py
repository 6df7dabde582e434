"""Oracle: mean-pool block-score mask builder with joint top-p / top-k selection.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The paper's online predictor scores block pairs by softmax(mean(Q) mean(K)^T)
(Sec. 3.2, Obs. 2), and masks are selected "via top-p with a top-k floor"
(Sec. 3.2, Mask Caching and Retrieval) where the floor keeps at least a
fraction ``min_top_k`` of the key blocks (Sec. 3.2, Minimum top-k guarantee;
knobs ``top_p`` / ``min_top_k`` in Sec. 4.1).  Steps, for one source request
and one head, in the paper's order:

1. Pool   q_i = mean of Q over the valid tokens of block i (float64 sum,
          divided by the valid-token count), k_j likewise.
2. Score  s_ij = sm_scale * <q_i, k_j>   (float64).
3. Mass   p_ij = softmax_j(s_ij) over all n kv-blocks of the row.
4. Order  j sorted by (s_ij descending, j ascending).
5. Top-p  k_p = the smallest k >= 1 whose cumulative mass in that order is
          >= top_p; k_p = 0 when top_p <= 0 and k_p = n when top_p >= 1.
6. Floor  k_min = ceil(min_top_k * n - 1e-9).
7. Keep   k = min(n, max(k_p, k_min, 1)) first blocks of the order, emitted
          in ascending block id (one CSR row).

Readings where the paper is silent (listed with the others in the design
notes): the sm_scale factor on the pooled scores (ranking is unaffected, only
the top-p mass is), pooling over valid tokens only, ">=" at the top-p
boundary, the floor applied per (head, q-block) row, never fewer than one
block per row, and index-ascending tie breaking.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

BLOCK = 64
FLOOR_EPS = 1e-9


def pool_means(xh, block: int = BLOCK) -> np.ndarray:
    """Step 1: per-block mean over valid tokens of ``xh [S, D]`` -> ``[n, D]``."""
    xh = np.asarray(xh, dtype=np.float64)
    S, D = xh.shape
    n = (S + block - 1) // block
    out = np.empty((n, D), dtype=np.float64)
    for i in range(n):
        seg = xh[i * block:min(i * block + block, S)]
        out[i] = seg.sum(axis=0) / seg.shape[0]
    return out


def block_scores(qbar: np.ndarray, kbar: np.ndarray, sm_scale: float) -> np.ndarray:
    """Step 2: s = sm_scale * qbar kbar^T in float64, ``[n_q, n_kv]``."""
    return sm_scale * (np.asarray(qbar, np.float64) @ np.asarray(kbar, np.float64).T)


def row_mass(s_row: np.ndarray) -> np.ndarray:
    """Step 3: softmax over one row of block scores."""
    e = np.exp(s_row - s_row.max())
    return e / e.sum()


def row_order(s_row: np.ndarray) -> np.ndarray:
    """Step 4: indices by (score descending, index ascending)."""
    n = s_row.shape[0]
    return np.lexsort((np.arange(n), -s_row))


def top_p_count(mass_sorted: np.ndarray, top_p: float) -> int:
    """Step 5: smallest k >= 1 with cumulative mass >= top_p."""
    n = mass_sorted.shape[0]
    if top_p <= 0.0:
        return 0
    if top_p >= 1.0:
        return n
    c = np.cumsum(mass_sorted)
    hit = np.nonzero(c >= top_p)[0]
    return int(hit[0]) + 1 if hit.size else n


def floor_count(min_top_k: float, n: int) -> int:
    """Step 6: the top-k floor."""
    return int(math.ceil(min_top_k * n - FLOOR_EPS))


def select_row(s_row, top_p: float, min_top_k: float) -> np.ndarray:
    """Steps 3-7 for one row; returns kept block ids ascending."""
    s_row = np.asarray(s_row, dtype=np.float64)
    n = s_row.shape[0]
    order = row_order(s_row)
    mass = row_mass(s_row)
    kp = top_p_count(mass[order], top_p)
    k = min(n, max(kp, floor_count(min_top_k, n), 1))
    return np.sort(order[:k])


@dataclass
class OracleMask:
    """CSR block mask: rows ``(b * H + h) * n + i``; ascending kv ids."""
    row_ptr: np.ndarray   # int64 [R + 1]
    col_idx: np.ndarray   # int64 [nnz]
    scores: np.ndarray    # float64 [R, n]
    n_blocks: int          # q-blocks per head (rows per head)
    H: int
    mask_batch: int
    n_kv: int = 0          # kv blocks per row (columns); 0 means n_blocks

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])

    @property
    def columns(self) -> int:
        return self.n_kv or self.n_blocks

    @property
    def density(self) -> float:
        R = self.row_ptr.shape[0] - 1
        return self.nnz / float(R * self.columns)

    def row(self, r: int) -> np.ndarray:
        return self.col_idx[self.row_ptr[r]:self.row_ptr[r + 1]]


def build_block_mask(q, k, sm_scale: float, top_p: float, min_top_k: float,
                     block: int = BLOCK, heads=None, kv_block: int | None = None) -> OracleMask:
    """Steps 1-7 for every request b and head h of ``q, k [B, S, H, D]``.

    Queries are pooled over blocks of ``block`` tokens (the mask's rows), keys
    over blocks of ``kv_block`` tokens (its columns; default ``block``): the
    paper's own kernel pairs q-blocks of 64 with kv blocks of 128.  ``heads``
    optionally restricts the heads built (rows of other heads are left
    empty); used to time a bounded sample.
    """
    kvb = block if kv_block is None else kv_block
    B, S, H, D = q.shape
    n = (S + block - 1) // block
    nk = (S + kvb - 1) // kvb
    counts = np.zeros(B * H * n, dtype=np.int64)
    rows = [None] * (B * H * n)
    scores = np.zeros((B * H * n, nk), dtype=np.float64)
    for b in range(B):
        for h in (range(H) if heads is None else heads):
            s = block_scores(pool_means(q[b, :, h, :], block), pool_means(k[b, :, h, :], kvb),
                             sm_scale)
            for i in range(n):
                r = (b * H + h) * n + i
                sel = select_row(s[i], top_p, min_top_k)
                rows[r] = sel
                counts[r] = sel.shape[0]
                scores[r] = s[i]
    row_ptr = np.zeros(B * H * n + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    col_idx = np.concatenate([x for x in rows if x is not None]) if row_ptr[-1] else \
        np.zeros(0, np.int64)
    return OracleMask(row_ptr, col_idx.astype(np.int64), scores, n, H, B, nk)
