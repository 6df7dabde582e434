"""Oracle: true block attention mass, the top-p / top-k mask taken from it,
and the coverage of a mask on a request (float64, plain NumPy).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The paper's high-quality masks are not predicted: a historical request runs
dense attention anyway, and a block mask is selected from its attention map
by top-p with a top-k floor and stored for reuse (Sec. 3.2, "Mask Caching and
Retrieval").  A mask is judged by its coverage, the fraction of a target
request's true token-level attention mass that lies in the blocks it selects
(Sec. 3.2, Obs. 1).  Written out for one request b and head h, with dense
attention probabilities P[r, c] = softmax_c(sm_scale <q_r, k_c>) over all
keys c < S:

    M[i, j]  = (1 / |T_i|) * sum_{r in T_i} sum_{c in T_j} P[r, c]
               (T_i: the valid tokens of block i; every row of M sums to 1)
    mask row i = the blocks kept when the row M[i, :] is ranked by (M
               descending, j ascending) and cut at cumulative mass >= top_p
               with the top-k floor -- the same rule as the pooled-score
               predictor (``mask.select_row``), applied to the true mass
    coverage = sum_i |T_i| sum_{j in G_i} M[i, j] / sum_i |T_i|
             = (1 / S) * sum_r sum_{c in selected blocks of r} P[r, c]

Readings (listed with the others in the design notes): the block mass of a
q-block is the mean over its valid queries (each query row of the attention
map weighs the same, and every row of M is a distribution); coverage weighs
every valid query equally; the top-p cut is taken on M's row as is (it
already sums to 1).
"""

from __future__ import annotations

import numpy as np

from . import mask as om

BLOCK = 64


def attention_probs(qh, kh, sm_scale: float) -> np.ndarray:
    """Dense attention probabilities P [S, S] of one (request, head)."""
    qh = np.asarray(qh, dtype=np.float64)
    kh = np.asarray(kh, dtype=np.float64)
    z = sm_scale * (qh @ kh.T)
    z = z - z.max(axis=1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=1, keepdims=True)


def block_mass(qh, kh, sm_scale: float, block: int = BLOCK, kv_block: int | None = None) -> np.ndarray:
    """M [n, n_kv]: mean over the valid queries of q-block i (``block``
    tokens) of their attention mass on the keys of kv block j (``kv_block``
    tokens, default ``block``)."""
    kvb = block if kv_block is None else kv_block
    P = attention_probs(qh, kh, sm_scale)
    S = P.shape[0]
    n = (S + block - 1) // block
    nk = (S + kvb - 1) // kvb
    M = np.empty((n, nk), dtype=np.float64)
    for i in range(n):
        rows = P[i * block:min(i * block + block, S)]
        for j in range(nk):
            M[i, j] = rows[:, j * kvb:min(j * kvb + kvb, S)].sum() / rows.shape[0]
    return M


def block_mass_all(q, k, sm_scale: float, block: int = BLOCK, kv_block: int | None = None) -> np.ndarray:
    """M for every request and head of ``q, k [B, S, H, D]`` -> [B, H, n, n_kv]."""
    kvb = block if kv_block is None else kv_block
    B, S, H, _ = q.shape
    n = (S + block - 1) // block
    nk = (S + kvb - 1) // kvb
    out = np.empty((B, H, n, nk), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            out[b, h] = block_mass(q[b, :, h], k[b, :, h], sm_scale, block, kvb)
    return out


def select_row_from_mass(m_row, top_p: float, min_top_k: float) -> np.ndarray:
    """One mask row from block masses: order (mass desc, index asc), the
    smallest prefix whose share of the row's mass reaches top_p, the top-k
    floor, at least one block; ids ascending.  A row of zero total mass has
    zero shares, so a top_p > 0 is never reached and every block is kept."""
    m_row = np.asarray(m_row, dtype=np.float64)
    n = m_row.shape[0]
    order = np.lexsort((np.arange(n), -m_row))
    total = m_row.sum()
    share = m_row[order] / total if total > 0 else np.zeros(n)
    kp = om.top_p_count(share, top_p)
    k = min(n, max(kp, om.floor_count(min_top_k, n), 1))
    return np.sort(order[:k])


def mask_from_mass(M, top_p: float, min_top_k: float):
    """CSR mask (mask_batch = B) from block masses ``M [B, H, n, n_kv]``."""
    B, H, n, _ = M.shape
    rows = [select_row_from_mass(M[b, h, i], top_p, min_top_k)
            for b in range(B) for h in range(H) for i in range(n)]
    counts = np.array([len(r) for r in rows], dtype=np.int64)
    row_ptr = np.zeros(B * H * n + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    col_idx = np.concatenate(rows).astype(np.int64)
    return row_ptr, col_idx


def valid_counts(S: int, block: int = BLOCK) -> np.ndarray:
    """|T_i|: valid tokens of every block."""
    n = (S + block - 1) // block
    return np.array([min(block, S - i * block) for i in range(n)], dtype=np.float64)


def coverage(row_ptr, col_idx, mask_batch: int, M, S: int, block: int = BLOCK) -> np.ndarray:
    """Coverage [B, H] of a CSR mask on the requests whose block masses are
    ``M [B, H, n, n_kv]`` (row m = ((b if mask_batch > 1 else 0) * H + h) * n + i;
    ``block`` is the q-block size, the weights |T_i| are its valid tokens)."""
    B, H, n, _ = M.shape
    w = valid_counts(S, block)
    out = np.empty((B, H), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            kept = 0.0
            for i in range(n):
                r = ((b if mask_batch > 1 else 0) * H + h) * n + i
                kept += w[i] * M[b, h, i, col_idx[row_ptr[r]:row_ptr[r + 1]]].sum()
            out[b, h] = kept / w.sum()
    return out
