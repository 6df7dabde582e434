"""Oracle: block-masked softmax attention (float64, plain NumPy).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Definition followed (Chorus II, Sec. 3.2 "Efficient block-sparse kernel" and
Sec. 3.2 Obs. 2 for attention = softmax(Q K^T)): the token sequence is cut into
blocks of ``block`` tokens; a query in q-block ``i`` may attend only to keys in
the kv-blocks listed for its mask row, and pruned pairs contribute exactly
nothing to QK^T, the softmax or PV.  Written out for one query row ``r`` of
batch ``b``, head ``h`` (mask row ``m``):

    A(r)   = { c < S : floor(c / block) in M[m] }
    z_c    = sm_scale * <Q[b,r,h,:], K[b,c,h,:]>    for c in A(r), -inf otherwise
    O[r]   = sum_c softmax(z)_c * V[b,c,h,:]
    lse[r] = ln sum_{c in A(r)} exp(z_c)

A row with A(r) empty has O = 0 and lse = -inf (reading: a mask given from
outside may contain empty rows; the builder never emits one).

Layout: Q, K, V are ``[B, S, H, D]`` (token-major, heads interleaved, head dim
contiguous) -- the layout the paper indexes as ``K[:, 0:N0, :, :]`` in Eq. (1).
The mask is CSR over rows ``m = (b_m * H + h) * n_blocks + i`` with ascending
kv-block ids; ``mask_batch`` is B (one mask per request) or 1 (one mask reused
for every request -- the cross-request reuse of Sec. 3.2).

Two evaluation forms are provided and tested equal:
* ``literal`` -- all S logits of a q-block, disallowed ones set to -inf;
* ``gather``  -- only the allowed keys are gathered, then the same softmax.
"""

from __future__ import annotations

import math

import numpy as np

BLOCK = 64


def n_blocks(S: int, block: int = BLOCK) -> int:
    return (S + block - 1) // block


def allowed_keys(kv_blocks, S: int, block: int = BLOCK) -> np.ndarray:
    """Token indices c < S whose block is listed in ``kv_blocks``."""
    parts = [np.arange(j * block, min(j * block + block, S)) for j in kv_blocks]
    if not parts:
        return np.zeros(0, dtype=np.int64)
    return np.concatenate(parts).astype(np.int64)


def _softmax_rows(z: np.ndarray, v: np.ndarray):
    """Row softmax of logits z [n, m] (some -inf) applied to v [m, D]."""
    n = z.shape[0]
    D = v.shape[1]
    out = np.zeros((n, D), dtype=np.float64)
    lse = np.full(n, -np.inf, dtype=np.float64)
    if z.shape[1] == 0:
        return out, lse
    mx = z.max(axis=1)
    live = np.isfinite(mx)
    if not live.any():
        return out, lse
    e = np.exp(z[live] - mx[live, None])
    l = e.sum(axis=1)
    out[live] = (e @ v) / l[:, None]
    lse[live] = mx[live] + np.log(l)
    return out, lse


def attention_block(qh, kh, vh, kv_blocks, i: int, sm_scale: float,
                    block: int = BLOCK, form: str = "gather", kv_block: int | None = None):
    """Output rows of q-block ``i`` for one (batch, head).

    qh, kh, vh: ``[S, D]`` arrays holding the exact values the kernel reads.
    kv_blocks: the kv-block ids listed for this mask row (any order), in
    units of ``kv_block`` tokens (default ``block``; q-blocks are ``block``).
    Returns ``(O_i [rows, D], lse_i [rows])`` in float64, rows = valid queries.
    """
    kvb = block if kv_block is None else kv_block
    qh = np.asarray(qh, dtype=np.float64)
    kh = np.asarray(kh, dtype=np.float64)
    vh = np.asarray(vh, dtype=np.float64)
    S = qh.shape[0]
    rows = slice(i * block, min(i * block + block, S))
    qi = qh[rows]
    if form == "literal":
        z = sm_scale * (qi @ kh.T)
        allowed = np.zeros(S, dtype=bool)
        allowed[allowed_keys(kv_blocks, S, kvb)] = True
        z[:, ~allowed] = -np.inf
        return _softmax_rows(z, vh)
    if form == "gather":
        idx = allowed_keys(sorted(set(int(j) for j in kv_blocks)), S, kvb)
        z = sm_scale * (qi @ kh[idx].T)
        return _softmax_rows(z, vh[idx])
    raise ValueError(f"unknown form {form!r}")


def attention_weights_block(qh, kh, kv_blocks, i: int, sm_scale: float, block: int = BLOCK):
    """Explicit attention weights [rows, S] of q-block ``i`` (literal form).

    Used to check the invariants: rows sum to one, zero weight off the mask.
    """
    qh = np.asarray(qh, dtype=np.float64)
    kh = np.asarray(kh, dtype=np.float64)
    S = qh.shape[0]
    rows = slice(i * block, min(i * block + block, S))
    z = sm_scale * (qh[rows] @ kh.T)
    allowed = np.zeros(S, dtype=bool)
    allowed[allowed_keys(kv_blocks, S, block)] = True
    z[:, ~allowed] = -np.inf
    w = np.zeros_like(z)
    mx = z.max(axis=1)
    live = np.isfinite(mx)
    e = np.exp(z[live] - mx[live, None])
    w[live] = e / e.sum(axis=1, keepdims=True)
    return w


def mask_row_index(b: int, h: int, i: int, H: int, nb: int, mask_batch: int) -> int:
    bm = b if mask_batch > 1 else 0
    return (bm * H + h) * nb + i


def row_blocks(row_ptr, col_idx, r: int) -> np.ndarray:
    return np.asarray(col_idx[int(row_ptr[r]):int(row_ptr[r + 1])])


def attention(q, k, v, row_ptr, col_idx, sm_scale: float, mask_batch: int = 1,
              block: int = BLOCK, form: str = "gather", kv_block: int | None = None):
    """Full block-masked attention for ``[B, S, H, D]`` inputs.

    Mask rows are q-blocks of ``block`` tokens, its ids kv blocks of
    ``kv_block`` tokens (default ``block``).
    Returns ``O [B, S, H, D]`` and ``lse [B, H, S]`` (float64).
    """
    B, S, H, D = q.shape
    nb = n_blocks(S, block)
    if mask_batch not in (1, B):
        raise ValueError("mask_batch must be 1 or B")
    O = np.zeros((B, S, H, D), dtype=np.float64)
    lse = np.full((B, H, S), -np.inf, dtype=np.float64)
    for b in range(B):
        for h in range(H):
            qh = np.asarray(q[b, :, h, :], dtype=np.float64)
            kh = np.asarray(k[b, :, h, :], dtype=np.float64)
            vh = np.asarray(v[b, :, h, :], dtype=np.float64)
            for i in range(nb):
                r = mask_row_index(b, h, i, H, nb, mask_batch)
                o_i, l_i = attention_block(qh, kh, vh, row_blocks(row_ptr, col_idx, r), i,
                                           sm_scale, block, form, kv_block)
                rows = slice(i * block, i * block + o_i.shape[0])
                O[b, rows, h, :] = o_i
                lse[b, h, rows] = l_i
    return O, lse


def default_sm_scale(D: int) -> float:
    return 1.0 / math.sqrt(D)
