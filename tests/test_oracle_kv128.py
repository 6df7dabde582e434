"""Pins for the oracle's kv blocks of 128 tokens with q-blocks of 64 (the
paper's own kernel geometry, Sec. 4.1): scalar brute force with separate q
and kv block sizes, and the identities that tie a kv-128 mask to the kv-64
mask listing both halves of each of its blocks (attention, pooled scores,
block mass, coverage).  CPU only."""

import math

import numpy as np
import pytest

from oracle import attention as oa
from oracle import mask as om
from oracle import mass as ms
from workloads import random_csr


def expand(rp, ci, n64):
    """kv-128 CSR -> kv-64 CSR listing blocks 2J and 2J + 1 (< n64) for each J."""
    rows = []
    for r in range(len(rp) - 1):
        sub = [x for J in ci[rp[r]:rp[r + 1]] for x in (2 * J, 2 * J + 1) if x < n64]
        rows.append(sub)
    counts = [len(x) for x in rows]
    out_rp = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    out_ci = np.array([x for r in rows for x in r], dtype=np.int64)
    return out_rp, out_ci


def brute(q, k, v, rp, ci, sm, qb, kvb):
    B, S, H, D = q.shape
    nq = (S + qb - 1) // qb
    O = np.zeros((B, S, H, D))
    for b in range(B):
        for h in range(H):
            for r in range(S):
                m = h * nq + r // qb
                allowed = set(int(x) for x in ci[rp[m]:rp[m + 1]])
                keys = [c for c in range(S) if c // kvb in allowed]
                if not keys:
                    continue
                z = [sm * sum(float(q[b, r, h, d]) * float(k[b, c, h, d]) for d in range(D)) for c in keys]
                mx = max(z)
                w = [math.exp(x - mx) for x in z]
                tot = sum(w)
                for d in range(D):
                    O[b, r, h, d] = sum(wi * float(v[b, c, h, d]) for wi, c in zip(w, keys)) / tot
    return O


def test_brute_force_separate_block_sizes():
    rng = np.random.default_rng(1)
    B, S, H, D, qb, kvb = 1, 23, 2, 3, 4, 8
    q, k, v = (rng.standard_normal((B, S, H, D)) for _ in range(3))
    nq, nk = (S + qb - 1) // qb, (S + kvb - 1) // kvb
    rp, ci = random_csr(rng, H * nq, nk, 0.5, empty_frac=0.1)
    O, _ = oa.attention(q, k, v, rp, ci, 0.4, 1, block=qb, kv_block=kvb)
    np.testing.assert_allclose(O, brute(q, k, v, rp, ci, 0.4, qb, kvb), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("S", [128, 200, 257])
def test_attention_equals_expanded_kv64_mask(S):
    rng = np.random.default_rng(S)
    B, H, D = 1, 2, 8
    q, k, v = (rng.standard_normal((B, S, H, D)) for _ in range(3))
    n64, n128 = (S + 63) // 64, (S + 127) // 128
    rp, ci = random_csr(rng, H * n64, n128, 0.6)
    O1, L1 = oa.attention(q, k, v, rp, ci, 0.3, 1, kv_block=128)
    erp, eci = expand(rp, ci, n64)
    O2, L2 = oa.attention(q, k, v, erp, eci, 0.3, 1)
    np.testing.assert_allclose(O1, O2, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(L1, L2, rtol=1e-13, atol=1e-14)


def test_pooled_kv128_scores_are_count_weighted_halves():
    rng = np.random.default_rng(2)
    S, D = 300, 16                           # kv-128 blocks of 128, 128, 44 tokens
    qh, kh = rng.standard_normal((S, D)), rng.standard_normal((S, D))
    qbar = om.pool_means(qh, 64)
    s64 = om.block_scores(qbar, om.pool_means(kh, 64), 0.5)
    s128 = om.block_scores(qbar, om.pool_means(kh, 128), 0.5)
    cnt64 = np.array([min(64, S - 64 * j) for j in range(5)], float)
    for J in range(3):
        lo, hi = 2 * J, min(2 * J + 2, 5)
        ref = (s64[:, lo:hi] * cnt64[lo:hi]).sum(axis=1) / cnt64[lo:hi].sum()
        np.testing.assert_allclose(s128[:, J], ref, rtol=1e-12, atol=1e-14)


def test_builder_kv128_shape_and_floor():
    rng = np.random.default_rng(3)
    B, S, H, D = 1, 700, 2, 8
    q, k = rng.standard_normal((B, S, H, D)), rng.standard_normal((B, S, H, D))
    m = om.build_block_mask(q, k, 0.3, 0.0, 0.5, kv_block=128)
    nq, nk = 11, 6
    assert m.n_blocks == nq and m.columns == nk and m.scores.shape == (B * H * nq, nk)
    counts = np.diff(m.row_ptr)
    assert np.all(counts == math.ceil(0.5 * nk - 1e-9))      # top_p = 0: the floor alone
    assert m.col_idx.max() < nk


def test_block_mass_kv128_columns_sum_halves_and_coverage_agrees():
    rng = np.random.default_rng(4)
    S, D = 330, 8
    qh, kh = rng.standard_normal((S, D)), rng.standard_normal((S, D))
    M64 = ms.block_mass(qh, kh, 0.4)
    M128 = ms.block_mass(qh, kh, 0.4, kv_block=128)
    n64 = M64.shape[1]
    for J in range(M128.shape[1]):
        np.testing.assert_allclose(M128[:, J], M64[:, 2 * J:min(2 * J + 2, n64)].sum(axis=1), rtol=1e-12)
    np.testing.assert_allclose(M128.sum(axis=1), 1.0, rtol=1e-12)
    rp, ci = random_csr(rng, M128.shape[0], M128.shape[1], 0.5)
    erp, eci = expand(rp, ci, n64)
    c128 = ms.coverage(rp, ci, 1, M128[None, None], S)
    c64 = ms.coverage(erp, eci, 1, M64[None, None], S)
    np.testing.assert_allclose(c128, c64, rtol=1e-12)
