"""Pins of the true block-mass oracle (oracle/mass.py): brute force, closed
forms, a hand-derived example, the identity with the pooled-score selection,
and coverage invariants.  CPU only."""

import json
import math
import os

import numpy as np
import pytest

from oracle import mask as om
from oracle import mass as ms

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "block_mass_example.json")


@pytest.fixture
def rng():
    return np.random.default_rng(2606)


def brute_mass(q, k, sm, block):
    """Pure-Python loops: token probabilities, then block sums / valid rows."""
    S = len(q)
    n = (S + block - 1) // block
    P = []
    for r in range(S):
        z = [sm * sum(q[r][d] * k[c][d] for d in range(len(q[r]))) for c in range(S)]
        mx = max(z)
        e = [math.exp(x - mx) for x in z]
        tot = sum(e)
        P.append([x / tot for x in e])
    M = [[0.0] * n for _ in range(n)]
    for i in range(n):
        rows = range(i * block, min(i * block + block, S))
        for j in range(n):
            s = 0.0
            for r in rows:
                for c in range(j * block, min(j * block + block, S)):
                    s += P[r][c]
            M[i][j] = s / len(rows)
    return np.array(M), np.array(P)


@pytest.mark.parametrize("S,block,D", [(1, 4, 3), (7, 4, 2), (16, 4, 5), (37, 8, 4), (50, 16, 6)])
def test_block_mass_matches_brute_force(rng, S, block, D):
    q = rng.standard_normal((S, D))
    k = rng.standard_normal((S, D))
    M = ms.block_mass(q, k, 0.7, block)
    ref, _ = brute_mass(q.tolist(), k.tolist(), 0.7, block)
    np.testing.assert_allclose(M, ref, rtol=1e-12, atol=1e-15)


def test_rows_are_distributions(rng):
    q = rng.standard_normal((300, 16)) * 2
    k = rng.standard_normal((300, 16)) * 2
    M = ms.block_mass(q, k, 0.3, 64)
    np.testing.assert_allclose(M.sum(axis=1), 1.0, rtol=0, atol=1e-12)
    assert (M > 0).all()


def test_uniform_attention_closed_form():
    """q = 0: every query attends uniformly, so M[i, j] = |T_j| / S."""
    S, block = 150, 64
    q = np.zeros((S, 8))
    k = np.random.default_rng(1).standard_normal((S, 8))
    M = ms.block_mass(q, k, 1.0, block)
    w = ms.valid_counts(S, block)
    np.testing.assert_allclose(M, np.tile(w / S, (len(w), 1)), rtol=1e-14)


def test_hand_derived_example():
    g = json.load(open(GOLDEN))
    q = np.array(g["q"])[:, None]
    k = (np.array(g["k_ln3_multiples"]) * math.log(3.0))[:, None]
    M = ms.block_mass(q, k, 1.0, g["block"])
    np.testing.assert_allclose(M, np.array(g["mass"]), rtol=1e-14)
    rows = [ms.select_row_from_mass(M[i], g["top_p"], g["min_top_k"]).tolist() for i in range(2)]
    assert rows == g["mask_rows"]
    for key, cov_key in (("mask_rows", "coverage_of_mask_rows"),
                         ("diagonal_mask_rows", "coverage_of_diagonal_mask_rows")):
        rr = g[key]
        rp = np.array([0, len(rr[0]), len(rr[0]) + len(rr[1])])
        ci = np.array(rr[0] + rr[1])
        cov = ms.coverage(rp, ci, 1, M[None, None], 4, g["block"])
        assert abs(cov[0, 0] - g[cov_key]) < 1e-14


def test_selection_from_mass_equals_score_selection_of_log_mass(rng):
    """softmax(log m) = m / sum(m): selecting on masses is the pooled-score
    rule applied to log-masses."""
    for _ in range(200):
        n = int(rng.integers(1, 60))
        m = rng.random(n) ** 3 + 1e-9
        if rng.random() < 0.3:
            m[rng.integers(0, n, size=n // 3)] = m[0]          # exact ties
        top_p = float(rng.choice([0.0, 0.3, 0.9, 1.0, rng.random()]))
        mk = float(rng.choice([0.0, 0.1, 0.5, rng.random()]))
        a = ms.select_row_from_mass(m, top_p, mk)
        b = om.select_row(np.log(m), top_p, mk)
        if not np.array_equal(a, b):
            # only a rounding-level top-p boundary may differ
            order = np.lexsort((np.arange(n), -m))
            c = np.cumsum(m[order] / m.sum())
            assert abs(len(a) - len(b)) == 1
            assert np.min(np.abs(c - top_p)) < 1e-12


def test_selection_from_mass_brute_force(rng):
    for _ in range(200):
        n = int(rng.integers(1, 40))
        m = np.round(rng.random(n) * 8) / 8 + 1e-3             # many ties
        top_p = float(rng.choice([0.25, 0.5, 0.75, rng.random()]))
        mk = float(rng.choice([0.0, 0.2, rng.random()]))
        order = sorted(range(n), key=lambda j: (-m[j], j))
        tot = sum(m)
        run, kp = 0.0, n
        for pos, j in enumerate(order):
            run += m[j] / tot
            if run >= top_p:
                kp = pos + 1
                break
        k = min(n, max(kp, math.ceil(mk * n - 1e-9), 1))
        want = sorted(order[:k])
        got = ms.select_row_from_mass(m, top_p, mk).tolist()
        if got != want:
            # summation-order rounding at the exact boundary only
            assert abs(len(got) - len(want)) == 1
        else:
            assert got == want


def test_coverage_invariants_and_brute_force(rng):
    S, block, H = 130, 16, 2
    q = rng.standard_normal((1, S, H, 8))
    k = rng.standard_normal((1, S, H, 8))
    M = ms.block_mass_all(q, k, 0.5, block)
    n = M.shape[-1]
    # full mask covers everything
    rp = np.arange(0, H * n * n + 1, n)
    ci = np.tile(np.arange(n), H * n)
    np.testing.assert_allclose(ms.coverage(rp, ci, 1, M, S, block), 1.0, atol=1e-12)
    # a mask selected from M itself covers at least top_p of every head
    rp, ci = ms.mask_from_mass(M, 0.7, 0.0)
    cov = ms.coverage(rp, ci, 1, M, S, block)
    assert (cov >= 0.7 - 1e-12).all()
    # brute force: mean over queries of the token mass inside the kept blocks
    for h in range(H):
        _, P = brute_mass(q[0, :, h].tolist(), k[0, :, h].tolist(), 0.5, block)
        tot = 0.0
        for r in range(S):
            i = r // block
            row = h * n + i
            for j in ci[rp[row]:rp[row + 1]]:
                tot += P[r, j * block:min(j * block + block, S)].sum()
        assert abs(tot / S - cov[0, h]) < 1e-12
