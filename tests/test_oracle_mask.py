"""Pins for the mask-builder oracle (CPU only).

Checked against: hand-derived worked examples (tests/golden), a pure-Python
brute force of every step, a library sort (numpy lexsort) in the pure top-k
case, the selection invariants, and closed-form pooling cases.
"""

import json
import math
import os

import numpy as np
import pytest

from oracle import mask as om

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mask_worked_examples.json")


def brute_select(scores, top_p, min_top_k):
    """Pure Python: sorted() by (-s, j), explicit cumulative loop."""
    n = len(scores)
    mx = max(scores)
    e = [math.exp(s - mx) for s in scores]
    tot = sum(e)
    order = sorted(range(n), key=lambda j: (-scores[j], j))
    if top_p <= 0:
        kp = 0
    elif top_p >= 1:
        kp = n
    else:
        kp = n
        acc = 0.0
        for pos, j in enumerate(order):
            acc += e[j] / tot
            if acc >= top_p:
                kp = pos + 1
                break
    kmin = math.ceil(min_top_k * n - 1e-9)
    k = min(n, max(kp, kmin, 1))
    return sorted(order[:k])


def test_golden_row_examples():
    g = json.load(open(GOLDEN))
    for ex in g["row_examples"]:
        s = np.log(np.array(ex["scores_ln"], dtype=np.float64))
        for case in ex["cases"]:
            got = om.select_row(s, case["top_p"], case["min_top_k"]).tolist()
            assert got == case["keep"], (ex, case)


def _builder_example_tokens():
    S, D = 160, 2
    ln2, ln4, ln8 = math.log(2), math.log(4), math.log(8)
    q = np.zeros((1, S, 1, D))
    k = np.zeros((1, S, 1, D))
    q[0, 0:64, 0] = (1, 0)
    q[0, 64:128:2, 0] = (0, 2)
    q[0, 128:160, 0] = (1, 1)
    k[0, 0:64:2, 0] = (2 * ln4, 0)
    k[0, 64:128, 0] = (ln2, ln8)
    k[0, 128:160:2, 0] = (0, 2 * ln2)
    return q, k


def test_golden_builder_example():
    g = json.load(open(GOLDEN))["builder_example"]
    q, k = _builder_example_tokens()
    qbar = om.pool_means(q[0, :, 0])
    kbar = om.pool_means(k[0, :, 0])
    np.testing.assert_allclose(qbar, [[1, 0], [0, 1], [1, 1]], rtol=0, atol=1e-15)
    np.testing.assert_allclose(kbar, [[math.log(4), 0], [math.log(2), math.log(8)],
                                      [0, math.log(2)]], rtol=1e-14, atol=1e-15)
    s = om.block_scores(qbar, kbar, 1.0)
    np.testing.assert_allclose(np.exp(s), g["scores_exp"], rtol=1e-14)
    for case in g["cases"]:
        m = om.build_block_mask(q, k, 1.0, case["top_p"], case["min_top_k"])
        rows = [m.row(r).tolist() for r in range(3)]
        assert rows == case["rows"], case


def test_matches_pure_python_brute_force(rng):
    for trial in range(400):
        n = int(rng.integers(1, 40))
        if trial % 3 == 0:
            s = rng.integers(-3, 4, size=n).astype(np.float64)      # many exact ties
        else:
            s = rng.standard_normal(n) * rng.uniform(0.1, 6)
        top_p = float(rng.choice([0.0, 1.0, rng.uniform(0, 1)]))
        min_top_k = float(rng.choice([0.0, 1.0, rng.uniform(0, 0.6)]))
        got = om.select_row(s, top_p, min_top_k).tolist()
        want = brute_select(s.tolist(), top_p, min_top_k)
        if got != want:
            # only a cumulative sum within rounding of top_p may differ
            e = np.exp(s - s.max())
            c = np.cumsum((e / e.sum())[np.lexsort((np.arange(n), -s))])
            assert np.min(np.abs(c - top_p)) < 1e-12, (s, top_p, min_top_k)


def test_full_mass_or_full_floor_keeps_everything(rng):
    s = rng.standard_normal(37)
    assert om.select_row(s, 1.0, 0.0).tolist() == list(range(37))
    assert om.select_row(s, 0.0, 1.0).tolist() == list(range(37))
    assert om.select_row(s, 0.3, 1.0).tolist() == list(range(37))


def test_pure_top_k_equals_library_sort(rng):
    for n in (5, 64, 427, 512):
        s = rng.standard_normal(n)
        s[::7] = s[0]                          # add exact ties
        for kk in (1, 3, n // 4, n):
            got = om.select_row(s, 0.0, kk / n)
            want = np.sort(np.lexsort((np.arange(n), -s))[:kk])
            np.testing.assert_array_equal(got, want)


def test_duplicate_pooled_keys_take_lowest_index():
    s = np.array([0.5, 2.0, 2.0, 1.0, 2.0])
    assert om.select_row(s, 0.0, 0.2).tolist() == [1]
    assert om.select_row(s, 0.0, 0.4).tolist() == [1, 2]
    assert om.select_row(s, 0.0, 0.6).tolist() == [1, 2, 4]


def test_selected_mass_invariants(rng):
    for _ in range(300):
        n = int(rng.integers(2, 200))
        s = rng.standard_normal(n) * rng.uniform(0.2, 5)
        top_p = float(rng.uniform(0.05, 0.99))
        kmin_frac = float(rng.uniform(0, 0.3))
        sel = om.select_row(s, top_p, kmin_frac)
        p = np.exp(s - s.max())
        p /= p.sum()
        assert p[sel].sum() >= top_p - 1e-12
        k = len(sel)
        kmin = math.ceil(kmin_frac * n - 1e-9)
        order = np.lexsort((np.arange(n), -s))
        assert sorted(order[:k].tolist()) == sel.tolist()
        if k > max(kmin, 1):
            # the last kept block was needed to reach top_p
            assert p[order[:k - 1]].sum() < top_p + 1e-12


def test_pool_constant_block_and_partial_block():
    S, D = 150, 3
    x = np.zeros((S, D))
    x[0:64] = [1.5, -2.0, 0.25]
    x[64:128] = np.arange(64)[:, None] * np.array([1.0, 0.0, -1.0])
    x[128:150] = 7.0                              # 22 valid tokens in the last block
    p = om.pool_means(x)
    np.testing.assert_array_equal(p[0], [1.5, -2.0, 0.25])
    np.testing.assert_allclose(p[1], [31.5, 0.0, -31.5], rtol=0, atol=1e-15)
    np.testing.assert_array_equal(p[2], [7.0, 7.0, 7.0])


def _brute_builder(q, k, sm_scale, top_p, min_top_k, block):
    B, S, H, D = q.shape
    n = (S + block - 1) // block
    rows = []
    for b in range(B):
        for h in range(H):
            def pooled(x, i):
                toks = range(i * block, min(S, i * block + block))
                return [sum(float(x[b, t, h, d]) for t in toks) / len(toks) for d in range(D)]
            qb = [pooled(q, i) for i in range(n)]
            kb = [pooled(k, j) for j in range(n)]
            for i in range(n):
                s = [sm_scale * sum(qb[i][d] * kb[j][d] for d in range(D)) for j in range(n)]
                rows.append(brute_select(s, top_p, min_top_k))
    return rows


@pytest.mark.parametrize("S,block", [(100, 16), (64, 16), (70, 32)])
def test_builder_matches_brute_force(rng, S, block):
    B, H, D = 2, 2, 6
    q = rng.standard_normal((B, S, H, D))
    k = q + 0.3 * rng.standard_normal((B, S, H, D))
    for top_p, mk in [(0.5, 0.0), (0.8, 0.2), (0.0, 0.3)]:
        m = om.build_block_mask(q, k, 0.9, top_p, mk, block)
        want = _brute_builder(q, k, 0.9, top_p, mk, block)
        got = [m.row(r).tolist() for r in range(len(want))]
        assert got == want
