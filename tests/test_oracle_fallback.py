"""Pins of the visit-refresh oracle (oracle/fallback.py): brute force over
pairs, the group invariant, and hand cases.  CPU only."""

import numpy as np
import pytest

from oracle import fallback as fb


@pytest.fixture
def rng():
    return np.random.default_rng(7)


def test_csr_round_trip(rng):
    D = rng.random((13, 9)) < 0.3
    rp, ci = fb.csr_of(D)
    assert np.array_equal(fb.dense_of(rp, ci, 13, 9), D)
    for r in range(13):
        row = ci[rp[r]:rp[r + 1]]
        assert np.all(np.diff(row) > 0)


def test_hand_case():
    # 1 row, 4 blocks; layers keep {0}, {1}, then the last layer {0}
    m = [np.array([[1, 0, 0, 0]], bool), np.array([[0, 1, 0, 0]], bool), np.array([[1, 0, 0, 0]], bool)]
    used, V = fb.run_group(m, 4)
    assert used[0].tolist() == m[0].tolist() and used[1].tolist() == m[1].tolist()
    # blocks 2 and 3 were never visited: forced into the last layer
    assert used[2].tolist() == [[True, False, True, True]]
    assert V.all()


def test_group_invariant_and_brute_force(rng):
    for _ in range(50):
        rows, n, N = int(rng.integers(1, 12)), int(rng.integers(1, 20)), int(rng.integers(1, 9))
        masks = [rng.random((rows, n)) < rng.uniform(0.0, 0.5) for _ in range(N)]
        used, V = fb.run_group(masks, n)
        # every pair is touched at least once per group
        assert V.all()
        # the last layer keeps its own pairs and adds exactly the unvisited ones
        before = np.zeros((rows, n), bool)
        for M in masks[:-1]:
            before |= M
        for r in range(rows):
            for j in range(n):
                want = masks[-1][r, j] or not before[r, j]
                assert used[-1][r, j] == want
        for a, b in zip(used[:-1], masks[:-1]):
            assert np.array_equal(a, b)


def test_single_layer_group_is_dense(rng):
    M = rng.random((5, 7)) < 0.2
    used, _ = fb.run_group([M], 7)
    assert used[0].all()
