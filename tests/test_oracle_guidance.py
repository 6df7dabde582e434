"""Pins for the first-frame key enhancement oracle (oracle/guidance.py),
Sec. 3.4 Eq. (1).  CPU only: a hand case in closed form, scalar brute force
with the logits of first-frame keys multiplied by beta, the all-frames case
(the same as a larger softmax scale), identities, and the effect on the
pooled-score predictor and the block mass."""

import math

import numpy as np
import pytest

from oracle import attention as oa
from oracle import guidance as og
from oracle import mask as om
from oracle import mass as ms
from workloads import random_csr


def test_first_frame_tokens():
    assert og.first_frame_tokens((21, 45, 80)) == 3600
    assert og.first_frame_tokens((31, 22, 40)) == 880


def test_identities():
    rng = np.random.default_rng(0)
    k = rng.standard_normal((2, 70, 3, 8))
    assert np.array_equal(og.enhance_first_frame_keys(k, 0, 3.0), k)
    assert np.array_equal(og.enhance_first_frame_keys(k, 70, 1.0), k)
    e = og.enhance_first_frame_keys(k, 33, 2.5)
    assert np.array_equal(e[:, 33:], k[:, 33:])
    assert np.allclose(e[:, :33], 2.5 * k[:, :33], rtol=0, atol=0)
    with pytest.raises(ValueError):
        og.enhance_first_frame_keys(k, 71, 2.0)


def test_hand_case_closed_form():
    # one query, two keys: key 0 in the first frame, key 1 after it
    q = np.zeros((1, 2, 1, 2)); q[0, 0, 0] = [1.0, 0.0]
    k = np.zeros((1, 2, 1, 2)); k[0, 0, 0] = [0.5, 0.0]; k[0, 1, 0] = [0.25, 0.0]
    v = np.zeros((1, 2, 1, 2)); v[0, 0, 0] = [1.0, 0.0]; v[0, 1, 0] = [0.0, 1.0]
    beta, sm = 3.0, 1.0
    ke = og.enhance_first_frame_keys(k, 1, beta)
    O, L = oa.attention(q, ke, v, np.array([0, 1]), np.array([0]), sm, 1, block=2)
    # weights exp(beta * 0.5) and exp(0.25)
    w0, w1 = math.exp(1.5), math.exp(0.25)
    assert O[0, 0, 0, 0] == pytest.approx(w0 / (w0 + w1), rel=1e-15)
    assert O[0, 0, 0, 1] == pytest.approx(w1 / (w0 + w1), rel=1e-15)
    assert L[0, 0, 0] == pytest.approx(math.log(w0 + w1), rel=1e-15)


def brute_force_scaled_logits(q, k, v, row_ptr, col_idx, sm, n_first, beta, block):
    """Scalar loops: the logit of key c is multiplied by beta when c < n_first."""
    B, S, H, D = q.shape
    nb = (S + block - 1) // block
    O = np.zeros((B, S, H, D))
    for b in range(B):
        for h in range(H):
            for r in range(S):
                m = (h * nb) + r // block
                blocks = set(int(x) for x in col_idx[row_ptr[m]:row_ptr[m + 1]])
                keys = [c for c in range(S) if c // block in blocks]
                z = []
                for c in keys:
                    dot = sum(float(q[b, r, h, d]) * float(k[b, c, h, d]) for d in range(D))
                    z.append(sm * dot * (beta if c < n_first else 1.0))
                if not z:
                    continue
                mx = max(z)
                w = [math.exp(x - mx) for x in z]
                tot = sum(w)
                for d in range(D):
                    O[b, r, h, d] = sum(wi * float(v[b, c, h, d]) for wi, c in zip(w, keys)) / tot
    return O


@pytest.mark.parametrize("n_first,beta", [(5, 1.7), (8, 0.6), (13, 2.0), (19, 1.25)])
def test_brute_force(n_first, beta):
    rng = np.random.default_rng(n_first)
    B, S, H, D, blk = 1, 19, 2, 4, 4
    q = rng.standard_normal((B, S, H, D))
    k = rng.standard_normal((B, S, H, D))
    v = rng.standard_normal((B, S, H, D))
    nb = (S + blk - 1) // blk
    rp, ci = random_csr(rng, H * nb, nb, 0.6)
    O, _ = oa.attention(q, og.enhance_first_frame_keys(k, n_first, beta), v, rp, ci, 0.5, 1, block=blk)
    ref = brute_force_scaled_logits(q, k, v, rp, ci, 0.5, n_first, beta, blk)
    np.testing.assert_allclose(O, ref, rtol=1e-12, atol=1e-12)


def test_all_tokens_scaled_is_a_larger_softmax_scale():
    rng = np.random.default_rng(3)
    B, S, H, D = 1, 40, 1, 8
    q, k, v = (rng.standard_normal((B, S, H, D)) for _ in range(3))
    rp, ci = np.array([0, 3, 6, 9]), np.array([0, 1, 2] * 3)
    O1, L1 = oa.attention(q, og.enhance_first_frame_keys(k, S, 1.8), v, rp, ci, 0.3, 1, block=16)
    O2, L2 = oa.attention(q, k, v, rp, ci, 0.3 * 1.8, 1, block=16)
    np.testing.assert_allclose(O1, O2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(L1, L2, rtol=1e-12, atol=1e-13)


def test_pooled_scores_follow_linearity():
    # pooled key of a block = mean of the (scaled) keys: a block wholly inside
    # the first frame has its scores multiplied by beta; a straddling block gets
    # the token-weighted mix
    rng = np.random.default_rng(5)
    S, D, blk, beta = 20, 6, 4, 1.5
    qh, kh = rng.standard_normal((S, D)), rng.standard_normal((S, D))
    n_first = 10                                    # blocks 0, 1 inside; block 2 straddles
    ke = og.enhance_first_frame_keys(kh[None, :, None, :], n_first, beta)[0, :, 0]
    s0 = om.block_scores(om.pool_means(qh, blk), om.pool_means(kh, blk), 0.7)
    s1 = om.block_scores(om.pool_means(qh, blk), om.pool_means(ke, blk), 0.7)
    np.testing.assert_allclose(s1[:, :2], beta * s0[:, :2], rtol=1e-13)
    np.testing.assert_allclose(s1[:, 3:], s0[:, 3:], rtol=0, atol=0)
    qbar = om.pool_means(qh, blk)
    k2 = (beta * kh[8:10].sum(0) + kh[10:12].sum(0)) / 4
    np.testing.assert_allclose(s1[:, 2], 0.7 * qbar @ k2, rtol=1e-13)


def test_block_mass_rows_stay_distributions_and_first_frame_gains():
    rng = np.random.default_rng(9)
    S, D = 130, 16
    base = rng.standard_normal(D)
    qh = base + 0.3 * rng.standard_normal((S, D))
    kh = base + 0.3 * rng.standard_normal((S, D))   # positive logits on average
    n_first = 64
    M0 = ms.block_mass(qh, kh, 0.25)
    ke = og.enhance_first_frame_keys(kh[None, :, None, :], n_first, 2.0)[0, :, 0]
    M1 = ms.block_mass(qh, ke, 0.25)
    np.testing.assert_allclose(M1.sum(axis=1), 1.0, rtol=1e-13)
    assert np.all(M1[:, 0] > M0[:, 0])
