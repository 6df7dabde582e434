"""Pins for the attention oracle (CPU only).

Each test checks the oracle against something other than itself: scalar
brute force, torch's dense scaled_dot_product_attention (library routine),
scipy's logsumexp, and invariants of the definition.
"""

import math

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import attention as oa
from workloads import random_csr


def _rand_qkv(rng, B, S, H, D, scale=1.0):
    q = rng.standard_normal((B, S, H, D)) * scale
    k = rng.standard_normal((B, S, H, D)) * scale
    v = rng.standard_normal((B, S, H, D))
    return q, k, v


def brute_force(q, k, v, row_ptr, col_idx, sm_scale, mask_batch, block):
    """Scalar loops over lists, no NumPy arithmetic."""
    B, S, H, D = q.shape
    nb = (S + block - 1) // block
    O = [[[[0.0] * D for _ in range(H)] for _ in range(S)] for _ in range(B)]
    L = [[[-math.inf] * S for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for h in range(H):
            for r in range(S):
                i = r // block
                m = ((b if mask_batch > 1 else 0) * H + h) * nb + i
                blocks = set(int(x) for x in col_idx[row_ptr[m]:row_ptr[m + 1]])
                keys = [c for c in range(S) if c // block in blocks]
                if not keys:
                    continue
                z = []
                for c in keys:
                    acc = 0.0
                    for d in range(D):
                        acc += float(q[b, r, h, d]) * float(k[b, c, h, d])
                    z.append(sm_scale * acc)
                mx = max(z)
                e = [math.exp(x - mx) for x in z]
                tot = sum(e)
                for d in range(D):
                    acc = 0.0
                    for w, c in zip(e, keys):
                        acc += w * float(v[b, c, h, d])
                    O[b][r][h][d] = acc / tot
                L[b][h][r] = mx + math.log(tot)
    return np.array(O), np.array(L)


@pytest.mark.parametrize("S,block,mask_batch,B", [(80, 16, 1, 1), (75, 16, 2, 2), (150, 64, 1, 2),
                                                  (64, 64, 1, 1), (33, 16, 1, 1)])
def test_matches_scalar_brute_force(rng, S, block, mask_batch, B):
    H, D = 2, 5
    q, k, v = _rand_qkv(rng, B, S, H, D)
    nb = (S + block - 1) // block
    row_ptr, col_idx = random_csr(rng, mask_batch * H * nb, nb, 0.5, empty_frac=0.2)
    sm = 0.37
    O_ref, L_ref = brute_force(q, k, v, row_ptr, col_idx, sm, mask_batch, block)
    for form in ("literal", "gather"):
        O, L = oa.attention(q, k, v, row_ptr, col_idx, sm, mask_batch, block, form)
        np.testing.assert_allclose(O, O_ref, rtol=0, atol=1e-12)
        both_inf = np.isinf(L) & np.isinf(L_ref)
        assert np.array_equal(np.isinf(L), np.isinf(L_ref))
        np.testing.assert_allclose(L[~both_inf], L_ref[~both_inf], rtol=0, atol=1e-12)


def test_full_mask_equals_dense_sdpa(rng):
    B, S, H, D, block = 2, 200, 3, 16, 64
    q, k, v = _rand_qkv(rng, B, S, H, D)
    nb = (S + block - 1) // block
    rows = H * nb
    row_ptr = np.arange(rows + 1) * nb
    col_idx = np.tile(np.arange(nb), rows)
    sm = 1.0 / math.sqrt(D)
    O, _ = oa.attention(q, k, v, row_ptr, col_idx, sm, 1, block)
    tq = torch.from_numpy(q).permute(0, 2, 1, 3)
    tk = torch.from_numpy(k).permute(0, 2, 1, 3)
    tv = torch.from_numpy(v).permute(0, 2, 1, 3)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=sm)
    np.testing.assert_allclose(O, ref.permute(0, 2, 1, 3).numpy(), rtol=0, atol=1e-12)


def test_block_mask_equals_sdpa_with_boolean_mask(rng):
    S, D, block = 130, 8, 64
    q, k, v = _rand_qkv(rng, 1, S, 1, D)
    nb = 3
    rows = [[1], [0, 2], [2]]
    row_ptr = np.cumsum([0] + [len(r) for r in rows])
    col_idx = np.concatenate(rows)
    sm = 0.5
    O, _ = oa.attention(q, k, v, row_ptr, col_idx, sm, 1, block)
    allow = np.zeros((S, S), dtype=bool)
    for r in range(S):
        for c in range(S):
            allow[r, c] = (c // block) in rows[r // block]
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q[:, :, 0][:, None]), torch.from_numpy(k[:, :, 0][:, None]),
        torch.from_numpy(v[:, :, 0][:, None]), attn_mask=torch.from_numpy(allow), scale=sm)
    np.testing.assert_allclose(O[0, :, 0], ref[0, 0].numpy(), rtol=0, atol=1e-12)
    assert nb == (S + block - 1) // block


def test_weights_rows_sum_to_one_and_zero_off_mask(rng):
    S, D, block = 300, 16, 64
    q, k, _ = _rand_qkv(rng, 1, S, 1, D, scale=2.0)
    blocks = [0, 3, 4]
    for i in range(5):
        w = oa.attention_weights_block(q[0, :, 0], k[0, :, 0], blocks, i, 0.3, block)
        np.testing.assert_allclose(w.sum(axis=1), 1.0, rtol=0, atol=1e-12)
        off = np.ones(S, dtype=bool)
        off[oa.allowed_keys(blocks, S, block)] = False
        assert np.all(w[:, off] == 0.0)
        assert np.all(w[:, ~off] > 0.0)


def test_constant_values_give_constant_output(rng):
    B, S, H, D, block = 1, 190, 2, 8, 64
    q, k, _ = _rand_qkv(rng, B, S, H, D, scale=3.0)
    v = np.ones((B, S, H, D))
    nb = 3
    row_ptr, col_idx = random_csr(rng, H * nb, nb, 0.6)
    O, _ = oa.attention(q, k, v, row_ptr, col_idx, 0.4, 1, block)
    for h in range(H):
        for i in range(nb):
            r = h * nb + i
            rows = slice(i * block, min(S, i * block + block))
            want = 1.0 if row_ptr[r + 1] > row_ptr[r] else 0.0
            np.testing.assert_allclose(O[0, rows, h], want, rtol=0, atol=1e-12)


def test_single_block_row_is_attention_on_that_slice(rng):
    S, D, block = 256, 16, 64
    q, k, v = _rand_qkv(rng, 1, S, 1, D)
    sm = 0.25
    for i, j in [(0, 3), (2, 2), (3, 0)]:
        o, lse = oa.attention_block(q[0, :, 0], k[0, :, 0], v[0, :, 0], [j], i, sm, block)
        qs = torch.from_numpy(q[0, i * 64:(i + 1) * 64, 0])[None, None]
        ks = torch.from_numpy(k[0, j * 64:(j + 1) * 64, 0])[None, None]
        vs = torch.from_numpy(v[0, j * 64:(j + 1) * 64, 0])[None, None]
        ref = torch.nn.functional.scaled_dot_product_attention(qs, ks, vs, scale=sm)[0, 0].numpy()
        np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)
        z = sm * (q[0, i * 64:(i + 1) * 64, 0] @ k[0, j * 64:(j + 1) * 64, 0].T)
        np.testing.assert_allclose(lse, logsumexp(z, axis=1), rtol=0, atol=1e-12)


def test_lse_matches_scipy_logsumexp(rng):
    S, D, block = 200, 8, 64
    q, k, v = _rand_qkv(rng, 1, S, 1, D, scale=2.0)
    blocks = [1, 3]
    idx = oa.allowed_keys(blocks, S, block)
    for i in range(4):
        _, lse = oa.attention_block(q[0, :, 0], k[0, :, 0], v[0, :, 0], blocks, i, 0.7, block)
        rows = slice(i * 64, min(S, i * 64 + 64))
        z = 0.7 * (q[0, rows, 0] @ k[0, idx, 0].T)
        np.testing.assert_allclose(lse, logsumexp(z, axis=1), rtol=0, atol=1e-12)


def test_kv_order_within_row_does_not_matter(rng):
    S, D, block = 640, 16, 64
    q, k, v = _rand_qkv(rng, 1, S, 1, D)
    blocks = [7, 1, 4, 9, 0]
    a, la = oa.attention_block(q[0, :, 0], k[0, :, 0], v[0, :, 0], blocks, 4, 0.2, block)
    b, lb = oa.attention_block(q[0, :, 0], k[0, :, 0], v[0, :, 0], sorted(blocks), 4, 0.2, block)
    c, lc = oa.attention_block(q[0, :, 0], k[0, :, 0], v[0, :, 0], sorted(blocks), 4, 0.2, block,
                               form="literal")
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    np.testing.assert_allclose(a, c, rtol=0, atol=1e-12)
    np.testing.assert_allclose(la, lc, rtol=0, atol=1e-12)


def test_empty_row_gives_zero_and_minus_inf(rng):
    S, D = 100, 4
    q, k, v = _rand_qkv(rng, 1, S, 1, D)
    o, lse = oa.attention_block(q[0, :, 0], k[0, :, 0], v[0, :, 0], [], 1, 0.5)
    assert o.shape == (36, D) and np.all(o == 0) and np.all(np.isneginf(lse))


def test_shared_mask_equals_repeated_mask(rng):
    B, S, H, D, block = 3, 130, 2, 8, 64
    q, k, v = _rand_qkv(rng, B, S, H, D)
    nb = 3
    rp, ci = random_csr(rng, H * nb, nb, 0.5)
    O1, L1 = oa.attention(q, k, v, rp, ci, 0.3, 1, block)
    counts = np.diff(rp)
    rp3 = np.concatenate([[0], np.cumsum(np.tile(counts, B))])
    ci3 = np.tile(ci, B)
    O3, L3 = oa.attention(q, k, v, rp3, ci3, 0.3, B, block)
    np.testing.assert_array_equal(O1, O3)
    np.testing.assert_array_equal(L1, L3)
