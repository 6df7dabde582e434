"""GPU parity of the true block-mass path (through the C ABI): block attention
mass from the dense forward pass's LSE, the mask cut from it, and coverage,
against the oracle in oracle/mass.py."""

import math

import numpy as np
import pytest
import torch

from oracle import mask as om
from oracle import mass as ms
from paper_2606_25040_amd import ops
import workloads as wk
from tests.compare import compare_masks, compare_row

pytestmark = pytest.mark.gpu

# Mass tolerance: logits are fp32 MFMA sums and lse comes from the fp32
# online softmax, so each probability carries ~1e-6 relative error plus the
# lse error (~sqrt(S) fp32 ulps); the block sums add 4096 fp32 terms.
MASS_ATOL = 2e-6
MASS_RTOL = 2e-4




def mass_tie(sa: float, sb: float) -> bool:
    """Two blocks whose GPU masses may come out in either order: each GPU
    mass is within MASS_ATOL + MASS_RTOL * m of the float64 one, so the order
    of two masses closer than twice that bound is not fixed (sa, sb are the
    oracle's log-masses)."""
    ma, mb = math.exp(sa), math.exp(sb)
    return abs(ma - mb) <= 2.0 * (MASS_ATOL + MASS_RTOL * max(ma, mb))


def mass_boundary(n: int) -> float:
    """Bound on the difference of a cumulative mass share between the GPU's
    masses and the oracle's (rows of M sum to 1): the kept masses contribute
    at most k * MASS_ATOL + MASS_RTOL, the row total the same again, k <= n."""
    return 2.0 * (n * MASS_ATOL + MASS_RTOL)


@pytest.fixture(scope="module", autouse=True)
def device():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    ops.load_library()
    torch.cuda.set_device(0)
    yield


def np64(t):
    return t.float().cpu().numpy()


def positional(B, S, H, dtype, seed, scale=0.5):
    g = np.random.Generator(np.random.PCG64(seed))
    f = np.stack([np.sin(2 * np.pi * np.arange(S) / P) for P in (29.0, 170.0, 640.0)] +
                 [np.cos(2 * np.pi * np.arange(S) / P) for P in (29.0, 170.0, 640.0)], 1)
    q = np.empty((B, S, H, 128), np.float32)
    k = np.empty((B, S, H, 128), np.float32)
    for h in range(H):
        W = g.standard_normal((6, 128)) * scale * (1 + h)
        for b in range(B):
            q[b, :, h] = f @ W + 0.5 * g.standard_normal((S, 128))
            k[b, :, h] = f @ W + 0.5 * g.standard_normal((S, 128))
    return torch.from_numpy(q).to(dtype), torch.from_numpy(k).to(dtype)


def gpu_mass(q, k, sm):
    """Dense forward pass for the LSE, then the block mass (V = K: only the
    LSE of the forward pass is used)."""
    qd, kd = q.cuda(), k.cuda()
    _, lse = ops.block_sparse_attn_fwd(qd, kd, kd, None, sm_scale=sm, return_lse=True)
    return ops.attn_block_mass(qd, kd, lse, sm_scale=sm)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
@pytest.mark.parametrize("S,B,H", [(64, 1, 1), (1000, 2, 3), (130, 1, 2)])
def test_block_mass_matches_oracle(dtype, S, B, H):
    q, k = positional(B, S, H, dtype, S + H)
    sm = 1.0 / math.sqrt(128)
    M = gpu_mass(q, k, sm).cpu().numpy().astype(np.float64)
    ref = ms.block_mass_all(np64(q), np64(k), sm)
    assert np.all(np.abs(M - ref) <= MASS_ATOL + MASS_RTOL * ref), float(np.max(np.abs(M - ref)))
    np.testing.assert_allclose(M.sum(axis=-1), 1.0, atol=1e-4)


def oracle_mask_of(M, top_p, mk, mask_batch):
    """OracleMask whose 'scores' are log-masses: softmax(log m) = m / sum(m),
    so the comparator's near-tie and boundary rules apply to the mass shares."""
    B, H, n, _ = M.shape
    rp, ci = ms.mask_from_mass(M, top_p, mk)
    with np.errstate(divide="ignore"):
        scores = np.log(M.reshape(B * H * n, n))
    return om.OracleMask(rp, ci, scores, n, H, mask_batch)


@pytest.mark.parametrize("top_p,mk", [(0.9, 0.0), (0.5, 0.1), (0.0, 0.25), (1.0, 0.0), (0.97, 0.05)])
def test_mask_from_mass_matches_oracle(top_p, mk):
    S, B, H = 1500, 2, 2
    q, k = positional(B, S, H, torch.bfloat16, 77)
    sm = 1.0 / math.sqrt(128)
    Md = gpu_mass(q, k, sm)
    m = ops.select_block_mask(Md, S, top_p, mk)
    rp, ci = m.to_host()
    assert ops.validate_block_mask(m) == 0
    M = Md.cpu().numpy().astype(np.float64)
    # same masses on both sides: the selection itself must agree exactly
    o = oracle_mask_of(M, top_p, mk, B)
    rep = compare_masks(rp, ci, o, range(m.rows), top_p, mk)
    assert rep.ok and not rep.failing, rep.failing[:3]
    # against the oracle's own float64 masses: every row exact, or a near-tie
    # within what the GPU mass error allows
    ref = ms.block_mass_all(np64(q), np64(k), sm)
    o2 = oracle_mask_of(ref, top_p, mk, B)
    n = ref.shape[-1]
    rep2 = compare_masks(rp, ci, o2, range(m.rows), top_p, mk, tie=mass_tie, boundary=mass_boundary(n))
    assert rep2.ok, rep2.failing[:3]


def test_selection_of_exact_mass_ties_and_zero_rows():
    S, H = 64 * 20, 2
    n = 20
    M = np.zeros((1, H, n, n), np.float32)
    M[0, 0] = 1.0 / n                                       # every block tied
    M[0, 1, :, ::2] = 0.1                                   # ten-way ties
    M[0, 1, 3] = 0.0                                        # a row without mass
    Md = torch.from_numpy(M).cuda()
    for top_p, mk in ((0.5, 0.0), (0.35, 0.2), (0.0, 0.15)):
        m = ops.select_block_mask(Md, S, top_p, mk)
        rp, ci = m.to_host()
        o = oracle_mask_of(M.astype(np.float64), top_p, mk, 1)
        rep = compare_masks(rp, ci, o, range(m.rows), top_p, mk)
        assert rep.ok, rep.failing[:3]
        # a row without mass never reaches top_p > 0: every block is kept
        if top_p > 0:
            r = (0 * H + 1) * n + 3
            assert list(ci[rp[r]:rp[r + 1]]) == list(range(n))


@pytest.mark.parametrize("n", [300, 1182, 2048, 3000, 4096])
@pytest.mark.parametrize("top_p,mk", [(0.5, 0.0), (0.999999, 0.0), (0.9999, 0.6), (0.3, 0.95)])
def test_selection_over_masses_spanning_many_magnitudes(n, top_p, mk):
    """Masses spread log-uniformly over 30 decades give the first radix digit
    of the keys (sign and top exponent bits) several distinct values, and
    top_p near 1 or a large floor puts the boundary deep in the order: the
    selection's walk over the first digit's top values runs out and the
    histogram takes over.  Same masses on both sides: exact agreement."""
    H = 2
    S = 64 * n
    rng = np.random.Generator(np.random.PCG64(n))
    M = (10.0 ** rng.uniform(-30, 0, (1, H, 8, n))).astype(np.float32)
    M[0, 1, 5, rng.integers(0, n, n // 3)] = 0.0             # zero-mass blocks in one row
    # a q-block count of 8 rows per head: pad the mass tensor to the n q-blocks S implies
    Mfull = np.zeros((1, H, n, n), np.float32)
    Mfull[:, :, :8] = M
    Mfull[:, :, 8:] = 1.0 / n
    Md = torch.from_numpy(Mfull).cuda()
    m = ops.select_block_mask(Md, S, top_p, mk)
    rp, ci = m.to_host()
    assert ops.validate_block_mask(m) == 0
    for h in range(H):
        for i in range(8):
            r = h * n + i
            row = Mfull[0, h, i].astype(np.float64)
            with np.errstate(divide="ignore"):
                res = compare_row(ci[rp[r]:rp[r + 1]], ms.select_row_from_mass(row, top_p, mk), np.log(row),
                                  top_p, mk)
            assert res in ("exact", "excused"), (h, i, res)


def test_coverage_matches_oracle():
    S, B, H = 1000, 2, 3
    q, k = positional(B, S, H, torch.bfloat16, 5)
    sm = 1.0 / math.sqrt(128)
    Md = gpu_mass(q, k, sm)
    M = Md.cpu().numpy().astype(np.float64)
    n = M.shape[-1]
    rng = np.random.Generator(np.random.PCG64(3))
    for mask_batch in (1, B):
        rp, ci = wk.random_csr(rng, mask_batch * H * n, n, 0.4)
        mask = ops.BlockMask.from_host(rp, ci, mask_batch, H, n)
        cov = ops.mask_coverage(mask, Md, S).cpu().numpy()
        ref = ms.coverage(rp, ci, mask_batch, M, S)
        np.testing.assert_allclose(cov, ref, rtol=1e-12, atol=1e-12)
        ref64 = ms.coverage(rp, ci, mask_batch, ms.block_mass_all(np64(q), np64(k), sm), S)
        np.testing.assert_allclose(cov, ref64, atol=1e-4)
    full = ops.BlockMask.from_host(np.arange(0, H * n * n + 1, n), np.tile(np.arange(n), H * n), 1, H, n)
    np.testing.assert_allclose(ops.mask_coverage(full, Md, S).cpu().numpy(), 1.0, atol=1e-4)
    own = ops.select_block_mask(Md, S, 0.8, 0.0)
    assert (ops.mask_coverage(own, Md, S).cpu().numpy() >= 0.8 - 1e-6).all()


def test_full_size_reuse_workload_sampled_rows():
    """Historical request of the 480p reuse workload at full size: sampled
    rows of the GPU block mass against rows the oracle computes one by one
    from the dense attention probabilities of those q-blocks."""
    wl = wk.WORKLOADS["wan14b_480p_reuse_bf16"]
    inp = wk.make_inputs(wl)
    qh, kh = inp.mask_q[:, :, :4].contiguous(), inp.mask_k[:, :, :4].contiguous()   # 4 heads
    Md = gpu_mass(qh, kh, wl.sm_scale)
    M = Md.cpu().numpy()
    S, n = wl.S, wl.n_blocks
    rng = np.random.default_rng(11)
    w = ms.valid_counts(S)
    for h in range(4):
        K = qh[0, :, h].float().numpy().astype(np.float64), kh[0, :, h].float().numpy().astype(np.float64)
        for i in list(rng.choice(n - 1, 3, replace=False)) + [n - 1]:
            Q = K[0][i * 64:min(i * 64 + 64, S)]
            z = wl.sm_scale * (Q @ K[1].T)
            z -= z.max(axis=1, keepdims=True)
            P = np.exp(z)
            P /= P.sum(axis=1, keepdims=True)
            row = np.array([P[:, j * 64:min(j * 64 + 64, S)].sum() for j in range(n)]) / w[i]
            assert np.all(np.abs(M[0, h, i] - row) <= MASS_ATOL + MASS_RTOL * row), (h, i)
