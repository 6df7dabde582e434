"""GPU parity of the first-frame key enhancement (Eq. 1) through the C ABI:
attention (f16, bf16, fp8), the mask builder and the block mass with a key
scale, against the oracle applied to explicitly scaled keys
(oracle/guidance.py)."""

import math

import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import fp8 as of
from oracle import guidance as og
from oracle import mask as om
from oracle import mass as ms
from paper_2606_25040_amd import ops
import workloads as wk
from tests.compare import compare_masks, max_abs_err

pytestmark = pytest.mark.gpu

TOL16 = 2e-3
TOL8 = 3e-2
MASS_ATOL = 2e-6
MASS_RTOL = 2e-4


@pytest.fixture(scope="module", autouse=True)
def device():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    ops.load_library()
    torch.cuda.set_device(0)
    yield


def np64(t):
    return t.float().cpu().numpy().astype(np.float64)


def rand_qkv(seed, B, S, H, dtype, scale=0.5):
    gen = torch.Generator().manual_seed(seed)
    q = (torch.randn(B, S, H, 128, generator=gen) * scale).to(dtype)
    k = (torch.randn(B, S, H, 128, generator=gen) * scale).to(dtype)
    v = torch.randn(B, S, H, 128, generator=gen).to(dtype)
    return q, k, v


def within(got, ref, dtype, atol):
    rel = 2.0 ** -8 if dtype == torch.bfloat16 else 2.0 ** -10
    return bool(np.all(np.abs(got - ref) <= atol + rel * np.abs(ref)))


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
@pytest.mark.parametrize("n_first,beta,dense", [(300, 1.7, False), (64, 2.0, False), (1000, 1.3, False),
                                                (1, 0.5, False), (517, 1.5, True)])
def test_attention_with_key_scale(dtype, n_first, beta, dense):
    B, S, H = 2, 1000, 2
    q, k, v = rand_qkv(n_first, B, S, H, dtype)
    n = (S + 63) // 64
    if dense:
        rp, ci, mask = np.arange(0, H * n * n + 1, n), np.tile(np.arange(n), H * n), None
    else:
        rng = np.random.Generator(np.random.PCG64(n_first))
        rp, ci = wk.random_csr(rng, H * n, n, 0.4)
        mask = ops.BlockMask.from_host(rp, ci, 1, H, n)
    sm = 1.0 / math.sqrt(128)
    out, lse = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), mask, sm_scale=sm,
                                         return_lse=True, key_scale=(n_first, beta))
    torch.cuda.synchronize()
    ke = og.enhance_first_frame_keys(np64(k), n_first, beta)
    O, L = oa.attention(np64(q), ke, np64(v), rp, ci, sm, 1)
    assert within(np64(out), O, dtype, TOL16), float(np.max(np.abs(np64(out) - O)))
    lg = lse.cpu().numpy()
    fin = np.isfinite(L)
    assert np.array_equal(np.isfinite(lg), fin)
    assert np.max(np.abs(lg[fin] - L[fin])) <= 1e-3


def test_plain_key_scale_is_bitwise_the_plain_path():
    B, S, H = 1, 700, 2
    q, k, v = (x.cuda() for x in rand_qkv(1, B, S, H, torch.bfloat16))
    n = (S + 63) // 64
    rp, ci = wk.random_csr(np.random.Generator(np.random.PCG64(1)), H * n, n, 0.5)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n)
    ref = ops.block_sparse_attn_fwd(q, k, v, mask)
    for ks in ((0, 3.0), (500, 1.0)):
        out = ops.block_sparse_attn_fwd(q, k, v, mask, key_scale=ks)
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16))


def test_attention_fp8_with_key_scale():
    B, S, H = 2, 1000, 3
    q, k, v = rand_qkv(5, B, S, H, torch.bfloat16)
    n = (S + 63) // 64
    rng = np.random.Generator(np.random.PCG64(5))
    rp, ci = wk.random_csr(rng, H * n, n, 0.5)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n)
    (qc, qs), (kc, ks), (vc, vs) = (ops.quantize_fp8_blockwise(x.cuda()) for x in (q, k, v))
    n_first, beta = 333, 1.6
    out = ops.block_sparse_attn_fwd(qc, kc, vc, mask, scales=(qs, ks, vs), key_scale=(n_first, beta))
    torch.cuda.synchronize()
    deq = [of.dequantize_blockwise(c.cpu().numpy(), s.cpu().numpy()) for c, s in ((qc, qs), (kc, ks), (vc, vs))]
    ke = og.enhance_first_frame_keys(deq[1], n_first, beta)
    O, _ = oa.attention(deq[0], ke, deq[2], rp, ci, 1.0 / math.sqrt(128), 1)
    assert within(np64(out), O, torch.bfloat16, TOL8), float(np.max(np.abs(np64(out) - O)))


def positional(B, S, H, dtype, seed):
    g = np.random.Generator(np.random.PCG64(seed))
    f = np.stack([np.sin(2 * np.pi * np.arange(S) / P) for P in (37.0, 200.0, 911.0)] +
                 [np.cos(2 * np.pi * np.arange(S) / P) for P in (37.0, 200.0, 911.0)], 1)
    q = np.empty((B, S, H, 128), np.float32)
    k = np.empty((B, S, H, 128), np.float32)
    for h in range(H):
        W = g.standard_normal((6, 128)) * 0.5
        for b in range(B):
            q[b, :, h] = f @ W + 0.5 * g.standard_normal((S, 128))
            k[b, :, h] = f @ W + 0.5 * g.standard_normal((S, 128))
    return torch.from_numpy(q).to(dtype), torch.from_numpy(k).to(dtype)


@pytest.mark.parametrize("n_first,beta", [(600, 1.8), (128, 3.0), (2000, 0.7)])
def test_builder_with_key_scale(n_first, beta):
    B, S, H = 1, 2000, 2
    q, k = positional(B, S, H, torch.bfloat16, n_first)
    top_p, mk = 0.6, 0.05
    sm = 1.0 / math.sqrt(128)
    m = ops.build_block_mask(q.cuda(), k.cuda(), top_p, mk, sm_scale=sm, key_scale=(n_first, beta))
    rp, ci = m.to_host()
    o = om.build_block_mask(np64(q), og.enhance_first_frame_keys(np64(k), n_first, beta), sm, top_p, mk)
    rep = compare_masks(rp, ci, o, range(m.rows), top_p, mk)
    assert rep.ok and not rep.failing, rep.failing[:3]
    # the enhancement changes the mask: first-frame columns gain
    plain = ops.build_block_mask(q.cuda(), k.cuda(), top_p, mk, sm_scale=sm)
    if beta > 1:
        n_ff = (n_first + 63) // 64
        prp, pci = plain.to_host()
        assert np.sum(ci < n_ff) >= np.sum(pci < n_ff)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
def test_block_mass_with_key_scale(dtype):
    B, S, H = 1, 1000, 2
    q, k = positional(B, S, H, dtype, 17)
    sm = 1.0 / math.sqrt(128)
    ks = (450, 1.4)
    qd, kd = q.cuda(), k.cuda()
    _, lse = ops.block_sparse_attn_fwd(qd, kd, kd, None, sm_scale=sm, return_lse=True, key_scale=ks)
    M = ops.attn_block_mass(qd, kd, lse, sm_scale=sm, key_scale=ks).cpu().numpy().astype(np.float64)
    ref = ms.block_mass_all(np64(q), og.enhance_first_frame_keys(np64(k), *ks), sm)
    assert np.all(np.abs(M - ref) <= MASS_ATOL + MASS_RTOL * ref), float(np.max(np.abs(M - ref)))
    np.testing.assert_allclose(M.sum(axis=-1), 1.0, atol=1e-4)


def test_full_size_720p_fp8_with_first_frame_enhancement():
    """The 720p 14B workload (40 heads, 75 600 tokens, first frame 45 x 80 =
    3600 tokens) with its own mask and beta = 1.3: sampled q-blocks of every
    head against the oracle on dequantised, enhanced keys."""
    wl = wk.WORKLOADS["wan14b_720p_fp8"]
    inp = wk.make_inputs(wl)
    n_first = og.first_frame_tokens(wl.grid)
    beta = 1.3
    mask = ops.build_block_mask(inp.mask_q.cuda(), inp.mask_k.cuda(), wl.top_p, wl.min_top_k,
                                sm_scale=wl.sm_scale, key_scale=(n_first, beta))
    (qc, qs), (kc, ks), (vc, vs) = (ops.quantize_fp8_blockwise(x.cuda()) for x in (inp.q, inp.k, inp.v))
    out = ops.block_sparse_attn_fwd(qc, kc, vc, mask, scales=(qs, ks, vs), sm_scale=wl.sm_scale,
                                    key_scale=(n_first, beta))
    torch.cuda.synchronize()
    rp, ci = mask.to_host()
    n = wl.n_blocks
    rng = np.random.Generator(np.random.PCG64(3600))
    worst = 0.0
    for h in range(0, wl.H, 3):
        sl = lambda c, s: of.dequantize_blockwise(c[0:1, :, h:h + 1].cpu().numpy(),
                                                  s[0:1, h:h + 1].cpu().numpy())[0, :, 0]
        qh, kh, vh = sl(qc, qs), sl(kc, ks), sl(vc, vs)
        kh = og.enhance_first_frame_keys(kh[None, :, None, :], n_first, beta)[0, :, 0]
        oh = np64(out[0, :, h].cpu())
        for i in sorted({0, n_first // 64, n - 1} | set(rng.integers(0, n, 2).tolist())):
            r = oa.mask_row_index(0, h, i, wl.H, n, 1)
            o_ref, _ = oa.attention_block(qh, kh, vh, oa.row_blocks(rp, ci, r), i, wl.sm_scale)
            worst = max(worst, max_abs_err(oh[i * 64:i * 64 + o_ref.shape[0]], o_ref))
    assert worst <= TOL8, worst

