"""Sequence-length sweep through the C ABI: every stage at lengths around the
block boundaries (a single token, one block minus / plus one, two kv blocks
of 128 minus / plus one, a few thousand tokens), against the oracle.  The
quantiser is bit-exact; masks follow the mask comparator; outputs follow the
attention tolerances."""

import math

import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import fp8 as of
from oracle import mask as om
from paper_2606_25040_amd import ops
import workloads as wk
from tests.compare import compare_masks

pytestmark = pytest.mark.gpu

LENGTHS = [1, 2, 63, 64, 65, 127, 128, 129, 255, 256, 257, 1983, 4097]
SM = 1.0 / math.sqrt(128)


@pytest.fixture(scope="module", autouse=True)
def device():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    ops.load_library()
    torch.cuda.set_device(0)
    yield


def np64(t):
    return t.float().cpu().numpy().astype(np.float64)


def qkv(S, dtype, seed, B=1, H=2):
    gen = torch.Generator().manual_seed(seed)
    q = (torch.randn(B, S, H, 128, generator=gen) * 0.5).to(dtype)
    k = (torch.randn(B, S, H, 128, generator=gen) * 0.5).to(dtype)
    v = torch.randn(B, S, H, 128, generator=gen).to(dtype)
    return q, k, v


def within(got, ref, dtype, atol):
    rel = 2.0 ** -8 if dtype == torch.bfloat16 else 2.0 ** -10
    return bool(np.all(np.abs(got - ref) <= atol + rel * np.abs(ref)))


@pytest.mark.parametrize("S", LENGTHS)
def test_quantizer_lengths(S):
    q, _, _ = qkv(S, torch.bfloat16, S)
    codes, scales = ops.quantize_fp8_blockwise(q.cuda())
    torch.cuda.synchronize()
    oc, os_ = of.quantize_blockwise(np64(q))
    assert np.array_equal(codes.cpu().numpy(), oc)
    assert np.array_equal(scales.cpu().numpy(), os_)
    # the variant with block sums: the same codes and scales, and sums / valid
    # count equal to the oracle's block means
    c2, s2, sums = ops.quantize_fp8_blockwise_sums(q.cuda())
    torch.cuda.synchronize()
    assert torch.equal(c2, codes) and torch.equal(s2.view(torch.int32), scales.view(torch.int32))
    cnt = np.array([min(64, S - 64 * i) for i in range((S + 63) // 64)], dtype=np.float64)
    means = sums.cpu().numpy() / cnt[None, None, :, None]
    for h in range(q.shape[2]):
        assert np.array_equal(means[0, h], om.pool_means(np64(q)[0, :, h]))


@pytest.mark.parametrize("kv_block", [64, 128])
@pytest.mark.parametrize("S", LENGTHS)
def test_builder_from_block_sums_lengths(S, kv_block):
    """The builder from the quantiser's block sums gives bitwise the mask of
    the builder reading the same bf16 Q and K at every length."""
    q, k, _ = qkv(S, torch.bfloat16, 3 * S + 1)
    q, k = q.cuda(), k.cuda()
    _, _, qs = ops.quantize_fp8_blockwise_sums(q)
    _, _, kss = ops.quantize_fp8_blockwise_sums(k)
    m = ops.build_block_mask_from_sums(qs, kss, S, 0.7, 0.1, sm_scale=SM, kv_block=kv_block)
    ref = ops.build_block_mask(q, k, 0.7, 0.1, sm_scale=SM, kv_block=kv_block)
    rp, ci = m.to_host()
    rrp, rci = ref.to_host()
    assert np.array_equal(rp, rrp) and np.array_equal(ci, rci), S


@pytest.mark.parametrize("kv_block", [64, 128])
@pytest.mark.parametrize("S", LENGTHS)
def test_builder_lengths(S, kv_block):
    q, k, _ = qkv(S, torch.bfloat16, 3 * S + 1)
    m = ops.build_block_mask(q.cuda(), k.cuda(), 0.7, 0.1, sm_scale=SM, kv_block=kv_block)
    rp, ci = m.to_host()
    assert ops.validate_block_mask(m) == 0
    o = om.build_block_mask(np64(q), np64(k), SM, 0.7, 0.1, kv_block=kv_block)
    rep = compare_masks(rp, ci, o, range(m.rows), 0.7, 0.1)
    assert rep.ok and not rep.failing, (S, rep.failing[:3])


@pytest.mark.parametrize("kv_block", [64, 128])
@pytest.mark.parametrize("dtype", ["bf16", "f16", "fp8"])
@pytest.mark.parametrize("S", LENGTHS)
def test_attention_lengths(S, dtype, kv_block):
    tdt = torch.float16 if dtype == "f16" else torch.bfloat16
    B, H = 2, 2
    q, k, v = qkv(S, tdt, 7 * S + kv_block, B, H)
    n = (S + 63) // 64
    nk = (S + kv_block - 1) // kv_block
    rng = np.random.Generator(np.random.PCG64(S + kv_block))
    rp, ci = wk.random_csr(rng, B * H * n, nk, 0.5, empty_frac=0.1 if n > 1 else 0.0)
    mask = ops.BlockMask.from_host(rp, ci, B, H, n, block=kv_block)
    if dtype == "fp8":
        cs = [ops.quantize_fp8_blockwise(x.cuda()) for x in (q, k, v)]
        out, lse = ops.block_sparse_attn_fwd(*[c for c, _ in cs], mask, sm_scale=SM,
                                             scales=tuple(s for _, s in cs), return_lse=True)
        ins = [of.dequantize_blockwise(c.cpu().numpy(), s.cpu().numpy()) for c, s in cs]
        atol = 3e-2
    else:
        out, lse = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), mask, sm_scale=SM, return_lse=True)
        ins = [np64(x) for x in (q, k, v)]
        atol = 2e-3
    torch.cuda.synchronize()
    O, L = oa.attention(*ins, rp, ci, SM, B, kv_block=kv_block)
    if dtype == "fp8":
        # P is rounded to e4m3 (relative error <= 2^-4 per weight) before PV, so
        # |dO| <= 2^-4 * sum_c p_c |v_c|; with few keys per row (short
        # sequences) that exceeds the 3e-2 budget the workloads are held to
        Oabs, _ = oa.attention(ins[0], ins[1], np.abs(ins[2]), rp, ci, SM, B, kv_block=kv_block)
        err = np.abs(np64(out) - O)
        bound = np.maximum(atol, 1e-3 + 2.0 ** -4 * Oabs) + 2.0 ** -8 * np.abs(O)
        assert np.all(err <= bound), float(np.max(err - bound))
    else:
        assert within(np64(out), O, tdt, atol), float(np.max(np.abs(np64(out) - O)))
    lg = lse.cpu().numpy()
    fin = np.isfinite(L)
    assert np.array_equal(np.isfinite(lg), fin)
    if fin.any():
        assert np.max(np.abs(lg[fin] - L[fin])) <= 1e-3
