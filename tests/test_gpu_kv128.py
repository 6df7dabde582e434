"""GPU parity of masks with kv blocks of 128 tokens and q-blocks of 64 (the
paper's own kernel geometry) through the C ABI: builder, attention (f16,
bf16, fp8), plan, checker, block mass, selection from mass, coverage and
visit refreshing, against the oracle with kv_block = 128."""

import math

import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import fallback as fb
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


def within(got, ref, dtype, atol):
    rel = 2.0 ** -8 if dtype == torch.bfloat16 else 2.0 ** -10
    return bool(np.all(np.abs(got - ref) <= atol + rel * np.abs(ref)))


def expand(rp, ci, n64):
    """kv-128 CSR -> kv-64 CSR listing the halves 2J, 2J + 1 (< n64) of each J."""
    rows = [[x for J in ci[rp[r]:rp[r + 1]] for x in (2 * J, 2 * J + 1) if x < n64] for r in range(len(rp) - 1)]
    out_rp = np.concatenate([[0], np.cumsum([len(x) for x in rows])]).astype(np.int64)
    out_ci = np.array([x for r in rows for x in r], dtype=np.int64)
    return out_rp, out_ci


# S values: n_q even / odd, last kv block full, half-full, or a 64-token stub
SHAPES = [(1000, 2, 2), (960, 1, 3), (1090, 2, 1), (128, 1, 2), (100, 1, 1)]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
@pytest.mark.parametrize("S,B,H", SHAPES)
def test_attention_kv128_matches_oracle(dtype, S, B, H):
    q, k, v = rand_qkv(S, B, S, H, dtype)
    n, nk = (S + 63) // 64, (S + 127) // 128
    rng = np.random.Generator(np.random.PCG64(S + 1))
    rp, ci = wk.random_csr(rng, H * n, nk, 0.5, empty_frac=0.1 if n > 2 else 0.0)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n, block=128)
    sm = 1.0 / math.sqrt(128)
    out, lse = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), mask, sm_scale=sm, return_lse=True)
    torch.cuda.synchronize()
    O, L = oa.attention(np64(q), np64(k), np64(v), rp, ci, sm, 1, kv_block=128)
    assert within(np64(out), O, dtype, TOL16), float(np.max(np.abs(np64(out) - O)))
    lg = lse.cpu().numpy()
    fin = np.isfinite(L)
    assert np.array_equal(np.isfinite(lg), fin)
    if fin.any():
        assert np.max(np.abs(lg[fin] - L[fin])) <= 1e-3
    # the same sub-blocks in the same order as the expanded kv-64 mask: bitwise equal
    erp, eci = expand(rp, ci, n)
    out64 = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), ops.BlockMask.from_host(erp, eci, 1, H, n),
                                      sm_scale=sm)
    assert torch.equal(out.view(torch.int16), out64.view(torch.int16))


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
@pytest.mark.parametrize("S,n_first,beta", [(1090, 300, 1.6), (1000, 1000, 0.8)])
def test_attention_kv128_key_scale_per_request_masks(dtype, S, n_first, beta):
    """kv blocks of 128 with the first-frame key enhancement and one mask per
    request (mask_batch = B): the KSCALE x KV2 instantiation of the 16-bit
    kernel against the oracle on explicitly scaled keys."""
    B, H = 2, 2
    q, k, v = rand_qkv(S + n_first, B, S, H, dtype)
    n, nk = (S + 63) // 64, (S + 127) // 128
    rng = np.random.Generator(np.random.PCG64(n_first))
    rp, ci = wk.random_csr(rng, B * H * n, nk, 0.4, empty_frac=0.1)
    mask = ops.BlockMask.from_host(rp, ci, B, H, n, block=128)
    sm = 1.0 / math.sqrt(128)
    out, lse = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), mask, sm_scale=sm, return_lse=True,
                                         key_scale=(n_first, beta))
    torch.cuda.synchronize()
    ke = og.enhance_first_frame_keys(np64(k), n_first, beta)
    O, L = oa.attention(np64(q), ke, np64(v), rp, ci, sm, B, kv_block=128)
    assert within(np64(out), O, dtype, TOL16), float(np.max(np.abs(np64(out) - O)))
    lg = lse.cpu().numpy()
    fin = np.isfinite(L)
    assert np.array_equal(np.isfinite(lg), fin)
    assert np.max(np.abs(lg[fin] - L[fin])) <= 1e-3
    erp, eci = expand(rp, ci, n)
    out64 = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), ops.BlockMask.from_host(erp, eci, B, H, n),
                                      sm_scale=sm, key_scale=(n_first, beta))
    assert torch.equal(out.view(torch.int16), out64.view(torch.int16))


@pytest.mark.parametrize("S", [1000, 960])
def test_attention_fp8_kv128(S):
    B, H = 2, 2
    q, k, v = rand_qkv(7, B, S, H, torch.bfloat16)
    n, nk = (S + 63) // 64, (S + 127) // 128
    rng = np.random.Generator(np.random.PCG64(8))
    rp, ci = wk.random_csr(rng, H * n, nk, 0.5, empty_frac=0.05)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n, block=128)
    (qc, qs), (kc, ks), (vc, vs) = (ops.quantize_fp8_blockwise(x.cuda()) for x in (q, k, v))
    out = ops.block_sparse_attn_fwd(qc, kc, vc, mask, scales=(qs, ks, vs), key_scale=(200, 1.4))
    torch.cuda.synchronize()
    deq = [of.dequantize_blockwise(c.cpu().numpy(), s.cpu().numpy()) for c, s in ((qc, qs), (kc, ks), (vc, vs))]
    O, _ = oa.attention(deq[0], og.enhance_first_frame_keys(deq[1], 200, 1.4), deq[2], rp, ci,
                        1.0 / math.sqrt(128), 1, kv_block=128)
    assert within(np64(out), O, torch.bfloat16, TOL8), float(np.max(np.abs(np64(out) - O)))
    erp, eci = expand(rp, ci, n)
    out64 = ops.block_sparse_attn_fwd(qc, kc, vc, ops.BlockMask.from_host(erp, eci, 1, H, n),
                                      scales=(qs, ks, vs), key_scale=(200, 1.4))
    assert torch.equal(out.view(torch.int16), out64.view(torch.int16))


@pytest.mark.parametrize("kind", ["bf16", "fp8"])
def test_attention_kv128_skips_out_of_range_ids(kind):
    """Ids of 128-token blocks outside [0, nk) are skipped: -1 ahead of a
    row's ids, or nk and nk + 5 after them, leave the output of the clean
    rows; both 64-token halves of such an id fall outside [0, n) and the
    rotated walk start has to land on the valid halves."""
    B, S, H = 1, 1090, 3
    q, k, v = rand_qkv(19, B, S, H, torch.bfloat16)
    n, nk = (S + 63) // 64, (S + 127) // 128
    rng = np.random.Generator(np.random.PCG64(23))
    rp, ci = wk.random_csr(rng, H * n, nk, 0.4, empty_frac=0.1)
    rows = []
    for r in range(H * n):
        ids = [int(j) for j in ci[rp[r]:rp[r + 1]]]
        if r % 3 == 0:
            ids = [-1] + ids
        elif r % 3 == 1:
            ids = ids + [nk, nk + 5]
        rows.append(ids)
    assert any(len(x) == 1 and x[0] == -1 for x in rows)
    rp2 = np.concatenate([[0], np.cumsum([len(x) for x in rows])])
    ci2 = np.array([j for x in rows for j in x], dtype=np.int64)
    mask = ops.BlockMask.from_host(rp2, ci2, 1, H, n, block=128)
    sm = 1.0 / math.sqrt(128)
    if kind == "fp8":
        (qc, qs), (kc, ks), (vc, vs) = (ops.quantize_fp8_blockwise(x.cuda()) for x in (q, k, v))
        out, lse = ops.block_sparse_attn_fwd(qc, kc, vc, mask, scales=(qs, ks, vs), sm_scale=sm,
                                             return_lse=True)
        deq = [of.dequantize_blockwise(c.cpu().numpy(), s_.cpu().numpy())
               for c, s_ in ((qc, qs), (kc, ks), (vc, vs))]
        O, L = oa.attention(*deq, rp, ci, sm, 1, kv_block=128)
        atol = TOL8
    else:
        out, lse = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), mask, sm_scale=sm,
                                             return_lse=True)
        O, L = oa.attention(np64(q), np64(k), np64(v), rp, ci, sm, 1, kv_block=128)
        atol = TOL16
    torch.cuda.synchronize()
    assert within(np64(out), O, torch.bfloat16, atol), float(np.max(np.abs(np64(out) - O)))
    lg = lse.cpu().numpy()
    fin = np.isfinite(L)
    assert np.array_equal(np.isfinite(lg), fin)
    assert np.max(np.abs(lg[fin] - L[fin])) <= 1e-3


@pytest.mark.parametrize("S,top_p,mk,key_scale", [(2000, 0.6, 0.05, None), (1090, 0.9, 0.0, None),
                                                  (960, 0.0, 0.3, (300, 1.7)), (64 * 4096, 0.5, 0.0, None)])
def test_builder_kv128_matches_oracle(S, top_p, mk, key_scale):
    B, H = 1, 1 if S > 10000 else 2
    q, k = positional(B, S, H, torch.bfloat16, S)
    sm = 1.0 / math.sqrt(128)
    m = ops.build_block_mask(q.cuda(), k.cuda(), top_p, mk, sm_scale=sm, kv_block=128, key_scale=key_scale,
                             return_scores=True)
    rp, ci = m.to_host()
    assert m.block == 128 and m.n_kv == (S + 127) // 128
    assert ops.validate_block_mask(m) == 0
    kk = np64(k) if key_scale is None else og.enhance_first_frame_keys(np64(k), *key_scale)
    rows = range(m.rows) if S < 10000 else range(0, m.rows, 97)
    o = om.build_block_mask(np64(q), kk, sm, top_p, mk, kv_block=128)
    rep = compare_masks(rp, ci, o, rows, top_p, mk)
    assert rep.ok and not rep.failing, rep.failing[:3]
    np.testing.assert_allclose(m.block_scores.cpu().numpy(), o.scores, rtol=1e-6, atol=1e-7)


def test_builder_kv128_on_fp8_codes():
    B, S, H = 1, 1500, 2
    q, k = positional(B, S, H, torch.bfloat16, 31)
    (qc, qs), (kc, ks) = (ops.quantize_fp8_blockwise(x.cuda()) for x in (q, k))
    sm = 1.0 / math.sqrt(128)
    m = ops.build_block_mask(qc, kc, 0.7, 0.05, sm_scale=sm, scales=(qs, ks), kv_block=128)
    rp, ci = m.to_host()
    dq = of.dequantize_blockwise(qc.cpu().numpy(), qs.cpu().numpy())
    dk = of.dequantize_blockwise(kc.cpu().numpy(), ks.cpu().numpy())
    o = om.build_block_mask(dq, dk, sm, 0.7, 0.05, kv_block=128)
    rep = compare_masks(rp, ci, o, range(m.rows), 0.7, 0.05)
    assert rep.ok and not rep.failing, rep.failing[:3]


def test_checker_and_plan_kv128():
    H, n = 2, 9                     # S in (512, 576]: 5 kv blocks of 128
    rp = np.array([0, 2, 3, 3, 5, 6, 8, 9, 9, 10] + [10 + x for x in range(1, 10)])
    ci = np.array([0, 4, 1, 2, 4, 0, 1, 2, 3, 0] + [3] * 9)
    good = ops.BlockMask.from_host(rp, ci, 1, H, n, block=128)
    assert ops.validate_block_mask(good) == 0
    bad = ci.copy()
    bad[1] = 5                                               # out of [0, 5)
    assert ops.validate_block_mask(ops.BlockMask.from_host(rp, bad, 1, H, n, block=128)) & 4
    # plan: a listed kv block of 128 costs two 64-token blocks
    B = 24
    rng = np.random.Generator(np.random.PCG64(5))
    Hp, nq = 5, 12
    nk = 6
    counts = rng.integers(0, nk + 1, B * Hp * nq)
    prp = np.concatenate([[0], np.cumsum(counts)])
    pci = np.concatenate([np.sort(rng.choice(nk, c, replace=False)) for c in counts])
    mask = ops.BlockMask.from_host(prp, pci, B, Hp, nq, block=128)
    order = ops.plan_block_mask(mask, B, 64 * nq).cpu().tolist()
    cost = [2 * (prp[(u + 1) * nq] - prp[u * nq]) + nq for u in range(B * Hp)]
    U = B * Hp
    by = sorted(range(U), key=lambda u: (-cost[u], u))
    cap = [U // 8 + (1 if x < U % 8 else 0) for x in range(8)]
    load, used, xcd = [0] * 8, [0] * 8, [0] * U
    for u in by:
        best = min((x for x in range(8) if used[x] < cap[x]), key=lambda x: (load[x], x))
        load[best] += cost[u]
        used[best] += 1
        xcd[u] = best
    assert order == [u for x in range(8) for u in range(U) if xcd[u] == x]


@pytest.mark.parametrize("dtype,key_scale", [(torch.bfloat16, None), (torch.float16, None),
                                             (torch.bfloat16, (450, 1.4))])
def test_block_mass_selection_coverage_kv128(dtype, key_scale):
    B, S, H = 1, 1090, 2
    q, k = positional(B, S, H, dtype, 41)
    sm = 1.0 / math.sqrt(128)
    qd, kd = q.cuda(), k.cuda()
    _, lse = ops.block_sparse_attn_fwd(qd, kd, kd, None, sm_scale=sm, return_lse=True, key_scale=key_scale)
    Md = ops.attn_block_mass(qd, kd, lse, sm_scale=sm, kv_block=128, key_scale=key_scale)
    M = Md.cpu().numpy().astype(np.float64)
    kref = np64(k) if key_scale is None else og.enhance_first_frame_keys(np64(k), *key_scale)
    ref = ms.block_mass_all(np64(q), kref, sm, kv_block=128)
    assert M.shape == ref.shape
    assert np.all(np.abs(M - ref) <= MASS_ATOL + MASS_RTOL * ref), float(np.max(np.abs(M - ref)))
    m = ops.select_block_mask(Md, S, 0.8, 0.1, kv_block=128)
    rp, ci = m.to_host()
    n = M.shape[2]
    with np.errstate(divide="ignore"):
        scores = np.log(M.reshape(B * H * n, -1))
    orp, oci = ms.mask_from_mass(M, 0.8, 0.1)
    o = om.OracleMask(orp, oci, scores, n, H, B, M.shape[3])
    rep = compare_masks(rp, ci, o, range(m.rows), 0.8, 0.1)
    assert rep.ok and not rep.failing, rep.failing[:3]
    cov = ops.mask_coverage(m, Md, S).cpu().numpy()
    np.testing.assert_allclose(cov, ms.coverage(rp, ci, B, M, S), rtol=1e-12, atol=1e-12)
    assert (cov >= 0.8 - 1e-6).all()


def test_visit_refresh_kv128_group():
    H, n = 3, 19
    nk = 10
    rows = H * n
    rng = np.random.Generator(np.random.PCG64(12))
    hm = [wk.random_csr(rng, rows, nk, float(rng.uniform(0.05, 0.3)), empty_frac=0.1) for _ in range(8)]
    masks = [ops.BlockMask.from_host(rp, ci, 1, H, n, block=128) for rp, ci in hm]
    V = ops.VisitMap(1, H, n, block=128)
    V.reset(masks[0])
    for m in masks[:-1]:
        V.update(m)
    last = V.refresh(masks[-1])
    V.update(last)
    torch.cuda.synchronize()
    used, Vref = fb.run_group([fb.dense_of(rp, ci, rows, nk) for rp, ci in hm], nk)
    rp, ci = last.to_host()
    erp, eci = fb.csr_of(used[-1])
    assert np.array_equal(rp, erp) and np.array_equal(ci, eci)
    assert np.array_equal(V.to_host(), Vref) and Vref.all()


def test_full_size_720p_fp8_kv128_sampled():
    """The 720p 14B workload with the paper's geometry (kv blocks of 128:
    591 per row, 1182 q-blocks): its builder mask on sampled heads and the fp8
    attention on sampled q-blocks against the oracle."""
    wl = wk.WORKLOADS["wan14b_720p_fp8"]
    inp = wk.make_inputs(wl)
    m = ops.build_block_mask(inp.mask_q.cuda(), inp.mask_k.cuda(), wl.top_p, wl.min_top_k,
                             sm_scale=wl.sm_scale, kv_block=128)
    rp, ci = m.to_host()
    n = wl.n_blocks
    heads = [0, wl.H - 1]
    o = om.build_block_mask(inp.mask_q.float().numpy(), inp.mask_k.float().numpy(), wl.sm_scale, wl.top_p,
                            wl.min_top_k, heads=heads, kv_block=128)
    rep = compare_masks(rp, ci, o, [h * n + i for h in heads for i in range(n)], wl.top_p, wl.min_top_k)
    assert rep.ok and not rep.failing, rep.failing[:3]
    (qc, qs), (kc, ks), (vc, vs) = (ops.quantize_fp8_blockwise(x.cuda()) for x in (inp.q, inp.k, inp.v))
    order = ops.plan_block_mask(m, wl.B, wl.S)
    out = ops.block_sparse_attn_fwd(qc, kc, vc, m, scales=(qs, ks, vs), sm_scale=wl.sm_scale, schedule=order)
    torch.cuda.synchronize()
    rng = np.random.Generator(np.random.PCG64(128))
    worst = 0.0
    for h in range(0, wl.H, 5):
        sl = lambda c, s: of.dequantize_blockwise(c[0:1, :, h:h + 1].cpu().numpy(),
                                                  s[0:1, h:h + 1].cpu().numpy())[0, :, 0]
        qh, kh, vh = sl(qc, qs), sl(kc, ks), sl(vc, vs)
        oh = np64(out[0, :, h].cpu())
        for i in sorted({0, n - 1} | set(rng.integers(0, n, 2).tolist())):
            r = oa.mask_row_index(0, h, i, wl.H, n, 1)
            o_ref, _ = oa.attention_block(qh, kh, vh, oa.row_blocks(rp, ci, r), i, wl.sm_scale, kv_block=128)
            worst = max(worst, max_abs_err(oh[i * 64:i * 64 + o_ref.shape[0]], o_ref))
    assert worst <= TOL8, worst
