"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Small cases compare every output; the full-size workloads compare sampled
rows and work items the oracle computes one by one.  Tolerances: masks
bit-exact apart from excused near-ties (tests/compare.py); outputs max-abs
2e-3 for f16/bf16 and 3e-2 for fp8; fp8 codes and scales bit-exact.
"""

import math

import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import fp8 as of
from oracle import guidance as og
from oracle import mask as om
from paper_2606_25040_amd import ops
import workloads as wk
from tests.compare import compare_masks, max_abs_err

pytestmark = pytest.mark.gpu

TOL16 = 2e-3
TOL8 = 3e-2


@pytest.fixture(scope="module", autouse=True)
def device():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    ops.load_library()
    torch.cuda.set_device(0)
    yield


def np64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy()


def rand_qkv(gen, B, S, H, dtype, scale=0.5):
    """Random Q, K (logit std ~ scale^2) and V ~ N(0, 1).  The default keeps
    attention diffuse like the workloads (|O| < 0.5), where the 16-bit output
    rounding stays inside the absolute tolerance; peaked cases use
    ``within_rounding`` instead."""
    q = (torch.randn(B, S, H, 128, generator=gen) * scale).to(dtype)
    k = (torch.randn(B, S, H, 128, generator=gen) * scale).to(dtype)
    v = torch.randn(B, S, H, 128, generator=gen).to(dtype)
    return q, k, v


def positional_qk(B, S, H, dtype, seed):
    """Block-structured Q/K (shared positional projection) for builder tests."""
    g = np.random.Generator(np.random.PCG64(seed))
    f = np.stack([np.sin(2 * np.pi * np.arange(S) / P) for P in (37.0, 200.0, 911.0, 3000.0)] +
                 [np.cos(2 * np.pi * np.arange(S) / P) for P in (37.0, 200.0, 911.0, 3000.0)], 1)
    q = np.empty((B, S, H, 128), np.float32)
    k = np.empty((B, S, H, 128), np.float32)
    for h in range(H):
        W = g.standard_normal((8, 128)) * 0.5
        for b in range(B):
            q[b, :, h] = f @ W + 0.5 * g.standard_normal((S, 128))
            k[b, :, h] = f @ W + 0.5 * g.standard_normal((S, 128))
    return torch.from_numpy(q).to(dtype), torch.from_numpy(k).to(dtype)


def within_rounding(got, ref, dtype, atol=TOL16, ref_abs=None):
    """Error bound for cases far from the workloads' diffuse regime: the
    absolute tolerance plus one unit of the 16-bit type's relative rounding
    on the output (|O|) and on the probabilities (sum_c p_c |v_c|, passed as
    ``ref_abs`` = attention applied to |V|)."""
    rel = 2.0 ** -8 if dtype == torch.bfloat16 else 2.0 ** -10
    bound = atol + rel * np.abs(ref)
    if ref_abs is not None:
        bound = bound + rel * ref_abs
    return bool(np.all(np.abs(got - ref) <= bound))


# --------------------------------------------------------------------------- quantiser
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
def test_quantizer_bit_exact(dtype):
    gen = torch.Generator().manual_seed(11)
    B, S, H = 2, 1000, 3
    x = torch.randn(B, S, H, 128, generator=gen) * torch.tensor([0.01, 1.0, 30.0]).view(1, 1, 3, 1)
    x[0, 64:128, 1] = 0.0                                  # amax == 0 block
    x[1, 128:192, 0] = -0.0
    x[1, 192:256, 2] *= 1e-3                               # values deep in the subnormal range
    x[0, 960:, 2] = 1e4 if dtype == torch.bfloat16 else 6e4
    if dtype == torch.bfloat16:
        # amax below 448 / FLT_MAX (the reciprocal is taken after a 2^64
        # pre-scale), with fp32-subnormal inputs and a subnormal scale
        x[1, 320:384, 1] *= 2.0 ** -123
    x = x.to(dtype)
    codes, scales = ops.quantize_fp8_blockwise(x.cuda())
    torch.cuda.synchronize()
    oc, os_ = of.quantize_blockwise(np64(x))
    assert np.array_equal(codes.cpu().numpy(), oc)
    assert np.array_equal(scales.cpu().numpy(), os_)


# --------------------------------------------------------------------------- builder
BUILD_CASES = [(0.5, 0.05), (0.9, 0.0), (0.0, 0.3), (1.0, 0.0), (0.3, 1.0), (0.75, 0.1)]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
def test_builder_small_all_rows(dtype):
    B, S, H = 2, 1000, 3                                    # 16 blocks, last one 40 tokens
    q, k = positional_qk(B, S, H, dtype, 5)
    qd, kd = q.cuda(), k.cuda()
    sm = 1.0 / math.sqrt(128)
    for top_p, mk in BUILD_CASES:
        m = ops.build_block_mask(qd, kd, top_p, mk, sm_scale=sm, return_scores=True)
        rp, ci = m.to_host()
        o = om.build_block_mask(np64(q), np64(k), sm, top_p, mk)
        rep = compare_masks(rp, ci, o, range(m.rows), top_p, mk)
        assert rep.ok, rep.failing[:5]
        assert ops.validate_block_mask(m) == 0
        s32 = m.block_scores.cpu().numpy()
        assert np.array_equal(s32, o.scores.astype(np.float32)) or \
            np.max(np.abs(s32 - o.scores) / (np.abs(o.scores) + 1e-30)) < 1.2e-7


def test_builder_single_block_and_tiny_sequences():
    sm = 1.0 / math.sqrt(128)
    for S in (1, 63, 64, 65, 130):
        q, k = positional_qk(1, S, 2, torch.bfloat16, S)
        m = ops.build_block_mask(q.cuda(), k.cuda(), 0.6, 0.0, sm_scale=sm)
        rp, ci = m.to_host()
        o = om.build_block_mask(np64(q), np64(k), sm, 0.6, 0.0)
        rep = compare_masks(rp, ci, o, range(m.rows), 0.6, 0.0)
        assert rep.ok, (S, rep.failing[:3])


@pytest.mark.parametrize("top_p,mk", [(0.5, 0.0), (0.3, 0.4), (0.0, 0.25), (0.97, 0.0)])
def test_builder_exact_ties(top_p, mk):
    """Bit-identical block scores: constant Q/K (every score of a row equal)
    and K whose blocks repeat with period 4 (four-way ties per row).  Equal
    scores are kept lowest index first."""
    sm = 1.0 / math.sqrt(128)
    S, H = 64 * 20, 2
    const = torch.full((1, S, H, 128), 0.25, dtype=torch.bfloat16)
    gen = torch.Generator().manual_seed(3)
    q = (torch.randn(1, S, H, 128, generator=gen) * 0.5).to(torch.bfloat16)
    base = (torch.randn(1, 4 * 64, H, 128, generator=gen) * 0.5).to(torch.bfloat16)
    k_rep = base.repeat(1, S // (4 * 64), 1, 1).contiguous()
    for qq, kk in ((const, const), (q, k_rep)):
        m = ops.build_block_mask(qq.cuda(), kk.cuda(), top_p, mk, sm_scale=sm)
        rp, ci = m.to_host()
        o = om.build_block_mask(np64(qq), np64(kk), sm, top_p, mk)
        rep = compare_masks(rp, ci, o, range(m.rows), top_p, mk)
        assert rep.ok, rep.failing[:3]
    # constant rows keep a prefix of indices: k = 10 of 20 in exact arithmetic
    # (the float64 running sum of ten 1/20 lands one ulp below 0.5, hence 11
    # is accepted too; the comparator above excuses that boundary)
    m = ops.build_block_mask(const.cuda(), const.cuda(), 0.5, 0.0, sm_scale=sm)
    rp, ci = m.to_host()
    for r in range(m.rows):
        row = ci[rp[r]:rp[r + 1]]
        assert len(row) in (10, 11) and np.array_equal(row, np.arange(len(row)))


@pytest.mark.parametrize("n_blocks", [511, 700, 1500, 2000])
def test_builder_row_lengths_every_selection_path(n_blocks):
    """Rows of 511, 700, 1500 and 2000 blocks (each register budget of the
    one-wave-per-row selection), every row against the oracle."""
    sm = 1.0 / math.sqrt(128)
    S = 64 * n_blocks - 13
    q, k = positional_qk(1, S, 1, torch.bfloat16, n_blocks)
    for top_p, mk in ((0.45, 0.02), (0.0, 0.07), (0.9, 0.0)):
        m = ops.build_block_mask(q.cuda(), k.cuda(), top_p, mk, sm_scale=sm)
        rp, ci = m.to_host()
        o = om.build_block_mask(np64(q), np64(k), sm, top_p, mk)
        rep = compare_masks(rp, ci, o, range(m.rows), top_p, mk)
        assert rep.ok, (n_blocks, top_p, mk, rep.failing[:3])


def test_builder_largest_supported_row():
    """n = 4096 blocks (the largest row): every row against the oracle."""
    sm = 1.0 / math.sqrt(128)
    S = 64 * 4096 - 7
    q, k = positional_qk(1, S, 1, torch.bfloat16, 21)
    for top_p, mk in ((0.4, 0.01), (0.0, 0.1)):
        m = ops.build_block_mask(q.cuda(), k.cuda(), top_p, mk, sm_scale=sm)
        rp, ci = m.to_host()
        o = om.build_block_mask(np64(q), np64(k), sm, top_p, mk)
        rep = compare_masks(rp, ci, o, range(m.rows), top_p, mk)
        assert rep.ok, rep.failing[:3]


# --------------------------------------------------------------------------- attention
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
def test_attention_peaked_logits(dtype):
    gen = torch.Generator().manual_seed(77)
    B, S, H = 1, 700, 2
    q, k, v = rand_qkv(gen, B, S, H, dtype, scale=1.6)      # logit std ~ 2.6
    n = (S + 63) // 64
    rng = np.random.Generator(np.random.PCG64(77))
    rp, ci = wk.random_csr(rng, H * n, n, 0.5)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n)
    out = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), mask)
    O, _ = oa.attention(np64(q), np64(k), np64(v), rp, ci, 1.0 / math.sqrt(128), 1)
    Oabs, _ = oa.attention(np64(q), np64(k), np.abs(np64(v)), rp, ci, 1.0 / math.sqrt(128), 1)
    assert within_rounding(np64(out), O, dtype, ref_abs=Oabs)


def attn_ref_full(q, k, v, rp, ci, mask_batch, sm):
    return oa.attention(np64(q), np64(k), np64(v), rp, ci, sm, mask_batch)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
@pytest.mark.parametrize("S,B,H,mask_batch", [(64, 1, 1, 1), (100, 2, 2, 1), (1000, 2, 3, 2),
                                              (1000, 2, 3, 1), (2048, 1, 2, 1)])
def test_attention_small_full(dtype, S, B, H, mask_batch):
    gen = torch.Generator().manual_seed(S + 7 * B + H)
    q, k, v = rand_qkv(gen, B, S, H, dtype)
    n = (S + 63) // 64
    rng = np.random.Generator(np.random.PCG64(S))
    rp, ci = wk.random_csr(rng, mask_batch * H * n, n, 0.4, empty_frac=0.1 if n > 1 else 0.0)
    mask = ops.BlockMask.from_host(rp, ci, mask_batch, H, n)
    sm = 1.0 / math.sqrt(128)
    out, lse = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), mask, sm_scale=sm,
                                         return_lse=True)
    torch.cuda.synchronize()
    O, L = attn_ref_full(q, k, v, rp, ci, mask_batch, sm)
    # few keys per row here, so |O| reaches ~0.7: allow the output rounding on top
    assert within_rounding(np64(out), O, dtype)
    lg = lse.cpu().numpy()
    fin = np.isfinite(L)
    assert np.array_equal(np.isfinite(lg), fin)
    if fin.any():
        assert np.max(np.abs(lg[fin] - L[fin])) <= 1e-3
    # empty rows are exactly zero
    counts = np.diff(rp)
    for b in range(B):
        for h in range(H):
            for i in range(n):
                r = oa.mask_row_index(b, h, i, H, n, mask_batch)
                if counts[r] == 0:
                    assert torch.all(out[b, i * 64:(i + 1) * 64, h] == 0)


def test_attention_full_density_equals_dense_sdpa():
    gen = torch.Generator().manual_seed(3)
    B, S, H = 1, 777, 2
    q, k, v = rand_qkv(gen, B, S, H, torch.bfloat16)
    n = (S + 63) // 64
    rp = np.arange(H * n + 1) * n
    ci = np.tile(np.arange(n), H * n)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n)
    out = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), mask)
    ref = torch.nn.functional.scaled_dot_product_attention(
        q.double().permute(0, 2, 1, 3), k.double().permute(0, 2, 1, 3),
        v.double().permute(0, 2, 1, 3)).permute(0, 2, 1, 3)
    assert within_rounding(np64(out), ref.numpy(), torch.bfloat16)


@pytest.mark.parametrize("dtype", ["bf16", "f16", "fp8"])
@pytest.mark.parametrize("key_scale", [None, (400, 1.5)])
def test_attention_without_mask_is_the_full_density_mask(dtype, key_scale):
    """mask = NULL (every kv block, the dense instantiations) gives bitwise the
    output of an explicit full-density mask, and that matches the oracle."""
    gen = torch.Generator().manual_seed(5)
    B, S, H = 2, 700, 2
    tdt = torch.float16 if dtype == "f16" else torch.bfloat16
    q, k, v = rand_qkv(gen, B, S, H, tdt)
    n = (S + 63) // 64
    rp = np.arange(H * n + 1) * n
    ci = np.tile(np.arange(n), H * n)
    full = ops.BlockMask.from_host(rp, ci, 1, H, n)
    if dtype == "fp8":
        cs = [ops.quantize_fp8_blockwise(x.cuda()) for x in (q, k, v)]
        args, kw = [c for c, _ in cs], {"scales": tuple(s_ for _, s_ in cs)}
        ins = [of.dequantize_blockwise(c.cpu().numpy(), s_.cpu().numpy()) for c, s_ in cs]
        tol = TOL8
    else:
        args, kw = [x.cuda() for x in (q, k, v)], {}
        ins = [np64(x) for x in (q, k, v)]
        tol = TOL16
    dense = ops.block_sparse_attn_fwd(*args, None, key_scale=key_scale, **kw)
    listed = ops.block_sparse_attn_fwd(*args, full, key_scale=key_scale, **kw)
    torch.cuda.synchronize()
    assert torch.equal(dense.view(torch.int16), listed.view(torch.int16))
    kk = ins[1] if key_scale is None else og.enhance_first_frame_keys(ins[1], *key_scale)
    O, _ = oa.attention(ins[0], kk, ins[2], rp, ci, 1.0 / math.sqrt(128), 1)
    assert within_rounding(np64(dense), O, tdt, atol=tol), float(np.max(np.abs(np64(dense) - O)))


def test_attention_strided_views_and_determinism():
    gen = torch.Generator().manual_seed(9)
    B, S, H = 2, 500, 2
    qkv = torch.randn(B, S, 3, H, 128, generator=gen).to(torch.bfloat16).cuda()
    q, k, v = qkv[:, :, 0], qkv[:, :, 1], qkv[:, :, 2]
    n = (S + 63) // 64
    rng = np.random.Generator(np.random.PCG64(1))
    rp, ci = wk.random_csr(rng, H * n, n, 0.5)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n)
    o1 = ops.block_sparse_attn_fwd(q, k, v, mask)
    o2 = ops.block_sparse_attn_fwd(q, k, v, mask)
    order = ops.plan_block_mask(mask, B, S)
    o3 = ops.block_sparse_attn_fwd(q, k, v, mask, schedule=order)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(o1.view(torch.int16), o3.view(torch.int16))
    assert sorted(order.cpu().tolist()) == list(range(B * H))
    O, _ = oa.attention(np64(q.cpu()), np64(k.cpu()), np64(v.cpu()), rp, ci,
                        1.0 / math.sqrt(128), 1)
    assert within_rounding(np64(o1), O, torch.bfloat16)


def greedy_plan(rp, B, H, n, mask_batch, xcds=8):
    """The plan rule restated in plain Python: unit cost = listed blocks +
    q-blocks; heaviest first (ties by id) to the least-loaded XCD with room
    (lowest XCD id on equal load); units listed XCD by XCD, ascending id."""
    U = B * H
    cost = []
    for u in range(U):
        b, h = divmod(u, H)
        r0 = ((b if mask_batch > 1 else 0) * H + h) * n
        cost.append(int(rp[r0 + n] - rp[r0]) + n)
    cap = [U // xcds + (1 if x < U % xcds else 0) for x in range(xcds)]
    load, used, where = [0] * xcds, [0] * xcds, [0] * U
    for u in sorted(range(U), key=lambda u: (-cost[u], u)):
        best = min((x for x in range(xcds) if used[x] < cap[x]), key=lambda x: (load[x], x))
        load[best] += cost[u]
        used[best] += 1
        where[u] = best
    return [u for x in range(xcds) for u in range(U) if where[u] == x]


@pytest.mark.parametrize("B,H,mask_batch", [(1, 24, 1), (4, 40, 1), (3, 7, 3), (1, 1, 1), (2, 600, 2)])
def test_plan_follows_greedy_rule(B, H, mask_batch):
    n = 9
    rng = np.random.Generator(np.random.PCG64(B * 1000 + H))
    rows = mask_batch * H * n
    counts = rng.integers(1, n + 1, size=rows)
    rp = np.zeros(rows + 1, np.int64)
    np.cumsum(counts, out=rp[1:])
    ci = np.concatenate([np.sort(rng.choice(n, c, replace=False)) for c in counts])
    mask = ops.BlockMask.from_host(rp, ci, mask_batch, H, n)
    order = ops.plan_block_mask(mask, B, 64 * n).cpu().tolist()
    assert order == greedy_plan(rp, B, H, n, mask_batch)


@pytest.mark.parametrize("B,H", [(1, 24), (2, 13), (1, 5)])
def test_plan_equal_costs_follow_the_tie_rules(B, H):
    # every unit lists every block: all costs equal, so only the tie rules
    # (units by id, XCDs by id on equal load) decide the order
    n = 6
    rows = H * n
    rp = np.arange(0, rows * n + 1, n, dtype=np.int64)
    ci = np.tile(np.arange(n), rows)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n)
    order = ops.plan_block_mask(mask, B, 64 * n).cpu().tolist()
    assert order == greedy_plan(rp, B, H, n, 1)
    assert sorted(order) == list(range(B * H))


def test_attention_fp8_small_full():
    gen = torch.Generator().manual_seed(21)
    B, S, H = 2, 1000, 3
    q, k, v = rand_qkv(gen, B, S, H, torch.bfloat16)
    n = (S + 63) // 64
    rng = np.random.Generator(np.random.PCG64(2))
    rp, ci = wk.random_csr(rng, H * n, n, 0.5, empty_frac=0.05)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n)
    qc, qs = ops.quantize_fp8_blockwise(q.cuda())
    kc, ks = ops.quantize_fp8_blockwise(k.cuda())
    vc, vs = ops.quantize_fp8_blockwise(v.cuda())
    out, lse = ops.block_sparse_attn_fwd(qc, kc, vc, mask, scales=(qs, ks, vs), return_lse=True)
    torch.cuda.synchronize()
    dq = of.dequantize_blockwise(qc.cpu().numpy(), qs.cpu().numpy())
    dk = of.dequantize_blockwise(kc.cpu().numpy(), ks.cpu().numpy())
    dv = of.dequantize_blockwise(vc.cpu().numpy(), vs.cpu().numpy())
    O, L = oa.attention(dq, dk, dv, rp, ci, 1.0 / math.sqrt(128), 1)
    assert within_rounding(np64(out), O, torch.bfloat16, atol=TOL8)
    lg = lse.cpu().numpy()
    fin = np.isfinite(L)
    assert np.array_equal(np.isfinite(lg), fin)
    if fin.any():
        assert np.max(np.abs(lg[fin] - L[fin])) <= 1e-3


@pytest.mark.parametrize("kind", ["bf16", "f16", "fp8"])
def test_attention_skips_out_of_range_ids(kind):
    """Ids outside [0, n) in a mask row are skipped (the contract in
    include/chorus.h): rows with -1 ahead of their ids, or n and n + 5 after
    them, give the output of the same rows without those ids, also where a
    row holds nothing else.  Each q-block's kv walk starts at a rotated
    position of its row, which has to land on the valid ids of such rows."""
    gen = torch.Generator().manual_seed(5)
    B, S, H = 1, 1000, 3
    q, k, v = rand_qkv(gen, B, S, H, torch.float16 if kind == "f16" else torch.bfloat16)
    n = (S + 63) // 64
    rng = np.random.Generator(np.random.PCG64(11))
    rp, ci = wk.random_csr(rng, H * n, n, 0.4, empty_frac=0.1)
    rows = []
    for r in range(H * n):
        ids = [int(j) for j in ci[rp[r]:rp[r + 1]]]
        if r % 3 == 0:
            ids = [-1] + ids
        elif r % 3 == 1:
            ids = ids + [n, n + 5]
        rows.append(ids)
    assert any(len(x) == 1 and x[0] == -1 for x in rows)   # a row of invalid ids only
    rp2 = np.concatenate([[0], np.cumsum([len(x) for x in rows])])
    ci2 = np.array([j for x in rows for j in x], dtype=np.int64)
    mask = ops.BlockMask.from_host(rp2, ci2, 1, H, n)
    sm = 1.0 / math.sqrt(128)
    if kind == "fp8":
        (qc, qs), (kc, ks), (vc, vs) = (ops.quantize_fp8_blockwise(x.cuda()) for x in (q, k, v))
        out, lse = ops.block_sparse_attn_fwd(qc, kc, vc, mask, scales=(qs, ks, vs), sm_scale=sm,
                                             return_lse=True)
        deq = [of.dequantize_blockwise(c.cpu().numpy(), s_.cpu().numpy())
               for c, s_ in ((qc, qs), (kc, ks), (vc, vs))]
        O, L = oa.attention(*deq, rp, ci, sm, 1)
        atol = TOL8
    else:
        out, lse = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), mask, sm_scale=sm,
                                             return_lse=True)
        O, L = attn_ref_full(q, k, v, rp, ci, 1, sm)
        atol = TOL16
    torch.cuda.synchronize()
    assert within_rounding(np64(out), O, torch.float16 if kind == "f16" else torch.bfloat16, atol=atol)
    lg = lse.cpu().numpy()
    fin = np.isfinite(L)
    assert np.array_equal(np.isfinite(lg), fin)
    assert np.max(np.abs(lg[fin] - L[fin])) <= 1e-3


def test_attention_fp8_extreme_value_block_scales():
    """V blocks whose fp8 scale is zero-input (scale 1), denormal (values of
    order 1e-37) or large sit next to ordinary blocks in the same rows: the
    per-block V scale folded into the exponent stays finite and the output
    matches the oracle on the dequantised inputs."""
    gen = torch.Generator().manual_seed(33)
    B, S, H = 1, 640, 2
    q, k, v = rand_qkv(gen, B, S, H, torch.bfloat16)
    n = S // 64
    v = v.float()
    v[:, 64:128] = 0.0                      # all-zero block: scale 1, codes 0
    v[:, 192:256] *= 1e-36                  # subnormal block scale (amax / 448 < FLT_MIN)
    v[:, 448:512] *= 2.0 ** -123            # amax below 448 / FLT_MAX
    v[:, 320:384] *= 3e3                    # large block next to unit ones
    v = v.to(torch.bfloat16)
    rp = np.arange(0, H * n * n + 1, n)
    ci = np.tile(np.arange(n), H * n)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n)
    (qc, qs), (kc, ks), (vc, vs) = (ops.quantize_fp8_blockwise(x.cuda()) for x in (q, k, v))
    assert float(vs[0, 0, 3].item()) < 1.17549435e-38   # the denormal case is present
    out = ops.block_sparse_attn_fwd(qc, kc, vc, mask, scales=(qs, ks, vs))
    torch.cuda.synchronize()
    got = np64(out)
    assert np.all(np.isfinite(got))
    deq = [of.dequantize_blockwise(c.cpu().numpy(), s_.cpu().numpy()) for c, s_ in ((qc, qs), (kc, ks), (vc, vs))]
    O, _ = oa.attention(*deq, rp, ci, 1.0 / math.sqrt(128), 1)
    # fp8 P~ (relative 2^-4 per weight) on values up to 3e3 in magnitude
    Oabs, _ = oa.attention(deq[0], deq[1], np.abs(deq[2]), rp, ci, 1.0 / math.sqrt(128), 1)
    bound = np.maximum(TOL8, 1e-3 + 2.0 ** -4 * Oabs) + 2.0 ** -8 * np.abs(O)
    assert np.all(np.abs(got - O) <= bound), float(np.max(np.abs(got - O) - bound))


# --------------------------------------------------------------------------- mask checker
def test_validate_flags():
    H, n = 2, 5
    good_rp = np.array([0, 2, 3, 3, 5, 6, 8, 9, 9, 10, 12])
    good_ci = np.array([0, 3, 1, 2, 4, 0, 1, 2, 3, 0, 1, 4])
    assert ops.validate_block_mask(ops.BlockMask.from_host(good_rp, good_ci, 1, H, n)) == 0
    bad = good_ci.copy()
    bad[1] = 0                                              # not ascending
    assert ops.validate_block_mask(ops.BlockMask.from_host(good_rp, bad, 1, H, n)) & 8
    bad = good_ci.copy()
    bad[4] = 5                                              # out of range
    assert ops.validate_block_mask(ops.BlockMask.from_host(good_rp, bad, 1, H, n)) & 4
    rp = good_rp.copy()
    rp[3] = 1                                               # decreasing
    assert ops.validate_block_mask(ops.BlockMask.from_host(rp, good_ci, 1, H, n)) & 2


def test_abi_rejects_bad_arguments_on_device():
    q = torch.zeros(2, 100, 2, 128, dtype=torch.bfloat16, device="cuda")
    n = 2
    mask = ops.BlockMask.from_host(np.arange(3 * 2 * n + 1), np.zeros(3 * 2 * n), 3, 2, n)
    with pytest.raises(RuntimeError, match="INVALID_ARG"):
        ops.block_sparse_attn_fwd(q, q, q, mask)
    with pytest.raises(RuntimeError, match="INVALID_ARG"):
        ops.build_block_mask(q, q, 1.5, 0.0)


# --------------------------------------------------------------------------- full-size workloads
_cache = {}


def workload_state(key):
    if key in _cache:
        return _cache[key]
    _cache.clear()
    torch.cuda.empty_cache()
    wl = wk.WORKLOADS[key]
    inp = wk.make_inputs(wl)
    st = {"wl": wl, "inp": inp}
    q, k, v = inp.q.cuda(), inp.k.cuda(), inp.v.cuda()
    mq, mk = inp.mask_q.cuda(), inp.mask_k.cuda()
    mask = ops.build_block_mask(mq, mk, wl.top_p, wl.min_top_k, sm_scale=wl.sm_scale)
    st.update(q=q, k=k, v=v, mask=mask)
    if wl.dtype == "fp8":
        st["q8"] = ops.quantize_fp8_blockwise(q)
        st["k8"] = ops.quantize_fp8_blockwise(k)
        st["v8"] = ops.quantize_fp8_blockwise(v)
    torch.cuda.synchronize()
    _cache[key] = st
    return st


FULL = ["wan5b_720p_bf16", "wan14b_480p_reuse_bf16", "wan14b_720p_fp8", "wan14b_480p_batch4_bf16"]


@pytest.mark.parametrize("key", FULL)
def test_full_size_mask_sampled_heads(key):
    st = workload_state(key)
    wl, inp, mask = st["wl"], st["inp"], st["mask"]
    rp, ci = mask.to_host()
    heads = sorted({0, wl.H // 2, wl.H - 1})
    o = om.build_block_mask(inp.mask_q.float().numpy(), inp.mask_k.float().numpy(), wl.sm_scale,
                            wl.top_p, wl.min_top_k, heads=heads)
    n = wl.n_blocks
    rows = [h * n + i for h in heads for i in range(n)]
    rep = compare_masks(rp, ci, o, rows, wl.top_p, wl.min_top_k)
    assert rep.ok, rep.failing[:5]
    assert abs(mask.density - wl.density) < 0.01
    assert ops.validate_block_mask(mask) == 0


def _check_heads(wl, out, lse, rp, ci, ins, heads, tol):
    """Every q-block (the partial last one included) of the listed heads of
    every request against the oracle, outputs and LSE.  ``ins(b, h)`` gives
    the float64 [S, D] q, k, v of (b, h) exactly as the kernel read them."""
    n = wl.n_blocks
    worst = worst_lse = 0.0
    for b in range(wl.B):
        for h in heads:
            qh, kh, vh = ins(b, h)
            oh = np64(out[b, :, h].cpu())
            lh = lse[b, h].cpu().numpy().astype(np.float64)
            for i in range(n):
                r = oa.mask_row_index(b, h, i, wl.H, n, 1)
                o_ref, l_ref = oa.attention_block(qh, kh, vh, oa.row_blocks(rp, ci, r), i, wl.sm_scale)
                rows = slice(i * 64, i * 64 + o_ref.shape[0])
                worst = max(worst, max_abs_err(oh[rows], o_ref))
                worst_lse = max(worst_lse, max_abs_err(lh[rows], l_ref))
    assert worst <= tol, worst
    assert worst_lse <= 1e-3, worst_lse
    return worst


@pytest.mark.parametrize("key", FULL)
def test_full_size_attention_every_q_block_of_two_heads(key):
    """Full-size launch (planned XCD order, as the benchmark runs it): every
    q-block of the sharpest and the most diffuse head of every request
    against the oracle; the unplanned order gives bitwise the same output."""
    st = workload_state(key)
    wl, mask = st["wl"], st["mask"]
    rp, ci = mask.to_host()
    order = ops.plan_block_mask(mask, wl.B, wl.S)
    if wl.dtype == "fp8":
        (qc, qs), (kc, ks), (vc, vs) = st["q8"], st["k8"], st["v8"]
        out, lse = ops.block_sparse_attn_fwd(qc, kc, vc, mask, scales=(qs, ks, vs), schedule=order,
                                             return_lse=True)
        out2 = ops.block_sparse_attn_fwd(qc, kc, vc, mask, scales=(qs, ks, vs))
        tol = TOL8

        def ins(b, h):
            sl = lambda c, s: of.dequantize_blockwise(c[b:b + 1, :, h:h + 1].cpu().numpy(),
                                                      s[b:b + 1, h:h + 1].cpu().numpy())[0, :, 0]
            return sl(qc, qs), sl(kc, ks), sl(vc, vs)
    else:
        out, lse = ops.block_sparse_attn_fwd(st["q"], st["k"], st["v"], mask, schedule=order,
                                             return_lse=True)
        out2 = ops.block_sparse_attn_fwd(st["q"], st["k"], st["v"], mask)
        tol = TOL16

        def ins(b, h):
            return tuple(np64(x[b, :, h].cpu()).astype(np.float64) for x in (st["q"], st["k"], st["v"]))
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16))
    _check_heads(wl, out, lse, rp, ci, ins, (0, wl.H - 1), tol)


def test_plan_beyond_4096_units_keeps_natural_order_and_results():
    """B * H > 4096 units: the plan keeps the natural order; any order gives
    bitwise the same attention output."""
    B, H, S = 65, 64, 64
    n = 1
    rng = np.random.Generator(np.random.PCG64(4097))
    rp = np.arange(B * H * n + 1, dtype=np.int64)
    ci = np.zeros(B * H * n, dtype=np.int64)
    mask = ops.BlockMask.from_host(rp, ci, B, H, n)
    order = ops.plan_block_mask(mask, B, S)
    assert order.cpu().tolist() == list(range(B * H))
    gen = torch.Generator().manual_seed(2)
    q, k, v = rand_qkv(gen, B, S, H, torch.bfloat16)
    q, k, v = q.cuda(), k.cuda(), v.cuda()
    ref = ops.block_sparse_attn_fwd(q, k, v, mask)
    perm = torch.from_numpy(rng.permutation(B * H).astype(np.int32)).cuda()
    out = ops.block_sparse_attn_fwd(q, k, v, mask, schedule=perm)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))


def test_tiny_f16_workload_every_element():
    """The tiny f16 check (B 1, H 2, S 4096 on a 4 x 32 x 32 grid, fixed
    random 25 % mask with the diagonal kept) through the C ABI: every output
    element and every LSE against the oracle's literal form (64 x S logits per
    q-block, unlisted blocks at -inf), plain and planned launch order."""
    wl = wk.WORKLOADS["tiny_f16"]
    inp = wk.make_inputs(wl)
    rp, ci = inp.random_mask
    mask = ops.BlockMask.from_host(rp, ci, 1, wl.H, wl.n_blocks)
    q, k, v = inp.q.cuda(), inp.k.cuda(), inp.v.cuda()
    out, lse = ops.block_sparse_attn_fwd(q, k, v, mask, sm_scale=wl.sm_scale, return_lse=True)
    order = ops.plan_block_mask(mask, wl.B, wl.S)
    out2 = ops.block_sparse_attn_fwd(q, k, v, mask, sm_scale=wl.sm_scale, schedule=order)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16))
    O, L = oa.attention(np64(inp.q), np64(inp.k), np64(inp.v), rp, ci, wl.sm_scale, 1, form="literal")
    assert max_abs_err(np64(out), O) <= TOL16
    assert max_abs_err(lse.cpu().numpy(), L) <= 1e-3


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("B,H", [(1, 13), (3, 3), (1, 1)])
def test_planned_order_with_units_not_a_multiple_of_eight(dtype, B, H):
    """B * H (request, head) units not a multiple of the 8 XCDs: each XCD
    walks exactly the units the plan gave it; any order gives bitwise the
    same output, and it matches the oracle."""
    gen = torch.Generator().manual_seed(B * 100 + H)
    S = 700
    q, k, v = rand_qkv(gen, B, S, H, torch.bfloat16)
    n = (S + 63) // 64
    rng = np.random.Generator(np.random.PCG64(B * 7 + H))
    rp, ci = wk.random_csr(rng, H * n, n, 0.4)
    mask = ops.BlockMask.from_host(rp, ci, 1, H, n)
    order = ops.plan_block_mask(mask, B, S)
    assert sorted(order.cpu().tolist()) == list(range(B * H))
    if dtype == "fp8":
        cs = [ops.quantize_fp8_blockwise(x.cuda()) for x in (q, k, v)]
        args, kw = [c for c, _ in cs], {"scales": tuple(s_ for _, s_ in cs)}
        ins = [of.dequantize_blockwise(c.cpu().numpy(), s_.cpu().numpy()) for c, s_ in cs]
        tol = TOL8
    else:
        args, kw = [x.cuda() for x in (q, k, v)], {}
        ins = [np64(x) for x in (q, k, v)]
        tol = TOL16
    natural = ops.block_sparse_attn_fwd(*args, mask, **kw)
    planned = ops.block_sparse_attn_fwd(*args, mask, schedule=order, **kw)
    perm = torch.from_numpy(rng.permutation(B * H).astype(np.int32)).cuda()
    shuffled = ops.block_sparse_attn_fwd(*args, mask, schedule=perm, **kw)
    torch.cuda.synchronize()
    assert torch.equal(natural.view(torch.int16), planned.view(torch.int16))
    assert torch.equal(natural.view(torch.int16), shuffled.view(torch.int16))
    O, _ = oa.attention(*ins, rp, ci, 1.0 / math.sqrt(128), 1)
    assert within_rounding(np64(natural), O, torch.bfloat16, atol=tol)
