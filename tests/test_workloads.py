"""Synthetic input generator: determinism, shapes, structure (CPU only)."""

import dataclasses

import numpy as np
import torch

from oracle import attention as oa
from oracle import mask as om
import workloads as wk


def small(key, **kw):
    wl = wk.WORKLOADS[key]
    return dataclasses.replace(wl, **kw)


def test_configs_shapes_and_blocks():
    want = {"tiny_f16": (1, 4096, 2, 64), "wan5b_720p_bf16": (1, 27280, 24, 427),
            "wan14b_480p_reuse_bf16": (1, 32760, 40, 512), "wan14b_720p_fp8": (1, 75600, 40, 1182),
            "wan14b_480p_batch4_bf16": (4, 32760, 40, 512)}
    for key, (B, S, H, n) in want.items():
        wl = wk.WORKLOADS[key]
        assert (wl.B, wl.S, wl.H, wl.n_blocks, wl.D) == (B, S, H, n, 128)
    assert [wk.WORKLOADS[k].S % 64 for k in wk.ORDER] == [0, 16, 56, 16, 56]


def test_generator_is_deterministic_and_typed():
    wl = wk.WORKLOADS["tiny_f16"]
    a = wk.make_inputs(wl)
    b = wk.make_inputs(wl)
    for x, y in ((a.q, b.q), (a.k, b.k), (a.v, b.v)):
        assert x.dtype == torch.float16 and x.shape == (1, 4096, 2, 128)
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))
    assert np.array_equal(a.random_mask[0], b.random_mask[0])
    assert np.array_equal(a.random_mask[1], b.random_mask[1])


def test_random_mask_structure():
    wl = wk.WORKLOADS["tiny_f16"]
    rp, ci = wk.random_mask(wl)
    n = wl.n_blocks
    assert rp.shape == (wl.H * n + 1,) and rp[-1] == wl.H * n * 16
    for r in range(wl.H * n):
        row = ci[rp[r]:rp[r + 1]]
        assert len(row) == 16 and np.all(np.diff(row) > 0) and (r % n) in row
        assert row.min() >= 0 and row.max() < n


def test_cross_request_perturbation_statistics():
    wl = small("wan14b_480p_batch4_bf16", grid=(2, 8, 16), H=3)
    inp = wk.make_inputs(wl)
    d = (inp.q[1] - inp.q[0]).float()
    # q_r - q_s = 0.3 (n_r - n_s): std 0.3 * sqrt(2)
    assert abs(d.std().item() - 0.3 * np.sqrt(2)) < 0.02
    assert torch.equal(inp.mask_q, inp.q[0:1])
    v01 = torch.corrcoef(torch.stack([inp.v[0].float().flatten(), inp.v[1].float().flatten()]))
    assert abs(v01[0, 1].item()) < 0.05
    wl2 = small("wan14b_480p_reuse_bf16", grid=(2, 8, 16), H=3)
    inp2 = wk.make_inputs(wl2)
    d2 = (inp2.q[0] - inp2.mask_q[0]).float()
    assert abs(d2.std().item() - 0.3) < 0.02


def test_heads_differ_in_sharpness():
    wl = small("wan5b_720p_bf16", grid=(4, 8, 16), H=4)
    inp = wk.make_inputs(wl, with_v=False)
    loc = [inp.q[0, :, h].float().std().item() for h in range(wl.H)]
    assert loc[-1] > loc[0]


def test_output_magnitude_fits_bf16_budget():
    # |O| < 0.5 keeps bf16 output rounding (2^-9 relative) well inside 2e-3.
    wl = wk.WORKLOADS["wan5b_720p_bf16"]
    inp = wk.make_inputs(wl)
    q = inp.q.float().numpy()
    k = inp.k.float().numpy()
    v = inp.v.float().numpy()
    n = wl.n_blocks
    for h in (0, wl.H - 1):
        s = om.block_scores(om.pool_means(q[0, :, h]), om.pool_means(k[0, :, h]), wl.sm_scale)
        for i in (0, n // 2, n - 1):
            sel = om.select_row(s[i], wl.top_p, wl.min_top_k)
            o, _ = oa.attention_block(q[0, :, h], k[0, :, h], v[0, :, h], sel, i, wl.sm_scale)
            assert np.abs(o).max() < 0.5


def test_similar_requests_reproduce_the_workload_recipe():
    """At sigma = 0.3 the swept generator gives exactly the workload's own
    historical and new requests."""
    small = wk.Workload("small_reuse", "bf16", 1, 3, (3, 8, 16), 0.2, "historical", 9100)
    inp = wk.make_inputs(small)
    bq, bk, reqs = wk.make_similar_requests(small, [0.3, 1.0])
    assert torch.equal(bq, inp.mask_q) and torch.equal(bk, inp.mask_k)
    assert torch.equal(reqs[0][0], inp.q) and torch.equal(reqs[0][1], inp.k)
    # larger sigma moves the request further from the base
    d03 = (reqs[0][0].float() - bq.float()).pow(2).mean().item()
    d10 = (reqs[1][0].float() - bq.float()).pow(2).mean().item()
    assert d10 > 5 * d03
    sub = wk.make_similar_requests(small, [0.3], heads=[2])
    assert torch.equal(sub[2][0][0][:, :, 0], inp.q[:, :, 2])
