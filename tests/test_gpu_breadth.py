"""GPU parity of the breadth items of the path (through the C ABI): the
mask builder on fp8 e4m3 input against the oracle on the dequantised codes,
and the f16 kernels at every full workload shape."""

import math

import numpy as np
import pytest
import torch

from oracle import fp8 as of
from oracle import guidance as og
from oracle import mask as om
from paper_2606_25040_amd import ops
import workloads as wk
from tests.compare import compare_masks

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def device():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    ops.load_library()
    torch.cuda.set_device(0)
    yield


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


# --------------------------------------------------------------------------- builder on fp8 input
@pytest.mark.parametrize("key_scale", [None, (700, 1.5)])
def test_builder_on_fp8_codes(key_scale):
    B, S, H = 2, 1500, 2
    q, k = positional(B, S, H, torch.bfloat16, 23)
    (qc, qs), (kc, ks) = (ops.quantize_fp8_blockwise(x.cuda()) for x in (q, k))
    top_p, mk = 0.7, 0.05
    sm = 1.0 / math.sqrt(128)
    m = ops.build_block_mask(qc, kc, top_p, mk, sm_scale=sm, scales=(qs, ks), key_scale=key_scale,
                             return_scores=True)
    rp, ci = m.to_host()
    dq = of.dequantize_blockwise(qc.cpu().numpy(), qs.cpu().numpy())
    dk = of.dequantize_blockwise(kc.cpu().numpy(), ks.cpu().numpy())
    if key_scale is not None:
        dk = og.enhance_first_frame_keys(dk, *key_scale)
    o = om.build_block_mask(dq, dk, sm, top_p, mk)
    rep = compare_masks(rp, ci, o, range(m.rows), top_p, mk)
    assert rep.ok and not rep.failing, rep.failing[:3]
    sc = m.block_scores.cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(sc, o.scores, rtol=1e-6, atol=1e-7)


def test_full_size_builder_on_fp8_codes_sampled_heads():
    """The 720p 14B workload's own Q/K quantised to fp8, the mask built from
    the codes: sampled heads against the oracle on the dequantised values."""
    wl = wk.WORKLOADS["wan14b_720p_fp8"]
    inp = wk.make_inputs(wl)
    (qc, qs), (kc, ks) = (ops.quantize_fp8_blockwise(x.cuda()) for x in (inp.mask_q, inp.mask_k))
    m = ops.build_block_mask(qc, kc, wl.top_p, wl.min_top_k, sm_scale=wl.sm_scale, scales=(qs, ks))
    rp, ci = m.to_host()
    heads = [0, wl.H // 2, wl.H - 1]
    sl = lambda c, s: of.dequantize_blockwise(c[:, :, heads].cpu().numpy(), s[:, heads].cpu().numpy())
    o = om.build_block_mask(sl(qc, qs), sl(kc, ks), wl.sm_scale, wl.top_p, wl.min_top_k)
    n = wl.n_blocks
    rows = [h * n + i for h in heads for i in range(n)]
    # the oracle ran on the three heads only: its row of head index t is t * n + i
    o_rows = {h * n + i: t * n + i for t, h in enumerate(heads) for i in range(n)}
    sub_rp = np.concatenate([[0], np.cumsum([rp[r + 1] - rp[r] for r in rows])])
    sub_ci = np.concatenate([ci[rp[r]:rp[r + 1]] for r in rows])
    rep = compare_masks(sub_rp, sub_ci, o, [o_rows[r] for r in rows], wl.top_p, wl.min_top_k)
    assert rep.ok and not rep.failing, rep.failing[:3]
    assert abs(m.density - wl.density) < 0.01


# --------------------------------------------------------------------------- f16 at the full shapes
def _max_err(a, b):
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))


@pytest.mark.parametrize("key", ["wan5b_720p_bf16", "wan14b_480p_reuse_bf16", "wan14b_720p_fp8",
                                 "wan14b_480p_batch4_bf16"])
def test_full_size_f16_builder_and_attention(key):
    """Every workload shape run in f16 (its inputs converted; the 720p 14B
    shape of the fp8 workload and the batch of four with its shared mask
    included): the builder on the sharpest and the most diffuse head, every
    row; the attention on every q-block of those heads of every request."""
    from oracle import attention as oa
    wl = wk.WORKLOADS[key]
    inp = wk.make_inputs(wl)
    q, k, v = (x.to(torch.float16) for x in (inp.q, inp.k, inp.v))
    mq, mk = (x.to(torch.float16) for x in (inp.mask_q, inp.mask_k))
    m = ops.build_block_mask(mq.cuda(), mk.cuda(), wl.top_p, wl.min_top_k, sm_scale=wl.sm_scale)
    rp, ci = m.to_host()
    heads = [0, wl.H - 1]
    o = om.build_block_mask(mq.double().numpy(), mk.double().numpy(), wl.sm_scale, wl.top_p, wl.min_top_k,
                            heads=heads)
    n = wl.n_blocks
    rep = compare_masks(rp, ci, o, [h * n + i for h in heads for i in range(n)], wl.top_p, wl.min_top_k)
    assert rep.ok and not rep.failing, rep.failing[:3]
    order = ops.plan_block_mask(m, wl.B, wl.S)
    out = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), m, sm_scale=wl.sm_scale, schedule=order)
    torch.cuda.synchronize()
    worst = 0.0
    for b in range(wl.B):
        for h in heads:
            qh, kh, vh = (x[b, :, h].double().numpy() for x in (q, k, v))
            oh = out[b, :, h].double().cpu().numpy()
            for i in range(n):
                r = oa.mask_row_index(b, h, i, wl.H, n, 1)
                o_ref, _ = oa.attention_block(qh, kh, vh, oa.row_blocks(rp, ci, r), i, wl.sm_scale)
                worst = max(worst, _max_err(oh[i * 64:i * 64 + o_ref.shape[0]], o_ref))
    assert worst <= 2e-3, worst
