"""The builder entry point that allocates nothing, through the C ABI, against
the workspace builder (chorus_build_block_mask): bitwise the same row_ptr,
col_idx and fp32 block scores, on two calls in a row, the second on a
smaller input, so the fixed scratch is reused with the first call's contents
still in it."""

import dataclasses

import numpy as np
import pytest
import torch

from paper_2606_25040_amd import ops
import workloads as wk

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def device():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    ops.load_library()
    torch.cuda.set_device(0)
    yield


def _both(q, k, top_p, mk, kv_block=64, key_scale=None, sm=None):
    ref = ops.build_block_mask(q, k, top_p, mk, sm_scale=sm, return_scores=True, kv_block=kv_block,
                               key_scale=key_scale)
    B, S, H, _ = q.shape
    n = (S + 63) // 64
    nk = (S + kv_block - 1) // kv_block
    rows = B * H * n
    out = ops.BlockMask(torch.full((rows + 1,), -7, dtype=torch.int32, device="cuda"),
                        torch.full((rows * nk,), -7, dtype=torch.int32, device="cuda"), B, H, n, kv_block)
    scores = torch.full((rows, nk), float("nan"), dtype=torch.float32, device="cuda")
    got = ops.build_block_mask_noalloc(q, k, top_p, mk, out, sm_scale=sm, key_scale=key_scale,
                                       kv_block=kv_block, block_scores=scores)
    torch.cuda.synchronize()
    rp_r, ci_r = ref.to_host()
    rp_g, ci_g = got.to_host()
    assert np.array_equal(rp_g, rp_r)
    assert np.array_equal(ci_g, ci_r)
    assert torch.equal(scores.view(torch.int32), ref.block_scores.view(torch.int32))
    return int(rp_r[-1])


def test_noalloc_builder_matches_workspace_builder_on_two_calls():
    # call 1: the mask source of the batch-4 workload (B 1, H 40, S 32,760,
    # bf16): 20,480 rows, the 40 heads in two chunks of the fixed scratch
    wl = dataclasses.replace(wk.WORKLOADS["wan14b_480p_batch4_bf16"], B=1)
    inp = wk.make_inputs(wl, with_v=False)
    q, k = inp.q.cuda(), inp.k.cuda()
    nnz = _both(q, k, wl.top_p, wl.min_top_k, sm=wl.sm_scale)
    assert 0.14 < nnz / (wl.H * wl.n_blocks ** 2) < 0.16
    del q, k, inp
    # call 2, smaller: two requests (one mask each), f16, kv blocks of 128,
    # first-frame key scale, a partial last block
    gen = torch.Generator().manual_seed(5)
    x = torch.randn(2, 1000, 3, 128, generator=gen)
    q2 = (x * 0.5).to(torch.float16).cuda()
    k2 = (x * 0.5 + 0.3 * torch.randn(2, 1000, 3, 128, generator=gen)).to(torch.float16).cuda()
    _both(q2, k2, 0.6, 0.05, kv_block=128, key_scale=(200, 1.4))
    _both(q2, k2, 0.9, 0.0)
