"""GPU parity of block-pair visit refreshing (through the C ABI): the visited
map of a layer group and the group's last-layer mask against the oracle in
oracle/fallback.py, bit-exact; attention on the refreshed mask against the
attention oracle."""

import math

import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import fallback as fb
from paper_2606_25040_amd import ops
import workloads as wk

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def device():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    ops.load_library()
    torch.cuda.set_device(0)
    yield


def gpu_group(masks, V):
    """Runs one layer group through the visited map: every layer but the last
    records its mask, the last is refreshed and then recorded.  Returns the
    refreshed mask and the map just before the last layer."""
    V.reset(masks[0])
    for m in masks[:-1]:
        V.update(m)
    before = V.to_host()
    last = V.refresh(masks[-1])
    V.update(last)
    return last, before


def host_masks(rng, N, rows, n, empty_frac=0.1):
    out = []
    for _ in range(N):
        rp, ci = wk.random_csr(rng, rows, n, float(rng.uniform(0.02, 0.3)), empty_frac=empty_frac)
        out.append((rp, ci))
    return out


def check_group(hm, mask_batch, H, n, V=None):
    rows = mask_batch * H * n
    masks = [ops.BlockMask.from_host(rp, ci, mask_batch, H, n) for rp, ci in hm]
    V = V or ops.VisitMap(mask_batch, H, n)
    last, before = gpu_group(masks, V)
    torch.cuda.synchronize()
    dense = [fb.dense_of(rp, ci, rows, n) for rp, ci in hm]
    used, Vref = fb.run_group(dense, n)
    Vprev = np.zeros((rows, n), bool)
    for D in dense[:-1]:
        Vprev = fb.visit_update(Vprev, D)
    assert np.array_equal(before, Vprev)
    rp, ci = last.to_host()
    erp, eci = fb.csr_of(used[-1])
    assert np.array_equal(rp, erp) and np.array_equal(ci, eci)
    assert ops.validate_block_mask(last) == 0
    assert np.array_equal(V.to_host(), Vref) and Vref.all()
    return last, V


@pytest.mark.parametrize("n", [1, 5, 31, 32, 33, 64, 100])
@pytest.mark.parametrize("N", [1, 2, 8])
def test_group_matches_oracle(n, N):
    rng = np.random.Generator(np.random.PCG64(1000 * n + N))
    H, mask_batch = 3, 1
    check_group(host_masks(rng, N, mask_batch * H * n, n), mask_batch, H, n)


def test_group_batched_masks_and_two_groups_on_one_map():
    rng = np.random.Generator(np.random.PCG64(5))
    mask_batch, H, n = 2, 2, 47
    rows = mask_batch * H * n
    _, V = check_group(host_masks(rng, 8, rows, n), mask_batch, H, n)
    # the next group starts from a cleared map, whatever the last one left
    check_group(host_masks(rng, 8, rows, n, empty_frac=0.5), mask_batch, H, n, V)


def test_group_with_every_pair_visited_leaves_last_mask_unchanged():
    n, H = 40, 2
    rows = H * n
    full = (np.arange(0, rows * n + 1, n, dtype=np.int32), np.tile(np.arange(n, dtype=np.int32), rows))
    rng = np.random.Generator(np.random.PCG64(9))
    last_h = wk.random_csr(rng, rows, n, 0.2)
    last, _ = check_group([full, last_h], 1, H, n)
    rp, ci = last.to_host()
    assert np.array_equal(rp, last_h[0]) and np.array_equal(ci, last_h[1])


def test_largest_rows():
    rng = np.random.Generator(np.random.PCG64(4096))
    n = 4096
    hm = [wk.random_csr(rng, n, n, p) for p in (0.001, 0.01, 0.003)]
    check_group(hm, 1, 1, n)


def test_refresh_rejects_bad_arguments():
    n, H = 8, 1
    rp, ci = wk.random_csr(np.random.Generator(np.random.PCG64(1)), H * n, n, 0.5)
    m = ops.BlockMask.from_host(rp, ci, 1, H, n)
    V = ops.VisitMap(1, H, n)
    L = ops.load_library()
    out = torch.empty(H * n * n, dtype=torch.int32, device="cuda")
    optr = torch.empty(H * n + 1, dtype=torch.int32, device="cuda")
    cm = m.as_c()
    need = L.chorus_visit_refresh_workspace_size(ctypes_ref(cm))
    ws = torch.empty(need + 256, dtype=torch.uint8, device="cuda")
    wsp = ops._aligned(ws)
    # col capacity below the worst case
    st = L.chorus_visit_refresh(ctypes_ref(cm), V.bits.data_ptr(), optr.data_ptr(), out.data_ptr(),
                                H * n * n - 1, wsp, need, ops._stream())
    assert st != 0
    # workspace too small
    st = L.chorus_visit_refresh(ctypes_ref(cm), V.bits.data_ptr(), optr.data_ptr(), out.data_ptr(),
                                H * n * n, wsp, need - 4, ops._stream())
    assert st != 0
    # NULL map
    assert L.chorus_visit_update(ctypes_ref(cm), None, ops._stream()) != 0
    with pytest.raises(ValueError):
        V.update(ops.BlockMask(m.row_ptr, m.col_idx, 2, H, n))


def ctypes_ref(x):
    import ctypes
    return ctypes.byref(x)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
def test_attention_on_refreshed_mask(dtype):
    B, S, H = 2, 1000, 2
    n = (S + 63) // 64
    rng = np.random.Generator(np.random.PCG64(21))
    hm = host_masks(rng, 4, H * n, n)
    last, _ = check_group(hm, 1, H, n)
    rp, ci = last.to_host()
    gen = torch.Generator().manual_seed(8)
    q, k, v = (0.5 * torch.randn(B, S, H, 128, generator=gen)).to(dtype), \
        (0.5 * torch.randn(B, S, H, 128, generator=gen)).to(dtype), \
        torch.randn(B, S, H, 128, generator=gen).to(dtype)
    sm = 1.0 / math.sqrt(128)
    out = ops.block_sparse_attn_fwd(q.cuda(), k.cuda(), v.cuda(), last, sm_scale=sm)
    O, _ = oa.attention(q.double().numpy(), k.double().numpy(), v.double().numpy(), rp, ci, sm, 1)
    # fp32 accumulation, one output rounding of the 16-bit type
    eps = 2.0 ** -8 if dtype == torch.bfloat16 else 2.0 ** -11
    err = np.abs(out.double().cpu().numpy() - O)
    assert np.all(err <= 2e-3 + eps * np.abs(O)), float(err.max())


def test_full_size_group_720p_shape():
    """A group of eight masks at the 720p 14B shape (40 heads, 1182 blocks per
    side, 47 280 rows) with per-row densities around the paper's 10 %."""
    wl = wk.WORKLOADS["wan14b_720p_fp8"]
    H, n = wl.H, wl.n_blocks
    rows = H * n
    rng = np.random.Generator(np.random.PCG64(720))
    hm = []
    for _ in range(8):
        dens = np.clip(rng.gamma(2.0, 0.05, rows), 0.0, 1.0)
        keep = rng.random((rows, n)) < dens[:, None]
        hm.append(tuple(a.astype(np.int32) for a in fb.csr_of(keep)))
    check_group(hm, 1, H, n)
