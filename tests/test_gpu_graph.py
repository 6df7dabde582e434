"""The whole hot path captured into a HIP graph (torch.cuda.CUDAGraph) and
replayed: mask build, plan, fp8 quantisation and attention allocate nothing
and use no memset nodes, so a captured step must reproduce the eager step
bit for bit on every replay, with unrelated eager work between replays.  The
fp8 step is also captured in its block-sums form (the quantiser writes the
block sums of Q and K, the mask is built from them)."""

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


class Step:
    """Preallocated buffers of one step: build + plan (+ quantise) + attention."""

    def __init__(self, q, k, v, top_p, mk, sm, fp8, kv_block=64, from_sums=False):
        B, S, H, D = q.shape
        n = (S + 63) // 64
        nk = (S + kv_block - 1) // kv_block
        self.q, self.k, self.v, self.top_p, self.mk, self.sm, self.fp8 = q, k, v, top_p, mk, sm, fp8
        self.kv_block = kv_block
        self.from_sums = from_sums
        self.mask = ops.BlockMask(torch.empty(B * H * n + 1, dtype=torch.int32, device="cuda"),
                                  torch.empty(B * H * n * nk, dtype=torch.int32, device="cuda"), B, H, n, kv_block)
        need = ops.load_library().chorus_build_block_mask_workspace_size(ops.ctypes.byref(ops._shape(q)))
        self.ws = torch.empty(need + 256, dtype=torch.uint8, device="cuda")
        self.order = torch.empty(B * H, dtype=torch.int32, device="cuda")
        self.out = torch.empty((B, S, H, D), dtype=torch.bfloat16 if fp8 else q.dtype, device="cuda")
        if fp8:
            self.codes = [torch.empty((B, S, H, D), dtype=torch.uint8, device="cuda") for _ in range(3)]
            self.scales = [torch.empty((B, H, n), dtype=torch.float32, device="cuda") for _ in range(3)]
        if from_sums:
            self.sums = [torch.empty((B, H, n, D), dtype=torch.float64, device="cuda") for _ in range(2)]

    def __call__(self):
        if self.from_sums:
            for x, c, s, t in zip((self.q, self.k), self.codes, self.scales, self.sums):
                ops.quantize_fp8_blockwise_sums(x, codes=c, scales=s, block_sums=t)
            ops.quantize_fp8_blockwise(self.v, codes=self.codes[2], scales=self.scales[2])
            m = ops.build_block_mask_from_sums(self.sums[0], self.sums[1], self.q.shape[1], self.top_p, self.mk,
                                               sm_scale=self.sm, out=self.mask, workspace=self.ws,
                                               kv_block=self.kv_block)
            ops.plan_block_mask(m, self.q.shape[0], self.q.shape[1], out=self.order)
            ops.block_sparse_attn_fwd(*self.codes, m, sm_scale=self.sm, scales=tuple(self.scales), out=self.out,
                                      schedule=self.order)
            return
        m = ops.build_block_mask(self.q, self.k, self.top_p, self.mk, sm_scale=self.sm, out=self.mask,
                                 workspace=self.ws, kv_block=self.kv_block)
        ops.plan_block_mask(m, self.q.shape[0], self.q.shape[1], out=self.order)
        if self.fp8:
            for x, c, s in zip((self.q, self.k, self.v), self.codes, self.scales):
                ops.quantize_fp8_blockwise(x, codes=c, scales=s)
            ops.block_sparse_attn_fwd(*self.codes, m, sm_scale=self.sm, scales=tuple(self.scales), out=self.out,
                                      schedule=self.order)
        else:
            ops.block_sparse_attn_fwd(self.q, self.k, self.v, m, sm_scale=self.sm, out=self.out,
                                      schedule=self.order)

    def snapshot(self):
        rp, ci = self.mask.to_host()
        snap = [rp, ci, self.order.cpu().numpy(), self.out.view(torch.int16).cpu().numpy()]
        if self.fp8:
            snap += [c.cpu().numpy() for c in self.codes] + [s.cpu().numpy() for s in self.scales]
        if self.from_sums:
            snap += [t.cpu().numpy() for t in self.sums]
        return snap


@pytest.mark.parametrize("fp8,kv_block,from_sums", [(False, 64, False), (True, 64, False), (False, 128, False),
                                                    (True, 64, True), (True, 128, True)])
def test_captured_step_replays_match_eager(fp8, kv_block, from_sums):
    gen = torch.Generator().manual_seed(11)
    B, S, H = 1, 3000, 4
    q, k, v = ((torch.randn(B, S, H, 128, generator=gen) * s).to(torch.bfloat16).cuda() for s in (0.5, 0.5, 1.0))
    step = Step(q, k, v, 0.8, 0.05, 128 ** -0.5, fp8, kv_block, from_sums)
    step()
    torch.cuda.synchronize()
    ref = step.snapshot()

    # other eager work on the same library between replays: a second step on
    # other inputs, writing its own buffers
    q2, k2, v2 = (x.flip(1).contiguous() for x in (q, k, v))
    other = Step(q2, k2, v2, 0.5, 0.1, 128 ** -0.5, fp8, kv_block, from_sums)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()                                   # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        for t in [step.out] + [step.order] + ([*step.codes] if fp8 else []) + (step.sums if from_sums else []):
            t.zero_()
        step.mask.col_idx.fill_(-7)
        graph.replay()
        other()
        torch.cuda.synchronize()
        got = step.snapshot()
        for a, b in zip(got, ref):
            assert np.array_equal(a, b), f"replay {rep} differs"
