"""Benchmark of the block-sparse attention hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload KEY]

A step is one pass of the whole hot path over one request batch with inputs
resident in HBM: mask builder (block mean-pool, float64 block scores, top-p /
top-k selection, CSR), work plan, [FP8 quantisation of Q, K, V for the fp8
workload], and the block-sparse attention forward pass.  When the fp8 path
builds the mask from the request's own Q and K, the quantiser writes their
float64 block sums as it reads them and the builder starts from those sums
(the block mean-pool without a second pass over Q and K).  The metric is the
effective TFLOP/s on computed blocks, 4 * 64 * 64 * 128 FLOP per computed
(q-block, kv-block) pair, over the measured time.  Prints ONE JSON line.

The default workload is the largest one that fits one GPU: four similar
requests (B 4, H 40, S 32,760 on a 21 x 30 x 52 latent grid, bf16) sharing one
15 %-density mask built from request 0.

Beside the step throughput the line carries: the attention kernel's own
throughput and MFMA-roofline fraction (HIP events on the launch stream), the
builder time and the routing-overhead ratio routing / (routing + attention)
(Eq. 3), the speedup over the same kernel code at 100% density, and the CPU
oracle's throughput on a bounded sample of the same workload.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"bf16": 2516.6, "f16": 2516.6, "fp8": 5033.2}   # 256 CU x 2.4 GHz x 4096 / 8192
FLOP_PER_PAIR = 4 * 64 * 64 * 128
DEFAULT_WORKLOAD = "wan14b_480p_batch4_bf16"
PROFILES = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work")
    ap.add_argument("--kv-block", type=int, default=64, choices=(64, 128),
                    help="tokens per kv block of the built mask (128 = the paper's kernel geometry)")
    ap.add_argument("--no-graph", action="store_true", help="skip the HIP-graph replay of the step")
    ap.add_argument("--f16", action="store_true",
                    help="run a 16-bit workload in f16 (its inputs converted) instead of bf16")
    ap.add_argument("--head-schedule", action="store_true",
                    help="instead of the throughput line, time the attention of the fp8 720p 14B workload on "
                         "each of 8 five-head sets (the one-GPU share of an 8-GPU head-parallel layout): the "
                         "plan's balanced sets against contiguous slices")
    ap.add_argument("--coverage", action="store_true",
                    help="instead of the throughput line, print the mask-coverage study (true block-mass "
                         "masks of a historical request reused on similar requests)")
    return ap.parse_args()


def source_hash(names) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2606_25040_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_from_profile(kernel_file: str, workload: str, src_hash: str):
    """HBM bytes per launch from the committed counter summary, or None when
    missing or taken on a different kernel source."""
    path = os.path.join(PROFILES, f"traffic_{workload}.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != src_hash or rec.get("kernel_file") != kernel_file:
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_baseline(wl, inp, budget_s: float, gpu=None):
    """Oracle (plain NumPy float64) on a bounded sample of the same workload:
    head by head of request 0, the oracle mask builder for the head (or the
    fixed mask's rows) followed by the oracle attention of that head's
    q-blocks in order, until about ``budget_s`` seconds of work are spent.
    Returns effective TFLOP/s on computed blocks and a description.

    With ``gpu = (row_ptr, col_idx, out)`` (the GPU mask of request 0 and the
    GPU attention output), every sampled q-block whose GPU mask row equals the
    oracle's is also compared with the GPU output (outside the timed work);
    the statistics are returned as a second value."""
    from oracle import attention as oa
    from oracle import mask as om
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = 1
    cores = len(os.sched_getaffinity(0))
    t_build = t_attn = 0.0
    pairs = 0
    blocks_done = 0
    heads_done = 0
    cmp = {"q_blocks": 0, "rows_differing": 0, "max_abs": 0.0, "sum_abs": 0.0, "n": 0, "d2": 0.0, "r2": 0.0}
    for h in range(wl.H):
        t0 = time.perf_counter()
        if inp.mask_q is not None:
            mq = inp.mask_q[0, :, h].float().numpy()
            mk = inp.mask_k[0, :, h].float().numpy()
            s = om.block_scores(om.pool_means(mq), om.pool_means(mk), wl.sm_scale)
            rows = [om.select_row(s[i], wl.top_p, wl.min_top_k) for i in range(wl.n_blocks)]
        else:
            rp, ci = inp.random_mask
            base = h * wl.n_blocks
            rows = [ci[rp[base + i]:rp[base + i + 1]] for i in range(wl.n_blocks)]
        if wl.dtype == "fp8":
            from oracle import fp8 as of
            qh, kh, vh = (of.dequantize_blockwise(*of.quantize_blockwise(x[:1, :, h:h + 1].float().numpy()))
                          [0, :, 0] for x in (inp.q, inp.k, inp.v))
        else:
            qh, kh, vh = (x[0, :, h].float().numpy() for x in (inp.q, inp.k, inp.v))
        oh = None if gpu is None else gpu[2][0, :, h].float().cpu().numpy().astype(np.float64)
        t1 = time.perf_counter()
        t_build += t1 - t0
        done = 0
        t_cmp = 0.0
        for i in range(wl.n_blocks):
            o_i, _ = oa.attention_block(qh, kh, vh, rows[i], i, wl.sm_scale)
            pairs += len(rows[i])
            done += 1
            if gpu is not None:
                tc = time.perf_counter()
                r = h * wl.n_blocks + i
                if np.array_equal(np.asarray(gpu[1][gpu[0][r]:gpu[0][r + 1]]), np.asarray(rows[i])):
                    d = np.abs(oh[i * 64:i * 64 + o_i.shape[0]] - o_i)
                    cmp["q_blocks"] += 1
                    cmp["max_abs"] = max(cmp["max_abs"], float(d.max()))
                    cmp["sum_abs"] += float(d.sum())
                    cmp["n"] += d.size
                    cmp["d2"] += float((d * d).sum())
                    cmp["r2"] += float((o_i * o_i).sum())
                else:
                    cmp["rows_differing"] += 1
                t_cmp += time.perf_counter() - tc
            if t_build + t_attn + (time.perf_counter() - t1 - t_cmp) > budget_s:
                break
        t_attn += time.perf_counter() - t1 - t_cmp
        blocks_done += done
        heads_done += 1
        if t_build + t_attn > budget_s:
            break
    value = pairs * FLOP_PER_PAIR / (t_build + t_attn) / 1e12
    sample = (f"request 0, heads 0..{heads_done - 1}: oracle mask builder per head ({t_build:.2f} s incl. "
              f"input casts) + oracle attention (gather form, float64) of {blocks_done} q-blocks in order "
              f"({pairs} computed block pairs, {t_attn:.2f} s); float64 NumPy, BLAS threads {threads}")
    base = {"value": value, "unit": "TFLOP/s", "cores": min(threads, cores), "kind": "oracle",
            "sample": sample}
    if gpu is None:
        return base, None
    par = {"q_blocks_compared": cmp["q_blocks"], "q_blocks_with_differing_mask_row": cmp["rows_differing"],
           "max_abs_err": cmp["max_abs"], "mean_abs_err": cmp["sum_abs"] / max(cmp["n"], 1),
           "rel_frobenius_err": (cmp["d2"] / cmp["r2"]) ** 0.5 if cmp["r2"] > 0 else None,
           "reference": "oracle (float64) on the cpu_baseline sample, where its mask row equals the GPU's"}
    return base, par


def coverage_study(args) -> None:
    """Synthetic analogue of the paper's reuse study (Sec. 3.2 Obs. 1): the
    true top-p (p = 0.9) block mask of a historical request, taken from its
    dense attention map, is applied to new requests drawn at increasing
    distance (noise level sigma) from it, and judged by coverage -- the share
    of the new request's attention mass inside the mask -- next to the new
    request's own true mask and the mean-pool predictor built on the new
    request with its top_p bisected to the same keep ratio.  One JSON line."""
    import torch

    from paper_2606_25040_amd import ops
    import workloads as wk

    torch.cuda.set_device(0)
    ops.load_library()
    key = args.workload if args.workload != DEFAULT_WORKLOAD else "wan14b_480p_reuse_bf16"
    wl = wk.WORKLOADS[key]
    if wl.dtype == "fp8":
        raise SystemExit("the coverage study runs on the 16-bit workloads")
    sigmas = [0.1, 0.3, 0.6, 1.0]
    true_p = 0.9
    S, sm, mk = wl.S, wl.sm_scale, wl.min_top_k
    bq, bk, reqs = wk.make_similar_requests(wl, sigmas)

    def event_ms(fn, reps=3):
        fn()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        e1.synchronize()
        return e0.elapsed_time(e1) / reps

    def mass_of(q, k):
        qd, kd = q.cuda(), k.cuda()
        _, lse = ops.block_sparse_attn_fwd(qd, kd, kd, None, sm_scale=sm, return_lse=True)
        return ops.attn_block_mass(qd, kd, lse, sm_scale=sm), qd, kd, lse

    m_base, qd, kd, lse = mass_of(bq, bk)
    mass_ms = event_ms(lambda: ops.attn_block_mass(qd, kd, lse, sm_scale=sm, out=m_base))
    hist = ops.select_block_mask(m_base, S, true_p, mk)
    select_ms = event_ms(lambda: ops.select_block_mask(m_base, S, true_p, mk, out=hist))
    pairs = wl.H * wl.n_blocks * wl.n_blocks
    mass_tflops = pairs * 2 * 64 * 64 * 128 / (mass_ms * 1e-3) / 1e12
    del qd, kd, lse
    # the true mask a second time, with its top_p bisected to the workload's
    # keep ratio (the density the attention kernels are measured at)
    lo, hi = 0.0, 1.0
    for _ in range(30):
        mid = 0.5 * (lo + hi)
        if ops.select_block_mask(m_base, S, mid, mk).density < wl.density:
            lo = mid
        else:
            hi = mid
    p_keep = hi
    hist_keep = ops.select_block_mask(m_base, S, p_keep, mk)

    def bisect_builder(qd, kd, target):
        lo, hi = 0.0, 1.0
        for _ in range(24):
            mid = 0.5 * (lo + hi)
            if ops.build_block_mask(qd, kd, mid, mk, sm_scale=sm).density < target:
                lo = mid
            else:
                hi = mid
        return ops.build_block_mask(qd, kd, hi, mk, sm_scale=sm)

    results = []
    for sig, (q, k) in zip(sigmas, reqs):
        m_r, qd, kd, _ = mass_of(q, k)
        row = {"sigma": sig}
        for tag, p_true, hmask in (("p0.9", true_p, hist), ("keep", p_keep, hist_keep)):
            own = ops.select_block_mask(m_r, S, p_true, mk)
            pred = bisect_builder(qd, kd, hmask.density)
            row[tag] = {"keep_ratio_reused": round(hmask.density, 5),
                        "keep_ratio_own": round(own.density, 5),
                        "keep_ratio_meanpool": round(pred.density, 5),
                        "coverage_own_true_mask": round(float(ops.mask_coverage(own, m_r, S).mean()), 5),
                        "coverage_reused_true_mask": round(float(ops.mask_coverage(hmask, m_r, S).mean()), 5),
                        "coverage_meanpool_predictor": round(float(ops.mask_coverage(pred, m_r, S).mean()), 5)}
        results.append(row)
        del qd, kd, m_r
    line = {"study": "mask coverage of a reused true top-p mask (synthetic analogue of Sec. 3.2 Obs. 1)",
            "workload": key, "true_top_p": true_p, "keep_setting_top_p": round(p_keep, 6), "min_top_k": mk,
            "data": "synthetic (seeded base request; new requests = base + sigma * N(0,1) on Q and K)",
            "block_mass_ms": round(mass_ms, 3), "block_mass_tflops": round(mass_tflops, 1),
            "select_from_mass_ms": round(select_ms, 4), "results": results}
    print(json.dumps(line), flush=True)


def head_schedule_study(args) -> None:
    """The one-GPU share of head-parallel attention (Sec. 3.2 "Head-level
    scheduling for load balancing", Appendix A): the 40 heads of the 720p 14B
    fp8 workload are split into 8 sets of 5, one per rank of an 8-GPU layout,
    either as contiguous slices or as the plan's balanced sets (the plan deals
    units heaviest first to the least-loaded of 8 bins of equal capacity --
    the rule the paper applies to GPUs, here read off the plan's unit order,
    5 units per bin).  Each set's attention (its heads' Q/K/V codes and mask
    rows) is launched alone on this GPU and timed; the imbalance is the
    max / mean of the 8 set times.  One JSON line."""
    import torch

    from paper_2606_25040_amd import ops
    import workloads as wk

    torch.cuda.set_device(0)
    ops.load_library()
    wl = wk.WORKLOADS["wan14b_720p_fp8"]
    G = 8
    inp = wk.make_inputs(wl)
    H, n, S = wl.H, wl.n_blocks, wl.S
    q, k, v = inp.q.cuda(), inp.k.cuda(), inp.v.cuda()
    mask = ops.build_block_mask(inp.mask_q.cuda(), inp.mask_k.cuda(), wl.top_p, wl.min_top_k,
                                sm_scale=wl.sm_scale)
    codes = [ops.quantize_fp8_blockwise(x) for x in (q, k, v)]
    del q, k, v
    order = ops.plan_block_mask(mask, 1, S).cpu().tolist()
    rp, ci = mask.to_host()
    cost = [int(rp[(h + 1) * n] - rp[h * n]) for h in range(H)]
    per = H // G
    sets = {"contiguous": [list(range(r * per, (r + 1) * per)) for r in range(G)],
            "planned": [order[r * per:(r + 1) * per] for r in range(G)]}

    def set_ms(heads):
        idx = torch.tensor(heads, device="cuda")
        cs = [(c.index_select(2, idx).contiguous(), s_.index_select(1, idx).contiguous()) for c, s_ in codes]
        rows = [np.asarray(ci[rp[h * n + i]:rp[h * n + i + 1]]) for h in heads for i in range(n)]
        sub_rp = np.zeros(len(rows) + 1, dtype=np.int64)
        np.cumsum([len(r) for r in rows], out=sub_rp[1:])
        sub = ops.BlockMask.from_host(sub_rp, np.concatenate(rows), 1, len(heads), n)
        sched = ops.plan_block_mask(sub, 1, S)
        out = torch.empty((1, S, len(heads), 128), dtype=torch.bfloat16, device="cuda")
        fn = lambda: ops.block_sparse_attn_fwd(cs[0][0], cs[1][0], cs[2][0], sub, sm_scale=wl.sm_scale,
                                               scales=(cs[0][1], cs[1][1], cs[2][1]), out=out, schedule=sched)
        fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        reps = 10
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        e1.synchronize()
        return e0.elapsed_time(e1) / reps

    result = {}
    for name, ss in sets.items():
        ms = [set_ms(hs) for hs in ss]
        loads = [sum(cost[h] for h in hs) for hs in ss]
        result[name] = {"heads": ss, "set_ms": [round(x, 4) for x in ms],
                        "imbalance_time": round(max(ms) / (sum(ms) / G), 4),
                        "listed_blocks": loads,
                        "imbalance_listed_blocks": round(max(loads) / (sum(loads) / G), 4)}
    line = {"study": "one-GPU share of head-level scheduling over 8 head sets (Sec. 3.2, Appendix A)",
            "workload": wl.key, "sets": G, "heads_per_set": per, "dtype": "fp8",
            "data": "synthetic (seeded Wan-class Q/K/V on the latent grid; no real latents)",
            "paper_imbalance": {"without_scheduler": 1.34, "with_scheduler": 1.12},
            "results": result}
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(what is measured is the single-GPU share of the path).", file=sys.stderr)
        sys.exit(2)
    if args.coverage:
        coverage_study(args)
        return
    if args.head_schedule:
        head_schedule_study(args)
        return
    import torch

    from paper_2606_25040_amd import ops
    import workloads as wk

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    ops.load_library()
    wl = wk.WORKLOADS[args.workload]
    inp = wk.make_inputs(wl)
    fp8 = wl.dtype == "fp8"
    if args.f16:
        if fp8:
            sys.exit("--f16 applies to the 16-bit workloads only")
        for name in ("q", "k", "v", "mask_q", "mask_k"):
            x = getattr(inp, name, None)
            if x is not None:
                setattr(inp, name, x.to(torch.float16))
    dtype_name = "f16" if args.f16 else wl.dtype
    q, k, v = inp.q.cuda(), inp.k.cuda(), inp.v.cuda()
    B, S, H = wl.B, wl.S, wl.H
    n = wl.n_blocks

    # ---- preallocated buffers: the timed region allocates nothing
    if wl.mask_source == "random":
        rp, ci = inp.random_mask
        fixed = ops.BlockMask.from_host(rp, ci, 1, H, n)
        mq = mk = None
    else:
        mq, mk = inp.mask_q.cuda(), inp.mask_k.cuda()
        fixed = None
    mask_buf = None
    ws_build = None
    if mq is not None:
        Bm = mq.shape[0]
        mask_buf = ops.BlockMask(torch.empty(Bm * H * n + 1, dtype=torch.int32, device="cuda"),
                                 torch.empty(Bm * H * n * n, dtype=torch.int32, device="cuda"),
                                 Bm, H, n)
        need = ops.load_library().chorus_build_block_mask_workspace_size(
            ops.ctypes.byref(ops.Shape(Bm, S, H, 128)))
        ws_build = torch.empty(need + 256, dtype=torch.uint8, device="cuda")
    order = torch.empty(B * H, dtype=torch.int32, device="cuda")
    ws_plan = torch.empty(4096 + B * H * 4, dtype=torch.uint8, device="cuda")
    out = torch.empty((B, S, H, 128), dtype=torch.bfloat16 if fp8 else q.dtype, device="cuda")
    if fp8:
        codes = [torch.empty((B, S, H, 128), dtype=torch.uint8, device="cuda") for _ in range(3)]
        scales = [torch.empty((B, H, n), dtype=torch.float32, device="cuda") for _ in range(3)]
    # a mask built from the request's own Q and K on the fp8 path takes the
    # block sums that the quantiser writes while it reads Q and K, instead of
    # a second pass over them
    from_sums = fp8 and wl.mask_source == "self"
    if from_sums:
        sums = [torch.empty((B, H, n, 128), dtype=torch.float64, device="cuda") for _ in range(2)]

    kvb = args.kv_block
    if kvb != 64 and mq is None:
        sys.exit("--kv-block 128 needs a workload whose mask is built")

    def build_from_qk():
        return ops.build_block_mask(mq, mk, wl.top_p, wl.min_top_k, sm_scale=wl.sm_scale,
                                    out=mask_buf, workspace=ws_build, kv_block=kvb)

    def build():
        if mq is None:
            return fixed
        if from_sums:
            return ops.build_block_mask_from_sums(sums[0], sums[1], S, wl.top_p, wl.min_top_k,
                                                  sm_scale=wl.sm_scale, out=mask_buf, workspace=ws_build,
                                                  kv_block=kvb)
        return build_from_qk()

    def plan(m):
        return ops.plan_block_mask(m, B, S, out=order, workspace=ws_plan)

    def quant_plain():
        for x, c, s in zip((q, k, v), codes, scales):
            ops.quantize_fp8_blockwise(x, codes=c, scales=s)

    def quant():
        if not from_sums:
            return quant_plain()
        for x, c, s, t in zip((q, k), codes, scales, sums):
            ops.quantize_fp8_blockwise_sums(x, codes=c, scales=s, block_sums=t)
        ops.quantize_fp8_blockwise(v, codes=codes[2], scales=scales[2])

    def attn(m, sched, dense=False, key_scale=None):
        mm = None if dense else m
        if fp8:
            return ops.block_sparse_attn_fwd(codes[0], codes[1], codes[2], mm, sm_scale=wl.sm_scale,
                                             scales=tuple(scales), out=out, schedule=sched,
                                             key_scale=key_scale)
        return ops.block_sparse_attn_fwd(q, k, v, mm, sm_scale=wl.sm_scale, out=out,
                                         schedule=sched, key_scale=key_scale)

    def step():
        if from_sums:
            quant()                   # codes, scales and the block sums of Q and K
        m = build()
        sched = plan(m)
        if fp8 and not from_sums:
            quant()
        attn(m, sched)

    # ---- whole-step throughput
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / args.steps

    # the same step captured once into a HIP graph and replayed (the path
    # allocates nothing and records no memset nodes), reported beside the
    # eager step
    graph_ms = None
    if not args.no_graph:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            graph.replay()
        torch.cuda.synchronize()
        graph_ms = (time.perf_counter() - t0) * 1e3 / args.steps
        del graph
    mask = build()
    sched = plan(mask)
    torch.cuda.synchronize()
    nnz = mask.nnz
    # computed 64 x 64 block pairs: a kv block of 128 is two, except a last
    # block of 64 tokens or fewer (odd number of q-blocks)
    sub = nnz
    if kvb == 128:
        _, ids = mask.to_host()
        sub = 2 * nnz - (int((ids == mask.n_kv - 1).sum()) if n % 2 else 0)
    pairs = B * sub
    flops = pairs * FLOP_PER_PAIR
    value = flops / (ms_per_step * 1e-3) / 1e12

    # ---- per-kernel times with HIP events on the launch stream
    def event_ms(fn, reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        e1.synchronize()
        return e0.elapsed_time(e1) / reps

    reps = max(args.steps, 10)
    attn_ms = event_ms(lambda: attn(mask, sched), reps)

    # per-launch spread of the attention kernel (one event pair per launch)
    def launch_stats(fn, reps):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in ev:
            a.record()
            fn()
            b.record()
        ev[-1][1].synchronize()
        t = sorted(a.elapsed_time(b) for a, b in ev)
        return {"median": round(t[len(t) // 2], 4), "min": round(t[0], 4),
                "p90": round(t[min(len(t) - 1, (9 * len(t)) // 10)], 4), "launches": len(t)}

    attn_stats = launch_stats(lambda: attn(mask, sched), max(reps, 20))
    # the same launch with the first-frame key enhancement (first latent frame
    # = grid_y * grid_x tokens, beta 1.3)
    first_frame = wl.grid[1] * wl.grid[2]
    attn_ks_ms = event_ms(lambda: attn(mask, sched, key_scale=(first_frame, 1.3)), reps)
    build_ms = event_ms(build, reps) if mq is not None else 0.0
    plan_ms = event_ms(lambda: plan(mask), reps)
    quant_ms = event_ms(quant, reps) if fp8 else 0.0
    # with the mask from block sums, the routing cost is the builder from sums
    # plus what the sums add to the quantiser; the builder that reads Q and K
    # itself is timed beside it
    build_qk_ms = quant_plain_ms = None
    routing_ms = build_ms
    if from_sums:
        quant_plain_ms = event_ms(quant_plain, reps)
        build_qk_ms = event_ms(build_from_qk, reps)
        quant()
        build()                       # the step's own mask again
        routing_ms = build_ms + max(0.0, quant_ms - quant_plain_ms)
    build_fp8_ms = None
    if fp8 and mq is not None:
        # the builder reading fp8 codes of the mask source instead of 16-bit values
        (mqc, mqs), (mkc, mks) = (ops.quantize_fp8_blockwise(x) for x in (mq, mk))
        build_fp8_ms = event_ms(lambda: ops.build_block_mask(
            mqc, mkc, wl.top_p, wl.min_top_k, sm_scale=wl.sm_scale, scales=(mqs, mks),
            out=mask_buf, workspace=ws_build), reps)
        del mqc, mqs, mkc, mks
        build()                       # the step's own mask again
    # block-pair visit refreshing of a layer group (outside the step: one
    # update per layer, one refresh at the group's last layer).  The refresh
    # is timed in its worst case: the map holds only this mask's own pairs,
    # so every other pair is forced in and the output is dense.
    vmap = ops.VisitMap(mask.mask_batch, H, n, block=mask.block)
    vmap.reset(mask)
    refreshed = ops.BlockMask(torch.empty_like(mask.row_ptr),
                              torch.empty(mask.rows * mask.n_kv, dtype=torch.int32, device="cuda"),
                              mask.mask_batch, H, n, mask.block)
    need = ops.load_library().chorus_visit_refresh_workspace_size(ops.ctypes.byref(mask.as_c()))
    ws_visit = torch.empty(need + 256, dtype=torch.uint8, device="cuda")
    visit_update_ms = event_ms(lambda: vmap.update(mask), reps)
    visit_refresh_ms = event_ms(lambda: vmap.refresh(mask, out=refreshed, workspace=ws_visit), reps)
    del vmap, refreshed, ws_visit
    dense_reps = max(3, reps // 4)
    dense_ms = event_ms(lambda: attn(mask, None, dense=True), dense_reps)
    attn_tflops = flops / (attn_ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[wl.dtype]

    kernel_file = "attn_fwd_fp8.hip" if fp8 else "attn_fwd.hip"
    src_hash = source_hash([kernel_file, "attn_common.h"])
    variant = ("_f16" if args.f16 else "") + ("_kv128" if kvb == 128 else "")
    traffic = traffic_from_profile(kernel_file, wl.key + variant, src_hash)

    line = {
        "metric": "effective TFLOP/s on computed blocks & % MFMA peak; speedup vs 100%-density",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "graph_ms_per_step": None if graph_ms is None else round(graph_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype_name,
        "data": "synthetic (seeded Wan-class Q/K/V on the latent grid; no real latents)",
        "config": {
            "workload": wl.key, "B": B, "S": S, "H": H, "D": 128, "block": 64,
            "grid_tyx": list(wl.grid), "mask_source": wl.mask_source,
            "kv_block": kvb,
            "target_density": wl.density, "density": round(sub / float(mask.rows * n), 5),
            "top_p": wl.top_p, "min_top_k": wl.min_top_k, "computed_pairs": pairs,
            "step": ("fp8 quantise (with Q, K block sums) + mask build from the sums + plan + attention"
                     if from_sums else
                     "mask build + plan" + (" + fp8 quantise" if fp8 else "") + " + attention"),
        },
        "attn_ms": round(attn_ms, 4),
        "attn_ms_per_launch": attn_stats,
        "attn_tflops": round(attn_tflops, 2),
        "attn_frac_mfma_peak": round(attn_tflops / peak, 4),
        "attn_key_scaled_ms": round(attn_ks_ms, 4),
        "builder_ms": round(build_ms, 4),
        "builder_input": "block sums from the quantiser" if from_sums else ("Q, K" if mq is not None else None),
        "builder_from_qk_ms": None if build_qk_ms is None else round(build_qk_ms, 4),
        "builder_fp8_input_ms": None if build_fp8_ms is None else round(build_fp8_ms, 4),
        "plan_ms": round(plan_ms, 4),
        "quant_ms": round(quant_ms, 4),
        "quant_plain_ms": None if quant_plain_ms is None else round(quant_plain_ms, 4),
        "routing_ms": round(routing_ms, 4),
        # HBM-bound stages: algorithmic bytes over time (the builder reads the
        # mask source's Q and K once; the quantiser reads 2 B and writes 1 B per
        # element of Q, K and V, plus the scales)
        "builder_gbps": (round(2 * mq.numel() * mq.element_size() / (build_ms * 1e-3) / 1e9, 1)
                         if mq is not None and build_ms > 0 and not from_sums else None),
        "quant_gbps": (round((3 * 3 * q.numel() + 3 * 4 * B * H * n + (16 * B * H * n * 128 if from_sums else 0))
                             / (quant_ms * 1e-3) / 1e9, 1)
                       if fp8 and quant_ms > 0 else None),
        "visit_update_ms": round(visit_update_ms, 4),
        "visit_refresh_worst_ms": round(visit_refresh_ms, 4),
        "routing_overhead_ratio": round(routing_ms / (routing_ms + attn_ms), 4),
        "dense_attn_ms": round(dense_ms, 4),
        "speedup_vs_dense": round(dense_ms / attn_ms, 3),
        "ideal_speedup": round(float(mask.rows * n) / sub, 3),
        "roofline": {
            "kernel": (f"attn_fwd_fp8_kernel<false, false, {str(kvb == 128).lower()}>" if fp8 else
                       f"attn_fwd_16_kernel<{str(not args.f16).lower()}, false, false, "
                       f"{str(kvb == 128).lower()}>"),
            "bound": "mfma",
            "achieved": round(attn_tflops, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(attn_tflops / peak, 4),
            "traffic": traffic,
            "source_hash": src_hash,
        },
    }
    if not args.no_cpu_baseline:
        attn(mask, sched)                # the step's attention output again (later runs overwrote it)
        torch.cuda.synchronize()
        grp, gci = mask.to_host()
        # (the oracle sample follows the kv-64 geometry; with --kv-block 128 no rows are compared)
        gpu = (grp, gci, out) if kvb == 64 else None
        line["cpu_baseline"], line["parity_sample"] = cpu_baseline(wl, inp, args.cpu_budget, gpu)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
