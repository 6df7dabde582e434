"""Calibrate the frozen ``top_p`` of each builder workload with the oracle.

The paper's selection is joint top-p with a top-k floor (Sec. 3.2, knobs in
Sec. 4.1); a workload is specified by a target density X instead.  Reading:
``min_top_k = X / 4`` (the paper's default floor 0.1 against a ~0.4 keep
ratio, Table 2) and ``top_p`` is bisected on the oracle builder so that the
mean density over all rows is X within 0.25 percentage points, then moved to
the middle of the widest nearby gap between any row's cumulative masses, so
that no row sits within rounding of its top-p boundary.

Prints the values to freeze in ``workloads.py``.
Test infrastructure: calls only ``oracle/`` and the input generator.

    python -m oracle.calibrate_top_p [workload ...]
"""

from __future__ import annotations

import sys
import time

import numpy as np

from oracle import mask as om
import workloads as wk


def cumulative_rows(q, k, sm_scale):
    """Per row: sorted cumulative mass (as the oracle's top-p step sees it)."""
    B, S, H, D = q.shape
    out = []
    for b in range(B):
        for h in range(H):
            s = om.block_scores(om.pool_means(q[b, :, h, :]), om.pool_means(k[b, :, h, :]),
                                sm_scale)
            for i in range(s.shape[0]):
                order = om.row_order(s[i])
                out.append(np.cumsum(om.row_mass(s[i])[order]))
    return np.stack(out)


def density(C: np.ndarray, top_p: float, k_min: int) -> float:
    n = C.shape[1]
    kp = (C < top_p).sum(axis=1) + 1
    k = np.minimum(n, np.maximum(np.maximum(kp, k_min), 1))
    return float(k.sum()) / (C.shape[0] * n)


def calibrate(wl: wk.Workload, tol: float = 0.0025):
    inp = wk.make_inputs(wl, with_v=False)
    q = inp.mask_q.float().numpy()
    k = inp.mask_k.float().numpy()
    C = cumulative_rows(q, k, wl.sm_scale)
    n = C.shape[1]
    min_top_k = wl.density / 4.0
    k_min = om.floor_count(min_top_k, n)
    lo, hi = 0.0, 1.0
    for _ in range(60):
        mid = 0.5 * (lo + hi)
        if density(C, mid, k_min) < wl.density:
            lo = mid
        else:
            hi = mid
    p0 = hi
    near = np.unique(C[np.abs(C - p0) < 5e-3])
    gaps = np.diff(near)
    best, best_gap = p0, 0.0
    for g in np.argsort(-gaps)[:200]:
        cand = 0.5 * (near[g] + near[g + 1])
        if abs(density(C, cand, k_min) - wl.density) <= tol and gaps[g] > best_gap:
            best, best_gap = float(cand), float(gaps[g])
    margin = float(np.min(np.abs(C - best)))
    return best, min_top_k, density(C, best, k_min), margin


def main(keys):
    for key in keys:
        wl = wk.WORKLOADS[key]
        if wl.mask_source == "random":
            continue
        t = time.time()
        top_p, mk, d, margin = calibrate(wl)
        print(f"{key}: top_p={top_p!r} min_top_k={mk!r} density={d:.5f} "
              f"(target {wl.density}) boundary margin={margin:.2e} [{time.time() - t:.0f}s]",
              flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or wk.ORDER)
