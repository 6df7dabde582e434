"""Thin ctypes binding of libchorus.so (C ABI in include/chorus.h).

Argument marshalling only: torch tensors are used for device memory and the
current HIP stream; every step of the mask builder, the plan, the FP8
quantiser and the attention runs in the library's HIP kernels.  There is no
fallback: if the library is missing or a call fails, a RuntimeError is raised.

Function names follow the C entry points without their ``chorus_`` prefix.
"""

from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libchorus.so")

F16, BF16, FP8_E4M3 = 0, 1, 2
BLOCK = 64
_STATUS = {0: "CHORUS_OK", 1: "CHORUS_ERR_INVALID_ARG", 2: "CHORUS_ERR_UNSUPPORTED",
           3: "CHORUS_ERR_CAPACITY", 4: "CHORUS_ERR_HIP", 5: "CHORUS_ERR_WORKSPACE"}


class Shape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("S", ctypes.c_int32), ("H", ctypes.c_int32),
                ("D", ctypes.c_int32)]


class Tensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("stride_b", ctypes.c_int64),
                ("stride_s", ctypes.c_int64), ("stride_h", ctypes.c_int64)]


class Mask(ctypes.Structure):
    _fields_ = [("mask_batch", ctypes.c_int32), ("H", ctypes.c_int32),
                ("n_blocks", ctypes.c_int32), ("block", ctypes.c_int32),
                ("row_ptr", ctypes.c_void_p), ("col_idx", ctypes.c_void_p)]


class Schedule(ctypes.Structure):
    _fields_ = [("order", ctypes.c_void_p), ("n_units", ctypes.c_int32)]


class KeyScale(ctypes.Structure):
    _fields_ = [("n_first", ctypes.c_int32), ("beta", ctypes.c_float)]


def _key_scale(key_scale):
    """(n_first, beta) -> pointer to a chorus_key_scale, None -> NULL."""
    if key_scale is None:
        return None
    n_first, beta = key_scale
    return ctypes.byref(KeyScale(int(n_first), float(beta)))


EXPORTS = [
    "chorus_build_block_mask_workspace_size", "chorus_build_block_mask", "chorus_build_block_mask_fp8",
    "chorus_build_block_mask_noalloc", "chorus_build_block_mask_from_sums",
    "chorus_plan_workspace_size", "chorus_plan_block_mask", "chorus_validate_block_mask",
    "chorus_quantize_fp8_blockwise", "chorus_quantize_fp8_blockwise_sums", "chorus_attn_workspace_size",
    "chorus_block_sparse_attn_fwd", "chorus_block_sparse_attn_fwd_f16",
    "chorus_block_sparse_attn_fwd_bf16", "chorus_block_sparse_attn_fwd_fp8",
    "chorus_attn_block_mass", "chorus_select_block_mask_workspace_size", "chorus_select_block_mask",
    "chorus_mask_coverage",
    "chorus_visit_map_bytes", "chorus_visit_reset", "chorus_visit_update",
    "chorus_visit_refresh_workspace_size", "chorus_visit_refresh",
    "chorus_status_string", "chorus_last_error", "chorus_version",
]

_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libchorus.so (once) and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2606_25040_amd.build` "
                           "(or __graft_entry__.build())")
    L = ctypes.CDLL(path)
    P, VP, I32, I64, F32, F64, SZ = (ctypes.POINTER, ctypes.c_void_p, ctypes.c_int32,
                                    ctypes.c_int64, ctypes.c_float, ctypes.c_double, ctypes.c_size_t)
    sig = {
        "chorus_build_block_mask_workspace_size": (SZ, [P(Shape)]),
        "chorus_build_block_mask": (I32, [I32, P(Shape), P(Tensor), P(Tensor), F64, F64, F64, I32,
                                          P(KeyScale), VP, VP, I64, VP, VP, SZ, VP]),
        "chorus_build_block_mask_fp8": (I32, [P(Shape), P(Tensor), VP, P(Tensor), VP, F64, F64, F64, I32,
                                              P(KeyScale), VP, VP, I64, VP, VP, SZ, VP]),
        "chorus_build_block_mask_noalloc": (I32, [I32, P(Shape), P(Tensor), P(Tensor), F64, F64, F64, I32,
                                                  P(KeyScale), VP, VP, I64, VP, VP]),
        "chorus_build_block_mask_from_sums": (I32, [P(Shape), VP, VP, F64, F64, F64, I32, VP, VP, I64, VP,
                                                    VP, SZ, VP]),
        "chorus_plan_workspace_size": (SZ, [P(Shape), P(Mask)]),
        "chorus_plan_block_mask": (I32, [P(Shape), P(Mask), VP, VP, SZ, VP]),
        "chorus_validate_block_mask": (I32, [P(Mask), I64, VP, VP]),
        "chorus_quantize_fp8_blockwise": (I32, [I32, P(Shape), P(Tensor), P(Tensor), VP, VP]),
        "chorus_quantize_fp8_blockwise_sums": (I32, [I32, P(Shape), P(Tensor), P(Tensor), VP, P(KeyScale), VP,
                                                     VP]),
        "chorus_attn_workspace_size": (SZ, [I32, P(Shape), P(Mask)]),
        "chorus_block_sparse_attn_fwd": (I32, [I32, P(Shape), P(Tensor), P(Tensor), P(Tensor), VP,
                                               VP, VP, P(Mask), P(Schedule), F32, P(KeyScale),
                                               P(Tensor), VP, VP, SZ, VP]),
        "chorus_block_sparse_attn_fwd_f16": (I32, [P(Shape), P(Tensor), P(Tensor), P(Tensor),
                                                   P(Mask), P(Schedule), F32, P(KeyScale),
                                                   P(Tensor), VP, VP, SZ, VP]),
        "chorus_block_sparse_attn_fwd_bf16": (I32, [P(Shape), P(Tensor), P(Tensor), P(Tensor),
                                                    P(Mask), P(Schedule), F32, P(KeyScale),
                                                    P(Tensor), VP, VP, SZ, VP]),
        "chorus_block_sparse_attn_fwd_fp8": (I32, [P(Shape), P(Tensor), P(Tensor), P(Tensor), VP,
                                                   VP, VP, P(Mask), P(Schedule), F32, P(KeyScale),
                                                   P(Tensor), VP, VP, SZ, VP]),
        "chorus_attn_block_mass": (I32, [I32, P(Shape), P(Tensor), P(Tensor), VP, F32, I32,
                                         P(KeyScale), VP, VP]),
        "chorus_select_block_mask_workspace_size": (SZ, [P(Shape)]),
        "chorus_select_block_mask": (I32, [P(Shape), VP, I32, F64, F64, VP, VP, I64, VP, SZ, VP]),
        "chorus_mask_coverage": (I32, [P(Shape), P(Mask), VP, VP, VP]),
        "chorus_visit_map_bytes": (SZ, [P(Mask)]),
        "chorus_visit_reset": (I32, [P(Mask), VP, VP]),
        "chorus_visit_update": (I32, [P(Mask), VP, VP]),
        "chorus_visit_refresh_workspace_size": (SZ, [P(Mask)]),
        "chorus_visit_refresh": (I32, [P(Mask), VP, VP, VP, I64, VP, SZ, VP]),
        "chorus_status_string": (ctypes.c_char_p, [I32]),
        "chorus_last_error": (ctypes.c_char_p, []),
        "chorus_version": (I32, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _check(status: int, what: str) -> None:
    if status != 0:
        L = load_library()
        raise RuntimeError(f"{what} failed: {_STATUS.get(status, status)}: "
                           f"{L.chorus_last_error().decode()}")


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float16:
        return F16
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.uint8:
        return FP8_E4M3
    raise TypeError(f"unsupported dtype {t.dtype}")


def _tensor(t: torch.Tensor) -> Tensor:
    if t.dim() != 4:
        raise ValueError("expected a [B, S, H, D] tensor")
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if t.stride(3) != 1:
        raise ValueError("head dim must be contiguous")
    return Tensor(t.data_ptr(), t.stride(0), t.stride(1), t.stride(2))


def _shape(t: torch.Tensor) -> Shape:
    B, S, H, D = t.shape
    return Shape(B, S, H, D)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _workspace(nbytes: int, device) -> torch.Tensor | None:
    if nbytes == 0:
        return None
    return torch.empty(nbytes + 256, dtype=torch.uint8, device=device)


def _aligned(ws: torch.Tensor | None) -> int | None:
    if ws is None:
        return None
    p = ws.data_ptr()
    return (p + 255) // 256 * 256


@dataclass
class BlockMask:
    """CSR block mask on device (rows (b_m * H + h) * n_blocks + i, ascending ids)."""
    row_ptr: torch.Tensor      # int32 [mask_batch * H * n_blocks + 1]
    col_idx: torch.Tensor      # int32 [capacity]
    mask_batch: int
    H: int
    n_blocks: int
    block: int = BLOCK
    block_scores: torch.Tensor | None = None

    @property
    def rows(self) -> int:
        return self.mask_batch * self.H * self.n_blocks

    @property
    def n_kv(self) -> int:
        """Columns: kv blocks of ``block`` tokens per row."""
        return (self.n_blocks * BLOCK + self.block - 1) // self.block

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1].item())

    @property
    def density(self) -> float:
        return self.nnz / float(self.rows * self.n_kv)

    def as_c(self) -> Mask:
        return Mask(self.mask_batch, self.H, self.n_blocks, self.block, self.row_ptr.data_ptr(),
                    self.col_idx.data_ptr())

    def to_host(self):
        """(row_ptr, col_idx[:nnz]) as int64 numpy arrays."""
        rp = self.row_ptr.cpu().numpy().astype("int64")
        return rp, self.col_idx[: int(rp[-1])].cpu().numpy().astype("int64")

    @staticmethod
    def from_host(row_ptr, col_idx, mask_batch: int, H: int, n_blocks: int, device="cuda",
                  block: int = BLOCK):
        rp = torch.as_tensor(row_ptr, dtype=torch.int32).to(device)
        ci = torch.as_tensor(col_idx, dtype=torch.int32)
        if ci.numel() == 0:
            ci = torch.zeros(1, dtype=torch.int32)
        return BlockMask(rp, ci.to(device), mask_batch, H, n_blocks, block)


def build_block_mask(q: torch.Tensor, k: torch.Tensor, top_p: float, min_top_k: float,
                     sm_scale: float | None = None, return_scores: bool = False,
                     out: BlockMask | None = None, workspace: torch.Tensor | None = None,
                     key_scale=None, scales=None, kv_block: int = BLOCK) -> BlockMask:
    """chorus_build_block_mask: one mask per request of ``q, k [B, S, H, D]``;
    ``key_scale = (n_first, beta)`` pools the first-frame-enhanced keys.  For
    fp8 codes (uint8) pass ``scales = (q_scale, k_scale)`` from the quantiser
    (chorus_build_block_mask_fp8).  ``kv_block`` = 64 or 128 tokens per kv
    block (the mask's columns)."""
    L = load_library()
    if q.shape != k.shape or q.dtype != k.dtype:
        raise ValueError("q and k must share shape and dtype")
    fp8 = q.dtype == torch.uint8
    if fp8 != (scales is not None):
        raise ValueError("scales are given exactly for fp8 codes")
    B, S, H, D = q.shape
    n = (S + BLOCK - 1) // BLOCK
    nk = (S + kv_block - 1) // kv_block
    rows = B * H * n
    shape = _shape(q)
    sm = 1.0 / math.sqrt(D) if sm_scale is None else float(sm_scale)
    if out is None:
        out = BlockMask(torch.empty(rows + 1, dtype=torch.int32, device=q.device),
                        torch.empty(rows * nk, dtype=torch.int32, device=q.device), B, H, n, kv_block)
    out.block = kv_block
    if return_scores and (out.block_scores is None or out.block_scores.shape != (rows, nk)):
        out.block_scores = torch.empty((rows, nk), dtype=torch.float32, device=q.device)
    need = L.chorus_build_block_mask_workspace_size(ctypes.byref(shape))
    if workspace is None or workspace.numel() < need + 256:
        workspace = _workspace(need, q.device)
    tail = (sm, float(top_p), float(min_top_k), int(kv_block), _key_scale(key_scale), out.row_ptr.data_ptr(),
            out.col_idx.data_ptr(), out.col_idx.numel(),
            _ptr(out.block_scores if return_scores else None), _aligned(workspace), need, _stream())
    if fp8:
        st = L.chorus_build_block_mask_fp8(ctypes.byref(shape), ctypes.byref(_tensor(q)),
                                           scales[0].data_ptr(), ctypes.byref(_tensor(k)),
                                           scales[1].data_ptr(), *tail)
        _check(st, "chorus_build_block_mask_fp8")
    else:
        st = L.chorus_build_block_mask(_dtype_code(q), ctypes.byref(shape), ctypes.byref(_tensor(q)),
                                       ctypes.byref(_tensor(k)), *tail)
        _check(st, "chorus_build_block_mask")
    return out


def build_block_mask_noalloc(q: torch.Tensor, k: torch.Tensor, top_p: float, min_top_k: float, out: BlockMask,
                             sm_scale: float | None = None, key_scale=None, kv_block: int = BLOCK,
                             block_scores: torch.Tensor | None = None) -> BlockMask:
    """chorus_build_block_mask_noalloc: the builder on f16 / bf16 ``q, k`` with
    the library's own fixed scratch; the caller passes the output mask
    buffers (``out``, and ``block_scores`` [rows, n_kv] fp32 to receive the
    scores) so that nothing is allocated."""
    L = load_library()
    if q.shape != k.shape or q.dtype != k.dtype:
        raise ValueError("q and k must share shape and dtype")
    B, S, H, D = q.shape
    sm = 1.0 / math.sqrt(D) if sm_scale is None else float(sm_scale)
    out.block = kv_block
    out.block_scores = block_scores
    st = L.chorus_build_block_mask_noalloc(_dtype_code(q), ctypes.byref(_shape(q)), ctypes.byref(_tensor(q)),
                                           ctypes.byref(_tensor(k)), sm, float(top_p), float(min_top_k),
                                           int(kv_block), _key_scale(key_scale), out.row_ptr.data_ptr(),
                                           out.col_idx.data_ptr(), out.col_idx.numel(), _ptr(block_scores),
                                           _stream())
    _check(st, "chorus_build_block_mask_noalloc")
    return out


def plan_block_mask(mask: BlockMask, B: int, S: int, out: torch.Tensor | None = None,
                    workspace: torch.Tensor | None = None) -> torch.Tensor:
    """chorus_plan_block_mask: (request, head) unit order for applying ``mask``
    to B requests (int32 [B * H])."""
    L = load_library()
    shape = Shape(B, S, mask.H, 128)
    cm = mask.as_c()
    order = out if out is not None else torch.empty(B * mask.H, dtype=torch.int32,
                                                    device=mask.row_ptr.device)
    need = L.chorus_plan_workspace_size(ctypes.byref(shape), ctypes.byref(cm))
    ws = workspace if workspace is not None and workspace.numel() >= need + 256 else \
        _workspace(need, mask.row_ptr.device)
    st = L.chorus_plan_block_mask(ctypes.byref(shape), ctypes.byref(cm), order.data_ptr(),
                                  _aligned(ws), need, _stream())
    _check(st, "chorus_plan_block_mask")
    return order


def validate_block_mask(mask: BlockMask) -> int:
    """chorus_validate_block_mask; synchronises and returns the flag word (0 = valid)."""
    L = load_library()
    flags = torch.empty(1, dtype=torch.int32, device=mask.row_ptr.device)
    cm = mask.as_c()
    st = L.chorus_validate_block_mask(ctypes.byref(cm), mask.col_idx.numel(), flags.data_ptr(),
                                      _stream())
    _check(st, "chorus_validate_block_mask")
    return int(flags.item())


def quantize_fp8_blockwise(x: torch.Tensor, codes: torch.Tensor | None = None,
                           scales: torch.Tensor | None = None):
    """chorus_quantize_fp8_blockwise: returns (codes uint8 [B,S,H,D], scales fp32 [B,H,n])."""
    L = load_library()
    B, S, H, D = x.shape
    n = (S + BLOCK - 1) // BLOCK
    if codes is None:
        codes = torch.empty((B, S, H, D), dtype=torch.uint8, device=x.device)
    if scales is None:
        scales = torch.empty((B, H, n), dtype=torch.float32, device=x.device)
    st = L.chorus_quantize_fp8_blockwise(_dtype_code(x), ctypes.byref(_shape(x)),
                                         ctypes.byref(_tensor(x)), ctypes.byref(_tensor(codes)),
                                         scales.data_ptr(), _stream())
    _check(st, "chorus_quantize_fp8_blockwise")
    return codes, scales


def quantize_fp8_blockwise_sums(x: torch.Tensor, codes: torch.Tensor | None = None,
                                scales: torch.Tensor | None = None, block_sums: torch.Tensor | None = None,
                                key_scale=None):
    """chorus_quantize_fp8_blockwise_sums: returns (codes, scales, block_sums float64 [B, H, n, 128]),
    the sums over each 64-token block's valid tokens (first-frame tokens times
    beta when ``key_scale = (n_first, beta)``)."""
    L = load_library()
    B, S, H, D = x.shape
    n = (S + BLOCK - 1) // BLOCK
    if codes is None:
        codes = torch.empty((B, S, H, D), dtype=torch.uint8, device=x.device)
    if scales is None:
        scales = torch.empty((B, H, n), dtype=torch.float32, device=x.device)
    if block_sums is None:
        block_sums = torch.empty((B, H, n, D), dtype=torch.float64, device=x.device)
    elif block_sums.shape != (B, H, n, D) or block_sums.dtype != torch.float64 or not block_sums.is_contiguous():
        raise ValueError(f"block_sums must be a contiguous float64 [{B}, {H}, {n}, {D}] tensor")
    st = L.chorus_quantize_fp8_blockwise_sums(_dtype_code(x), ctypes.byref(_shape(x)),
                                              ctypes.byref(_tensor(x)), ctypes.byref(_tensor(codes)),
                                              scales.data_ptr(), _key_scale(key_scale),
                                              block_sums.data_ptr(), _stream())
    _check(st, "chorus_quantize_fp8_blockwise_sums")
    return codes, scales, block_sums


def build_block_mask_from_sums(q_sums: torch.Tensor, k_sums: torch.Tensor, S: int, top_p: float,
                               min_top_k: float, sm_scale: float | None = None, return_scores: bool = False,
                               out: BlockMask | None = None, workspace: torch.Tensor | None = None,
                               kv_block: int = BLOCK) -> BlockMask:
    """chorus_build_block_mask_from_sums: the mask of sequence length ``S``
    from the quantiser's float64 block sums ``[B, H, n, 128]`` of Q and K."""
    L = load_library()
    if q_sums.shape != k_sums.shape or q_sums.dim() != 4:
        raise ValueError("q_sums and k_sums must share one [B, H, n, D] shape")
    for t in (q_sums, k_sums):
        if t.dtype != torch.float64 or not t.is_contiguous():
            raise ValueError("block sums must be contiguous float64")
    B, H, n, D = q_sums.shape
    if n != (S + BLOCK - 1) // BLOCK:
        raise ValueError(f"block sums hold {n} blocks, S = {S} needs {(S + BLOCK - 1) // BLOCK}")
    nk = (S + kv_block - 1) // kv_block
    rows = B * H * n
    shape = Shape(B, S, H, D)
    sm = 1.0 / math.sqrt(D) if sm_scale is None else float(sm_scale)
    dev = q_sums.device
    if out is None:
        out = BlockMask(torch.empty(rows + 1, dtype=torch.int32, device=dev),
                        torch.empty(rows * nk, dtype=torch.int32, device=dev), B, H, n, kv_block)
    out.block = kv_block
    if return_scores and (out.block_scores is None or out.block_scores.shape != (rows, nk)):
        out.block_scores = torch.empty((rows, nk), dtype=torch.float32, device=dev)
    need = L.chorus_build_block_mask_workspace_size(ctypes.byref(shape))
    if workspace is None or workspace.numel() < need + 256:
        workspace = _workspace(need, dev)
    st = L.chorus_build_block_mask_from_sums(ctypes.byref(shape), q_sums.data_ptr(), k_sums.data_ptr(), sm,
                                             float(top_p), float(min_top_k), int(kv_block), out.row_ptr.data_ptr(),
                                             out.col_idx.data_ptr(), out.col_idx.numel(),
                                             _ptr(out.block_scores if return_scores else None),
                                             _aligned(workspace), need, _stream())
    _check(st, "chorus_build_block_mask_from_sums")
    return out


def block_sparse_attn_fwd(q, k, v, mask: BlockMask | None, sm_scale: float | None = None,
                          scales=None, out: torch.Tensor | None = None, return_lse: bool = False,
                          schedule: torch.Tensor | None = None, key_scale=None):
    """chorus_block_sparse_attn_fwd (dtype taken from q: f16, bf16 or uint8 fp8 codes).

    ``scales`` = (q_scale, k_scale, v_scale) for fp8 codes; ``mask=None`` runs
    every block pair (dense attention); ``key_scale = (n_first, beta)`` applies
    the first-frame key enhancement.  Returns ``out`` (and ``lse [B, H, S]``
    fp32 when ``return_lse``).
    """
    L = load_library()
    dt = _dtype_code(q)
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError("q, k and v must share shape and dtype")
    B, S, H, D = q.shape
    sm = 1.0 / math.sqrt(D) if sm_scale is None else float(sm_scale)
    odt = torch.bfloat16 if dt == FP8_E4M3 else q.dtype
    if out is None:
        out = torch.empty((B, S, H, D), dtype=odt, device=q.device)
    elif out.shape != q.shape or out.dtype != odt:
        raise ValueError(f"out must be a {odt} tensor of q's shape")
    lse = torch.empty((B, H, S), dtype=torch.float32, device=q.device) if return_lse else None
    qs = ks = vs = None
    if dt == FP8_E4M3:
        if scales is None:
            raise ValueError("fp8 attention needs (q_scale, k_scale, v_scale)")
        qs, ks, vs = (s.data_ptr() for s in scales)
    shape = _shape(q)
    cm = ctypes.byref(mask.as_c()) if mask is not None else None
    sched = None
    if schedule is not None:
        sched = ctypes.byref(Schedule(schedule.data_ptr(), schedule.numel()))
    need = L.chorus_attn_workspace_size(dt, ctypes.byref(shape), cm)
    ws = _workspace(need, q.device)
    st = L.chorus_block_sparse_attn_fwd(dt, ctypes.byref(shape), ctypes.byref(_tensor(q)),
                                        ctypes.byref(_tensor(k)), ctypes.byref(_tensor(v)), qs, ks,
                                        vs, cm, sched, sm, _key_scale(key_scale),
                                        ctypes.byref(_tensor(out)),
                                        _ptr(lse), _aligned(ws), need, _stream())
    _check(st, "chorus_block_sparse_attn_fwd")
    return (out, lse) if return_lse else out


def block_sparse_attn_fwd_f16(q, k, v, mask, **kw):
    assert q.dtype == torch.float16
    return block_sparse_attn_fwd(q, k, v, mask, **kw)


def block_sparse_attn_fwd_bf16(q, k, v, mask, **kw):
    assert q.dtype == torch.bfloat16
    return block_sparse_attn_fwd(q, k, v, mask, **kw)


def block_sparse_attn_fwd_fp8(q, k, v, q_scale, k_scale, v_scale, mask, **kw):
    assert q.dtype == torch.uint8
    return block_sparse_attn_fwd(q, k, v, mask, scales=(q_scale, k_scale, v_scale), **kw)


def attn_block_mass(q: torch.Tensor, k: torch.Tensor, lse: torch.Tensor, sm_scale: float | None = None,
                    out: torch.Tensor | None = None, key_scale=None, kv_block: int = BLOCK) -> torch.Tensor:
    """chorus_attn_block_mass: true block attention mass [B, H, n, n_kv]
    (fp32) of ``q, k [B, S, H, D]`` given the dense attention's ``lse [B, H, S]``
    (computed with the same ``key_scale``); kv blocks of ``kv_block`` tokens."""
    L = load_library()
    if q.shape != k.shape or q.dtype != k.dtype:
        raise ValueError("q and k must share shape and dtype")
    B, S, H, D = q.shape
    n = (S + 63) // 64
    if lse.shape != (B, H, S) or lse.dtype != torch.float32 or not lse.is_contiguous():
        raise ValueError("lse must be a contiguous float32 [B, H, S] tensor")
    sm = (1.0 / math.sqrt(D)) if sm_scale is None else sm_scale
    nk = (S + kv_block - 1) // kv_block
    mass = out if out is not None else torch.empty((B, H, n, nk), dtype=torch.float32, device=q.device)
    if mass.shape != (B, H, n, nk) or mass.dtype != torch.float32 or not mass.is_contiguous():
        raise ValueError("out must be a contiguous float32 [B, H, n, n_kv] tensor")
    st = L.chorus_attn_block_mass(_dtype_code(q), ctypes.byref(_shape(q)), ctypes.byref(_tensor(q)),
                                  ctypes.byref(_tensor(k)), lse.data_ptr(), sm, int(kv_block),
                                  _key_scale(key_scale),
                                  mass.data_ptr(), _stream())
    _check(st, "chorus_attn_block_mass")
    return mass


def select_block_mask(mass: torch.Tensor, S: int, top_p: float, min_top_k: float,
                      out: BlockMask | None = None, workspace: torch.Tensor | None = None,
                      kv_block: int = BLOCK) -> BlockMask:
    """chorus_select_block_mask: CSR mask (mask_batch = B) cut from block
    masses ``mass [B, H, n, n_kv]`` of a sequence of S tokens."""
    L = load_library()
    B, H, n, nk = mass.shape
    if (n != (S + 63) // 64 or nk != (S + kv_block - 1) // kv_block or mass.dtype != torch.float32
            or not mass.is_contiguous()):
        raise ValueError("mass must be a contiguous float32 [B, H, ceil(S / 64), ceil(S / kv_block)] tensor")
    shape = Shape(B, S, H, 128)
    rows = B * H * n
    m = out if out is not None else BlockMask(
        torch.empty(rows + 1, dtype=torch.int32, device=mass.device),
        torch.empty(rows * nk, dtype=torch.int32, device=mass.device), B, H, n, kv_block)
    m.block = kv_block
    need = L.chorus_select_block_mask_workspace_size(ctypes.byref(shape))
    ws = workspace if workspace is not None and workspace.numel() >= need + 256 else \
        _workspace(need, mass.device)
    st = L.chorus_select_block_mask(ctypes.byref(shape), mass.data_ptr(), int(kv_block), top_p, min_top_k,
                                    m.row_ptr.data_ptr(), m.col_idx.data_ptr(), m.col_idx.numel(),
                                    _aligned(ws), need, _stream())
    _check(st, "chorus_select_block_mask")
    return m


def mask_coverage(mask: BlockMask, mass: torch.Tensor, S: int) -> torch.Tensor:
    """chorus_mask_coverage: coverage [B, H] (float64) of ``mask`` on the
    requests whose block masses are ``mass [B, H, n, n]``."""
    L = load_library()
    B, H, n, _ = mass.shape
    if mass.dtype != torch.float32 or not mass.is_contiguous():
        raise ValueError("mass must be a contiguous float32 tensor")
    cov = torch.empty((B, H), dtype=torch.float64, device=mass.device)
    cm = mask.as_c()
    st = L.chorus_mask_coverage(ctypes.byref(Shape(B, S, H, 128)), ctypes.byref(cm), mass.data_ptr(),
                                cov.data_ptr(), _stream())
    _check(st, "chorus_mask_coverage")
    return cov


class VisitMap:
    """Device visited bitmap of a layer group (chorus_visit_*), sized for
    masks with the given mask_batch / H / n_blocks."""

    def __init__(self, mask_batch: int, H: int, n_blocks: int, device="cuda", block: int = BLOCK):
        L = load_library()
        desc = Mask(mask_batch, H, n_blocks, block, None, None)
        nbytes = L.chorus_visit_map_bytes(ctypes.byref(desc))
        if nbytes == 0:
            raise ValueError("invalid mask description for a visited map")
        self.mask_batch, self.H, self.n_blocks, self.block = mask_batch, H, n_blocks, block
        self.n_kv = (n_blocks * BLOCK + block - 1) // block
        self.words = (self.n_kv + 31) // 32
        self.bits = torch.empty(nbytes // 4, dtype=torch.int32, device=device)

    def _check_mask(self, mask: BlockMask):
        if (mask.mask_batch, mask.H, mask.n_blocks, mask.block) != (self.mask_batch, self.H, self.n_blocks,
                                                                    self.block):
            raise ValueError("mask dimensions differ from the visited map's")

    def reset(self, like: BlockMask):
        self._check_mask(like)
        st = load_library().chorus_visit_reset(ctypes.byref(like.as_c()), self.bits.data_ptr(), _stream())
        _check(st, "chorus_visit_reset")

    def update(self, mask: BlockMask):
        self._check_mask(mask)
        st = load_library().chorus_visit_update(ctypes.byref(mask.as_c()), self.bits.data_ptr(), _stream())
        _check(st, "chorus_visit_update")

    def refresh(self, mask: BlockMask, out: BlockMask | None = None,
                workspace: torch.Tensor | None = None) -> BlockMask:
        """The group's last-layer mask: mask | (pairs not visited)."""
        self._check_mask(mask)
        L = load_library()
        rows = mask.rows
        m = out if out is not None else BlockMask(
            torch.empty(rows + 1, dtype=torch.int32, device=self.bits.device),
            torch.empty(rows * mask.n_kv, dtype=torch.int32, device=self.bits.device), mask.mask_batch, mask.H,
            mask.n_blocks, mask.block)
        cm = mask.as_c()
        need = L.chorus_visit_refresh_workspace_size(ctypes.byref(cm))
        ws = workspace if workspace is not None and workspace.numel() >= need + 256 else \
            _workspace(need, self.bits.device)
        st = L.chorus_visit_refresh(ctypes.byref(cm), self.bits.data_ptr(), m.row_ptr.data_ptr(),
                                    m.col_idx.data_ptr(), m.col_idx.numel(), _aligned(ws), need, _stream())
        _check(st, "chorus_visit_refresh")
        return m

    def to_host(self):
        """Boolean [rows, n_blocks] numpy view of the map."""
        import numpy as np
        w = self.bits.cpu().numpy().view(np.uint32).reshape(-1, self.words)
        bits = ((w[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).astype(bool)
        return bits.reshape(w.shape[0], -1)[:, : self.n_kv]
