"""Oracle: OCP FP8 e4m3fn codec and the blockwise quantiser of the FP8 path.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The paper's default backend runs QK^T and PV in FP8 with high-precision
accumulation (Sec. 3.2, "Efficient block-sparse kernel").  The format is the
OCP e4m3fn encoding (1 sign, 4 exponent bits with bias 7, 3 mantissa bits,
no infinities, only S.1111.111 is NaN, largest finite 448, smallest normal
2^-6, subnormal spacing 2^-9).  Scales are per (request, head, 64-token block)
in fp32.  For one block X of up to 64 x D values:

    amax  = max |x|                      (exact: inputs are 16-bit floats)
    inv   = fp32(448 / amax)             (correctly rounded fp32 divide)
    y     = fp32(x * inv)                (correctly rounded fp32 multiply)
    code  = e4m3fn_rne(clamp(y, -448, 448))
    scale = fp32(amax / 448)

amax == 0 gives inv = 0 (codes encode +-0) and scale = 1.  In a block with
0 < amax < 2^-64, x and amax are first multiplied by 2^64 (exact for 16-bit
inputs): the codes depend on x / amax only, so the scaled form gives the same
codes wherever the plain one is finite, and it keeps 448 / amax finite below
448 / FLT_MAX, where the plain fp32 reciprocal overflows.
The scale stays fp32(amax / 448) of the unscaled amax (subnormal for such
blocks).  The dequantised value the FP8 attention consumes is
code_value * scale (exact in float64).
"""

from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0
BLOCK = 64


def decode_table() -> np.ndarray:
    """float64 value of each of the 256 e4m3fn codes (NaN for 0x7F, 0xFF)."""
    t = np.empty(256, dtype=np.float64)
    for c in range(256):
        sign = -1.0 if c & 0x80 else 1.0
        e = (c >> 3) & 0xF
        m = c & 0x7
        if e == 0xF and m == 0x7:
            t[c] = np.nan
        elif e == 0:
            t[c] = sign * (m / 8.0) * 2.0 ** -6
        else:
            t[c] = sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return t


_TABLE = decode_table()


def decode(codes) -> np.ndarray:
    return _TABLE[np.asarray(codes, dtype=np.uint8)]


def encode_rne(x) -> np.ndarray:
    """Round finite values with |x| <= 448 to e4m3fn, ties to even mantissa.

    Uses the format's definition directly: below 2^-6 the grid spacing is
    2^-9; in binade [2^e, 2^(e+1)) it is 2^(e-3).
    """
    x = np.asarray(x, dtype=np.float64)
    if np.any(~np.isfinite(x)) or np.any(np.abs(x) > E4M3_MAX):
        raise ValueError("encode_rne expects finite values within +-448")
    sign = np.signbit(x).astype(np.uint8) << 7
    a = np.abs(x)
    code = np.zeros(a.shape, dtype=np.int64)
    sub = a < 2.0 ** -6
    # subnormal range: multiples of 2^-9; rounding up to 8 gives the code of 2^-6
    code[sub] = np.rint(a[sub] * 2.0 ** 9).astype(np.int64)
    nrm = ~sub
    if np.any(nrm):
        mant, exp2 = np.frexp(a[nrm])          # a = mant * 2^exp2, mant in [0.5, 1)
        e = exp2 - 1                           # a in [2^e, 2^(e+1))
        steps = np.rint(a[nrm] / 2.0 ** (e - 3)).astype(np.int64)   # in [8, 16]
        carry = steps == 16
        e = np.where(carry, e + 1, e)
        steps = np.where(carry, 8, steps)
        code[nrm] = ((e + 7) << 3) | (steps - 8)
    return (code.astype(np.uint8) | sign).astype(np.uint8)


def quantize_block(xb) -> tuple[np.ndarray, np.float32]:
    """Quantise one block (any shape) following the module docstring."""
    xb = np.asarray(xb, dtype=np.float32)
    amax = np.float32(np.max(np.abs(xb))) if xb.size else np.float32(0)
    up = np.float32(2.0 ** 64) if 0 < amax < np.float32(2.0 ** -64) else np.float32(1.0)
    if amax == 0:
        inv = np.float32(0.0)
        scale = np.float32(1.0)
    else:
        inv = np.float32(np.float32(E4M3_MAX) / np.float32(amax * up))
        scale = np.float32(amax / np.float32(E4M3_MAX))
    y = ((xb * up).astype(np.float32) * inv).astype(np.float32)
    y = np.clip(y, np.float32(-E4M3_MAX), np.float32(E4M3_MAX))
    return encode_rne(y), scale


def quantize_blockwise(x, block: int = BLOCK):
    """``x [B, S, H, D]`` (fp16/bf16 values as float32) -> codes, scales.

    codes: uint8 ``[B, S, H, D]``; scales: float32 ``[B, H, n_blocks]``.
    """
    x = np.asarray(x, dtype=np.float32)
    B, S, H, D = x.shape
    n = (S + block - 1) // block
    codes = np.zeros((B, S, H, D), dtype=np.uint8)
    scales = np.zeros((B, H, n), dtype=np.float32)
    for b in range(B):
        for h in range(H):
            for i in range(n):
                rows = slice(i * block, min(i * block + block, S))
                c, s = quantize_block(x[b, rows, h, :])
                codes[b, rows, h, :] = c
                scales[b, h, i] = s
    return codes, scales


def dequantize_blockwise(codes, scales, block: int = BLOCK) -> np.ndarray:
    """Exact float64 values code * scale, ``[B, S, H, D]``."""
    codes = np.asarray(codes, dtype=np.uint8)
    B, S, H, D = codes.shape
    vals = decode(codes)
    tok_block = np.arange(S) // block
    sc = np.asarray(scales, dtype=np.float64)          # [B, H, n]
    per_tok = sc[:, :, tok_block]                       # [B, H, S]
    return vals * np.transpose(per_tok, (0, 2, 1))[..., None]
