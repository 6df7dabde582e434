"""Pins for the FP8 e4m3fn codec and blockwise quantiser oracle (CPU only).

Checked against torch's float8_e4m3fn cast (library routine, round to nearest
even; clamped first because it maps values above 464 to NaN), a brute-force
nearest-value search over the decode table, and the format's error bound.
"""

import numpy as np
import pytest
import torch

from oracle import fp8 as of


def torch_encode(x32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.clip(x32, -448, 448).astype(np.float32))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_table_matches_torch():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    tab = of.decode_table()
    assert np.array_equal(np.isnan(ref), np.isnan(tab))
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(tab[ok], ref[ok])
    assert np.nanmax(tab) == 448.0 and np.nanmin(np.abs(tab[tab != 0])) == 2.0 ** -9


def test_encode_matches_torch_on_all_bf16_values():
    bits = np.arange(65536, dtype=np.uint32) << 16
    x = bits.view(np.float32)
    x = x[np.isfinite(x) & (np.abs(x) <= 448)]
    np.testing.assert_array_equal(of.encode_rne(x), torch_encode(x))


def test_encode_matches_torch_on_random_and_tie_values(rng):
    mags = np.exp2(rng.uniform(-14, 8.8, size=200000)).astype(np.float32)
    x = np.where(rng.random(200000) < 0.5, -mags, mags).astype(np.float32)
    x = x[np.abs(x) <= 448]
    np.testing.assert_array_equal(of.encode_rne(x), torch_encode(x))
    tab = of.decode_table()
    pos = np.sort(tab[np.isfinite(tab) & (tab >= 0)])
    mids = ((pos[:-1] + pos[1:]) / 2).astype(np.float32)      # exact ties in fp32
    for v in (mids, -mids):
        np.testing.assert_array_equal(of.encode_rne(v), torch_encode(v))


def test_encode_is_nearest_with_ties_to_even(rng):
    tab = of.decode_table()
    codes = np.array([c for c in range(256) if np.isfinite(tab[c])])
    vals = tab[codes]
    x = np.concatenate([rng.uniform(-448, 448, 5000), rng.uniform(-0.05, 0.05, 5000)])
    x = x.astype(np.float32).astype(np.float64)
    got = of.encode_rne(x)
    for xi, gi in zip(x, got):
        d = np.abs(vals - xi)
        best = codes[d == d.min()]
        best = best[(best & 0x80) == (0x80 if np.signbit(xi) else 0)] if len(best) > 1 else best
        if len(best) > 1:
            best = best[(best & 1) == 0]                   # tie: even mantissa
        assert gi == best[0] or (xi == 0 and (gi & 0x7F) == 0), (xi, gi, best)


def test_quantize_block_scale_and_codes(rng):
    x = rng.standard_normal((64, 128)).astype(np.float32)
    codes, scale = of.quantize_block(x)
    amax = np.max(np.abs(x))
    assert scale == np.float32(amax / np.float32(448))
    j = np.unravel_index(np.argmax(np.abs(x)), x.shape)
    assert codes[j] & 0x7F == 0x7E                          # |amax| maps to 448
    deq = of.decode(codes) * np.float64(scale)
    y = np.abs(x.astype(np.float64) * (448.0 / amax))
    normal = y >= 2.0 ** -6
    rel = np.abs(deq - x)[normal] / np.abs(x)[normal]
    assert rel.max() <= 2.0 ** -4 * (1 + 1e-6)


def test_quantize_zero_block():
    codes, scale = of.quantize_block(np.zeros((64, 128), np.float32))
    assert scale == 1.0 and np.all(codes == 0)


def test_blockwise_layout_and_dequantize(rng):
    B, S, H, D = 2, 150, 3, 8
    x = (rng.standard_normal((B, S, H, D)) * rng.uniform(0.1, 10, size=(1, 1, H, 1))).astype(
        np.float32)
    x[1, 64:128, 2] = 0
    codes, scales = of.quantize_blockwise(x)
    assert codes.shape == x.shape and scales.shape == (B, H, 3)
    assert scales[1, 2, 1] == 1.0
    for b in range(B):
        for h in range(H):
            for i in range(3):
                rows = slice(i * 64, min(S, i * 64 + 64))
                c, s = of.quantize_block(x[b, rows, h])
                assert np.array_equal(codes[b, rows, h], c) and scales[b, h, i] == s
    deq = of.dequantize_blockwise(codes, scales)
    np.testing.assert_array_equal(deq[0, 70, 1], of.decode(codes[0, 70, 1]) * float(scales[0, 1, 1]))
    assert np.max(np.abs(deq - x)) <= np.max(np.abs(x)) * 2.0 ** -4


def test_quantize_power_of_two_block_hand_codes():
    # amax = 56 = 448 / 8, so inv = 8 and scale = 1/8 exactly; each value below
    # lands, after x8, exactly on an e4m3 grid point or on a midpoint.
    x = np.zeros((64, 128), np.float32)
    cases = {
        (0, 0): (56.0, 0x7E),                    # 448 -> S.1111.110
        (0, 1): (-56.0, 0xFE),
        (1, 0): (1.1875 / 8, 0x3A),              # midpoint 1.125|1.25 -> even mantissa 1.25
        (1, 1): (1.0625 / 8, 0x38),              # midpoint 1.0|1.125 -> even mantissa 1.0
        (1, 2): (-1.3125 / 8, 0xBA),             # midpoint 1.25|1.375 -> 1.25
        (2, 0): (1.5 * 2.0 ** -9 / 8, 0x02),     # subnormal midpoint 1|2 (x 2^-9) -> 2
        (2, 1): (0.5 * 2.0 ** -9 / 8, 0x00),     # half the smallest subnormal -> 0 (even)
        (2, 2): (2.0 ** -6 / 8, 0x08),           # smallest normal
        (3, 0): (416.0 / 8, 0x7D),               # 416 = 1.625 * 2^8
        (3, 1): (432.0 / 8, 0x7E),               # midpoint 416|448 -> even (448)
    }
    for (r, c), (val, _) in cases.items():
        x[r, c] = val
    codes, scale = of.quantize_block(x)
    assert scale == np.float32(0.125)
    for (r, c), (_, code) in cases.items():
        assert codes[r, c] == code, (r, c, hex(codes[r, c]), hex(code))


def test_quantize_scale_is_correctly_rounded(rng):
    for _ in range(3000):
        x = (rng.standard_normal((4, 16)) * np.exp2(rng.uniform(-20, 20))).astype(np.float32)
        _, scale = of.quantize_block(x)
        exact = float(np.max(np.abs(x.astype(np.float64)))) / 448.0
        half_ulp = np.spacing(np.float32(scale)) / 2
        assert abs(float(scale) - exact) <= half_ulp


@pytest.mark.parametrize("k", [0, 40, 70, 123])
def test_quantize_codes_are_invariant_under_power_of_two_scaling(rng, k):
    """The codes depend on x / amax only: a block scaled by 2^-k (exactly
    representable in bf16 down to 2^-126) gets the codes of the
    unscaled block and a scale 2^-k times its scale (the nearest fp32 to
    amax / 448 once that is subnormal), including blocks below
    amax = 448 / FLT_MAX ~ 1.3e-36, where a plain fp32 448 / amax overflows."""
    x = (rng.standard_normal((64, 128)) * 2.0).astype(np.float32)
    x = np.where(np.abs(x) < 2.0 ** -3, np.float32(2.0 ** -3), x)
    x = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    c0, s0 = of.quantize_block(x)
    xs = (x.astype(np.float64) * 2.0 ** -k).astype(np.float32)
    assert np.array_equal(xs.astype(np.float64) * 2.0 ** k, x.astype(np.float64))   # exact scaling
    c1, s1 = of.quantize_block(xs)
    assert np.array_equal(c1, c0)
    exact = float(np.max(np.abs(xs))) / 448.0
    if exact >= float(np.finfo(np.float32).tiny):
        assert np.float64(s1) == np.float64(s0) * 2.0 ** -k
    else:
        # subnormal scale: still the nearest fp32 to amax / 448
        assert abs(float(s1) - exact) <= 2.0 ** -150
    if k >= 123:
        assert float(np.max(np.abs(xs))) < 448.0 / float(np.finfo(np.float32).max)
