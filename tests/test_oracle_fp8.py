"""Pins of oracle.fp8 (the FP8 E4M3 experts) against the format's defining
constants, brute force and hand-computed cases."""

import numpy as np
import pytest

import oracle
from oracle import fp8 as of8


def test_e4m3_format_constants():
    # OCP 8-bit floating point, E4M3: bias 7, no infinities, NaN only at
    # S.1111.111; largest 448 = 1.75 * 2^8, smallest normal 2^-6, smallest
    # subnormal 2^-9, 1.0 = 0.0111.000.
    t = of8.e4m3_decode_table()
    assert np.isnan(t[0x7F]) and np.isnan(t[0xFF])
    assert np.isfinite(t).sum() == 254
    assert t[0x7E] == 448.0 and t[0xFE] == -448.0
    assert t[0x08] == 2.0 ** -6 and t[0x07] == 7 * 2.0 ** -9 and t[0x01] == 2.0 ** -9
    assert t[0x38] == 1.0 and t[0x40] == 2.0 and t[0x44] == 3.0 and t[0x3C] == 1.5
    assert t[0x00] == 0.0 and t[0x80] == 0.0 and np.signbit(t[0x80])
    pos = t[0x00:0x7F]
    assert np.all(np.diff(pos) > 0)                      # codes 0..0x7E increase
    assert np.array_equal(t[0x80:0xFF], -pos)            # sign-magnitude


def test_encode_round_trips_every_code():
    t = of8.e4m3_decode_table()
    codes = np.array([c for c in range(256) if np.isfinite(t[c])], np.uint8)
    assert np.array_equal(of8.e4m3_encode(t[codes]), codes)


def _brute(v):
    """Nearest finite E4M3 value by search, ties to the even code (even
    mantissa), magnitudes beyond 448 to 448."""
    t = of8.e4m3_decode_table()
    cands = np.array([c for c in range(0x7F)], np.int64)     # non-negative codes
    a = min(abs(v), 448.0)
    dist = np.abs(t[cands] - a)
    best = cands[dist == dist.min()]
    c = int(best[0]) if len(best) == 1 else int(best[best % 2 == 0][0])
    return c | (0x80 if np.signbit(v) else 0)


def test_encode_matches_brute_force_nearest():
    g = np.random.default_rng(0)
    t = of8.e4m3_decode_table()
    pos = t[1:0x7F]
    mids = (pos[:-1] + pos[1:]) / 2                      # exact ties
    vals = np.concatenate([g.uniform(-500, 500, 3000), g.standard_normal(2000) * 1e-2,
                           mids, -mids, [2.0 ** -10, 3 * 2.0 ** -10, 0.0, -0.0, 464.0, 1e6]])
    vals = vals.astype(np.float32).astype(np.float64)
    got = of8.e4m3_encode(vals)
    want = np.array([_brute(v) for v in vals], np.uint8)
    assert np.array_equal(got, want)


def test_quantize_rows_properties():
    g = np.random.default_rng(1)
    x = (g.standard_normal((6, 64)) * np.exp(g.uniform(-6, 6, (6, 1)))).astype(np.float32)
    x[2] = 0.0
    codes, scales = of8.quantize_rows(x)
    assert scales.dtype == np.float32
    assert np.array_equal(codes[2], np.zeros(64, np.uint8)) and scales[2] == 1.0
    for r in (0, 1, 3, 4, 5):
        amax = np.max(np.abs(x[r]))
        assert scales[r] == np.float32(amax) / np.float32(448.0)
        i = int(np.argmax(np.abs(x[r])))
        assert of8.e4m3_decode(codes[r, i]) == np.copysign(448.0, x[r, i])
        # within half a spacing of E4M3 (relative 2^-4 for normals, 2^-10
        # absolute below 2^-6, in units of the scale)
        deq = of8.dequantize_rows(codes[r:r + 1], scales[r:r + 1])[0]
        bound = np.maximum(np.abs(x[r]) * 2.0 ** -4, 2.0 ** -10 * scales[r]) * 1.0001
        assert np.all(np.abs(deq - x[r]) <= bound)


def test_scaled_gemm_hand_value():
    # codes 2.0 (0x40) and 3.0 (0x44) with 1.5 (0x3C): row [2, 3] . [3, 1.5]
    # = 10.5, times scales 0.5 and 0.25 -> 1.3125
    a = np.array([[0x40, 0x44]], np.uint8)
    b = np.array([[0x44, 0x3C]], np.uint8)
    out = of8.scaled_gemm(a, np.float32([0.5]), b, np.float32([0.25]))
    assert out.shape == (1, 1) and out[0, 0] == 1.3125


def test_bf16_round_hand_values():
    v = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -20, -3.0])
    assert np.array_equal(of8.bf16_round(v), [1.0, 1.0 + 2.0 ** -6, 1.0 + 2.0 ** -7, -3.0])


def test_lossless_quantisation_reduces_to_the_bf16_expert():
    # When every row is an E4M3 grid times a power of two with its amax at
    # 448 times that power, quantisation is exact: the FP8 hidden
    # activation is the SwiGLU hidden activation rounded to bf16.
    g = np.random.default_rng(2)
    t = of8.e4m3_decode_table()
    grid = t[np.isfinite(t)]

    def exact_rows(n, cols, scale_exp):
        m = g.choice(grid, (n, cols))
        m[:, 0] = 448.0
        return m * 2.0 ** scale_exp

    d, F = 16, 8
    x = exact_rows(5, d, -9)
    gu = exact_rows(2 * F, d, -12)
    dn = exact_rows(d, F, -12)
    xq, xs = of8.quantize_rows(x)
    assert np.array_equal(of8.dequantize_rows(xq, xs), x)
    gq, gs = of8.quantize_rows(gu)
    H = of8.swiglu_fp8_hidden(xq, xs, gq, gs)
    gate, up = x @ gu[:F].T, x @ gu[F:].T
    assert np.array_equal(H, of8.bf16_round(oracle.silu(gate) * up))
    # and the full expert then equals the down product of H's quantisation
    dq, ds = of8.quantize_rows(dn)
    y, H2, (hq, hs) = of8.swiglu_fp8(x, gq, gs, dq, ds)
    assert np.array_equal(H2, H)
    assert np.allclose(y, of8.dequantize_rows(hq, hs) @ dn.T, rtol=1e-13, atol=0)
    # its distance from the unquantised expert is the quantisation of H
    ref = oracle.swiglu(x, gu, dn)
    assert np.sqrt(np.mean((y - ref) ** 2)) <= 0.05 * np.sqrt(np.mean(ref ** 2))


@pytest.mark.parametrize("seed", [3, 4])
def test_quantisation_error_bound(seed):
    # Random rows: the dequantised matrix differs from x by at most half an
    # E4M3 spacing per element, so a GEMM of dequantised operands stays
    # within the first-order bound sum |a||b| (2^-4 + 2^-4 + 2^-8).
    g = np.random.default_rng(seed)
    a = g.standard_normal((7, 96)).astype(np.float32)
    b = (0.02 * g.standard_normal((5, 96))).astype(np.float32)
    aq, as_ = of8.quantize_rows(a)
    bq, bs = of8.quantize_rows(b)
    got = of8.scaled_gemm(aq, as_, bq, bs)
    bound = (np.abs(a).astype(np.float64) @ np.abs(b).T) * (2 * 2.0 ** -4 + 2.0 ** -8) + 1e-12
    assert np.all(np.abs(got - a.astype(np.float64) @ b.T.astype(np.float64)) <= bound)
