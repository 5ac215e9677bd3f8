"""FP8 experts -- TEST INFRASTRUCTURE ONLY.

The paper's inference benchmark runs the experts in FP8 (Section 5.2, the
vLLM prefill runs).  The paper fixes no FP8 scheme; the reading taken here
(listed in the design notes) is W8A8 in the OCP FP8 E4M3 format:

  * every weight matrix row (output channel) and every activation row
    (token or expert row) has its own fp32 scale;
  * a row x is quantised as: amax = max_i |x_i|; for amax > 0,
    scale = fl32(amax / 448) and inv = fl32(448 / amax), each a correctly
    rounded fp32 division; v_i = fl32(x_i * inv), clamped to [-448, 448];
    code_i = E4M3 round-to-nearest-even of v_i.  An all-zero row has scale
    1 and zero codes.  The row is represented by dec(code_i) * scale;
  * a GEMM of quantised operands is sum_k dec(a_mk) dec(b_nk), times
    scale_a[m] * scale_b[n];
  * the SwiGLU expert: X and W quantised as above; gate and up are the
    scaled GEMMs; H = SiLU(gate) * up, rounded to bf16 as in the bf16 path;
    H is quantised per row like X; down is the scaled GEMM of H and W_down.

E4M3 (OCP 8-bit floating point, E4M3 variant): 1 sign bit, 4 exponent bits
with bias 7, 3 mantissa bits; exponent field 0 holds the subnormals
m * 2^-9 (m = 1..7); the largest finite value is 1.75 * 2^8 = 448; there is
no infinity, and S.1111.111 is NaN.

Floating point here is exact: codes decode exactly to fp64; fp32 steps that
decide codes (the scale, the reciprocal, the scaled value) are computed in
fp32, as the kernels compute them.
"""

import numpy as np

from .moe import silu

E4M3_MAX = 448.0


def e4m3_decode_table():
    """fp64 value of every code 0..255 (NaN for 0x7F and 0xFF)."""
    out = np.empty(256, np.float64)
    for c in range(256):
        s = -1.0 if c & 0x80 else 1.0
        e = (c >> 3) & 0xF
        m = c & 0x7
        if e == 0xF and m == 0x7:
            out[c] = np.nan
        elif e == 0:
            out[c] = s * m * 2.0 ** -9
        else:
            out[c] = s * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return out


_DEC = e4m3_decode_table()


def e4m3_decode(codes):
    return _DEC[np.asarray(codes, np.uint8)]


def e4m3_encode(v):
    """E4M3 code of each value, round to nearest, ties to even mantissa;
    magnitudes above the largest finite value give +-448.  v: finite values
    (any float dtype); -0.0 encodes with the sign bit."""
    v = np.asarray(v, np.float64)
    sign = np.signbit(v)
    a = np.abs(v)
    _, E = np.frexp(a)                       # a = f * 2^E, f in [0.5, 1)
    e = np.maximum(E - 1, -6)                # binade, subnormals share 2^-6's spacing
    ulp = np.ldexp(1.0, e - 3)
    r = np.rint(a / ulp)                     # exact quotient; rint rounds half to even
    val = np.minimum(r * ulp, E4M3_MAX)
    _, E2 = np.frexp(val)
    e2 = E2 - 1
    normal = (val >= 2.0 ** -6)
    exp_field = np.where(normal, e2 + 7, 0)
    mant = np.where(normal, val / np.ldexp(1.0, e2 - 3) - 8.0, val / 2.0 ** -9)
    code = (exp_field.astype(np.int64) << 3) | mant.astype(np.int64)
    code = np.where(val == 0, 0, code)
    return (code | (sign.astype(np.int64) << 7)).astype(np.uint8)


def quantize_rows(x):
    """Row-wise E4M3 quantisation (see the module notes).  x: [rows, cols]
    exactly representable in fp32.  Returns (codes uint8 [rows, cols],
    scales float32 [rows])."""
    x32 = np.asarray(x, np.float32)
    amax = np.max(np.abs(x32), axis=1) if x32.shape[1] else np.zeros(x32.shape[0], np.float32)
    pos = amax > 0
    safe = np.where(pos, amax, np.float32(1.0)).astype(np.float32)
    scale = np.where(pos, safe / np.float32(E4M3_MAX), np.float32(1.0)).astype(np.float32)
    inv = np.where(pos, np.float32(E4M3_MAX) / safe, np.float32(0.0)).astype(np.float32)
    v = (x32 * inv[:, None]).astype(np.float32)
    v = np.clip(v, -E4M3_MAX, E4M3_MAX)
    return e4m3_encode(v), scale


def dequantize_rows(codes, scales):
    return e4m3_decode(codes) * np.asarray(scales, np.float64)[:, None]


def scaled_gemm(a_codes, a_scales, b_codes, b_scales):
    """sum_k dec(a_mk) dec(b_nk) * scale_a[m] * scale_b[n] in fp64."""
    return (e4m3_decode(a_codes) @ e4m3_decode(b_codes).T) * np.outer(
        np.asarray(a_scales, np.float64), np.asarray(b_scales, np.float64))


def bf16_round(v):
    """Round fp64/fp32 values to bf16 (to nearest, ties to even) through fp32."""
    u = np.ascontiguousarray(np.asarray(v, np.float32)).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def swiglu_fp8_hidden(x_codes, x_scales, gu_codes, gu_scales):
    """H = SiLU(gate) * up of one expert from quantised operands, rounded to
    bf16.  gu_codes [2F, d]: gate rows [0, F), up rows [F, 2F)."""
    F = gu_codes.shape[0] // 2
    gate = scaled_gemm(x_codes, x_scales, gu_codes[:F], gu_scales[:F])
    up = scaled_gemm(x_codes, x_scales, gu_codes[F:], gu_scales[F:])
    return bf16_round(silu(gate) * up)


def swiglu_fp8(x, gu_codes, gu_scales, dn_codes, dn_scales, h_given=None):
    """One expert's FP8 SwiGLU on rows x: quantise x, gate/up, H (bf16),
    quantise H, down.  h_given: optional (codes, scales) of H to use in
    place of quantising this function's own H (where a different rounding
    of H moved a code across a rounding boundary, a caller takes the other
    side's codes after checking them).  Returns (y fp64 [rows, d], H bf16
    values as fp64, (H codes, H scales))."""
    xq, xs = quantize_rows(x)
    H = swiglu_fp8_hidden(xq, xs, gu_codes, gu_scales)
    hq, hs = quantize_rows(H) if h_given is None else h_given
    return scaled_gemm(hq, hs, dn_codes, dn_scales), H, (hq, hs)
