"""FP8 (OCP E4M3) row quantisation and the scaled FP8 linear layer.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's DiT runs its linear layers in bf16; FP8 is a throughput variant of
those layers, not part of the method, so nothing here follows a passage of the
paper.  The format and the scheme are fixed as follows.

Format: OCP 8-bit floating point E4M3 ("e4m3fn"): sign bit, 4 exponent bits
with bias 7, 3 mantissa bits.  Exponent field 0 holds the subnormals
(m / 8) * 2^-6; fields 1..15 hold (1 + m / 8) * 2^(e - 7), except the code
with all exponent and mantissa bits set, which is NaN (there is no infinity).
The largest finite magnitude is 448 (code 0x7e), the smallest 2^-9 (code 0x01).

Encoding: round to nearest, ties to the even code (the code whose mantissa
bit 0 is clear), in magnitude, then the sign bit; a negative value that rounds
to zero gives 0x80.  Magnitudes at or above 464 (halfway from 448 to the next
binade step) are out of range: the quantiser below never produces them.

Quantisation of a row x (float32 values): amax = max |x|; when amax >= A_MIN =
448 * 2^-126, mult = fl32(448 / amax), codes = encode(fl32(x * mult)) and the
dequantisation scale is d = fl32(amax / 448).  Every float32 step is one IEEE
operation rounded to nearest even, so codes are reproducible bit for bit on any
IEEE machine.  Two kinds of row fall outside that rule, by convention of this
scheme: a row with amax < A_MIN (zero rows included) gets codes 0 and d = 0 (its
entries are below 2^-117, and the bound keeps 448 / amax and amax / 448 finite
and normal); a row holding an infinity or a NaN gets the NaN code 0x7f in every
position and d = NaN.

Linear layer: out[m, n] = epi(d_a[m] * d_w[n] * sum_k dec(A[m, k]) dec(W[n, k])
+ bias[n]) with epi the identity or GELU-tanh.  The sum is formed exactly in
float64: a product of two E4M3 values is a multiple of 2^-18 below 2^18, so
sums of fewer than 2^33 of them stay within float64's 53 bits.
"""
from __future__ import annotations

import numpy as np

MAX_E4M3 = 448.0
A_MIN = np.float32(448.0 * 2.0 ** -126)    # smallest amax quantised; rows below it are zero rows


def decode_table() -> np.ndarray:
    """float64 value of each of the 256 codes (NaN for 0x7f and 0xff)."""
    out = np.empty(256, dtype=np.float64)
    for c in range(256):
        sign = -1.0 if c & 0x80 else 1.0
        e, m = (c >> 3) & 15, c & 7
        if e == 15 and m == 7:
            out[c] = np.nan
        elif e == 0:
            out[c] = sign * (m / 8.0) * 2.0 ** -6
        else:
            out[c] = sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return out


_TABLE = decode_table()
_POS = _TABLE[:0x7f]          # codes 0x00 .. 0x7e: 0 .. 448, strictly increasing


def decode(codes: np.ndarray) -> np.ndarray:
    return _TABLE[np.asarray(codes, dtype=np.uint8)]


def encode(y) -> np.ndarray:
    """Round-to-nearest-even E4M3 codes (uint8) of float values with |y| < 464."""
    y = np.asarray(y, dtype=np.float64)
    a = np.abs(y)
    if np.any(~np.isfinite(a)) or np.any(a >= 464.0):
        raise ValueError("E4M3 encode: value out of range")
    hi = np.searchsorted(_POS, a, side="left")          # first code with value >= a
    hi_c = np.minimum(hi, len(_POS) - 1)
    lo_c = np.maximum(hi - 1, 0)
    exact = _POS[hi_c] == a
    d_lo = a - _POS[lo_c]
    d_hi = _POS[hi_c] - a
    # above 448 (and below 464) everything rounds down to 448
    pick_hi = np.where(d_hi < d_lo, True, np.where(d_lo < d_hi, False, (lo_c & 1) == 1))
    code = np.where(exact, hi_c, np.where(hi >= len(_POS), len(_POS) - 1, np.where(pick_hi, hi_c, lo_c)))
    code = code.astype(np.uint8)
    return np.where(np.signbit(y), code | np.uint8(0x80), code).astype(np.uint8)


def quantize_rows(x: np.ndarray):
    """Rows of x [R, C] -> (codes uint8 [R, C], d float32 [R]) by the scheme in the module docstring."""
    x = np.asarray(x, dtype=np.float32)
    R = x.shape[0]
    codes = np.zeros(x.shape, dtype=np.uint8)
    d = np.zeros(R, dtype=np.float32)
    for r in range(R):
        if not np.all(np.isfinite(x[r])):
            codes[r] = 0x7F
            d[r] = np.float32(np.nan)
            continue
        amax = np.float32(np.max(np.abs(x[r]))) if x.shape[1] else np.float32(0)
        if amax >= A_MIN:
            mult = np.float32(MAX_E4M3) / amax
            codes[r] = encode(x[r] * mult)
            d[r] = amax / np.float32(MAX_E4M3)
    return codes, d


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def linear_fp8(a_codes, d_a, w_codes, d_w, bias=None, gelu=False) -> np.ndarray:
    """float64 [M, N] = epi(d_a[m] d_w[n] sum_k dec(A) dec(W) + bias)."""
    A = decode(a_codes)
    W = decode(w_codes)
    acc = A @ W.T                                      # exact: see the module docstring
    out = acc * np.asarray(d_a, dtype=np.float64)[:, None] * np.asarray(d_w, dtype=np.float64)[None, :]
    if bias is not None:
        out = out + np.asarray(bias, dtype=np.float64)[None, :]
    return gelu_tanh(out) if gelu else out
