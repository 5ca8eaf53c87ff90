"""Pins of the oracle's FP8 (OCP E4M3) quantisation and scaled linear layer (CPU only).

The decoding and the round-to-nearest-even encoding are checked against PyTorch's own
float8_e4m3fn conversions (an implementation of the same OCP format written by others) and
against values the format fixes; the quantiser against the format's error bound; the linear
layer against exact rational arithmetic on inputs whose codes decode to small integers."""
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import fp8 as F


def _torch_decode(codes):
    t = torch.from_numpy(np.asarray(codes, dtype=np.uint8)).view(torch.float8_e4m3fn)
    return t.to(torch.float64).numpy()


def _torch_encode(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_matches_format_and_torch():
    t = F.decode_table()
    ref = _torch_decode(np.arange(256))
    nan = np.isnan(ref)
    assert list(np.flatnonzero(nan)) == [0x7f, 0xff]
    np.testing.assert_array_equal(np.isnan(t), nan)
    np.testing.assert_array_equal(t[~nan], ref[~nan])
    # values the format fixes
    assert t[0x00] == 0.0 and np.signbit(t[0x80]) and t[0x80] == 0.0
    assert t[0x01] == 2.0 ** -9 and t[0x07] == 7 * 2.0 ** -9 and t[0x08] == 2.0 ** -6
    assert t[0x38] == 1.0 and t[0x40] == 2.0 and t[0x7e] == 448.0 and t[0xfe] == -448.0
    assert np.all(np.diff(t[:0x7f]) > 0)          # positive codes are ordered by value


def test_encode_matches_torch_round_to_nearest_even():
    rng = np.random.default_rng(3)
    mags = 2.0 ** rng.uniform(-13, np.log2(463.9), size=200000)
    x = (mags * rng.choice([-1.0, 1.0], size=mags.size)).astype(np.float32)
    pos = F.decode_table()[:0x7f]
    mids = ((pos[:-1] + pos[1:]) / 2).astype(np.float32)      # exact ties, all representable in float32
    x = np.concatenate([x, mids, -mids, pos.astype(np.float32), -pos.astype(np.float32),
                        np.float32([0.0, -0.0, 448.0, 463.9, -463.9])])
    got = F.encode(x)
    ref = _torch_encode(x)
    np.testing.assert_array_equal(got, ref)
    # ties go to the even code: 1 + 1/16 lies between 0x38 and 0x39
    assert F.encode(np.float32(1.0625)) == 0x38 and F.encode(np.float32(1.1875)) == 0x3a
    with pytest.raises(ValueError):
        F.encode(np.float32(464.0))


def test_quantize_rows_error_bound_and_edges():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((64, 300)) * np.exp(rng.uniform(-3, 3, size=(64, 1)))).astype(np.float32)
    x[3] = 0.0
    codes, d = F.quantize_rows(x)
    assert d.dtype == np.float32 and codes.dtype == np.uint8
    assert np.all(codes[3] == 0) and d[3] == 0
    deq = F.decode(codes) * d[:, None].astype(np.float64)
    for r in range(64):
        if r == 3:
            continue
        amax = np.abs(x[r]).max()
        i = np.argmax(np.abs(x[r]))
        assert codes[r, i] & 0x7f == 0x7e                    # the largest entry maps to 448
        y = np.abs(x[r].astype(np.float64)) * (448.0 / amax)
        err = np.abs(deq[r] - x[r])
        # half a unit in the last place: 2^-4 relative for normals (y >= 2^-6), 2^-10 * d below
        bound = np.where(y >= 2.0 ** -6, 2.0 ** -4 * np.abs(x[r]), 2.0 ** -10 * d[r]) * (1 + 1e-6) + 1e-30
        assert np.all(err <= bound)


def test_quantize_rows_out_of_range_rows():
    """Rows below A_MIN = 448 * 2^-126 are zero rows; at A_MIN the scale is exactly 2^-126 and
    mult exactly 2^126 (both powers of two, so the codes are those of x * 2^126); a row holding
    an infinity or a NaN is all NaN codes with d = NaN."""
    amin = np.float32(448.0 * 2.0 ** -126)
    x = np.zeros((6, 16), dtype=np.float32)
    x[0, 3] = np.float32(1e-37)                        # below A_MIN: a zero row
    x[1, 3] = -np.nextafter(amin, np.float32(0))       # just below, negative
    x[2, 3] = amin                                     # the smallest row quantised
    x[2, 7] = -amin / np.float32(4)
    x[3] = 1.0
    x[3, 5] = np.inf
    x[4] = 1.0
    x[4, 9] = np.nan
    x[5, 0] = -np.inf
    codes, d = F.quantize_rows(x)
    assert np.all(codes[:2] == 0) and np.all(d[:2] == 0)
    assert d[2] == np.float32(2.0 ** -126)
    assert codes[2, 3] == 0x7E and codes[2, 7] == F.encode(np.float32(-112.0)) and codes[2, 7] == 0xEE
    assert np.count_nonzero(codes[2]) == 2
    assert np.all(codes[3:] == 0x7F) and np.all(np.isnan(d[3:]))
    assert F.A_MIN == amin


def test_linear_fp8_exact_on_integer_codes():
    rng = np.random.default_rng(9)
    ints = np.array([0, 1, 2, 3, 4, 6, 8, 12, 16])
    vals_a = rng.choice(ints, size=(5, 40)) * rng.choice([-1, 1], size=(5, 40))
    vals_w = rng.choice(ints, size=(7, 40)) * rng.choice([-1, 1], size=(7, 40))
    a_codes = F.encode(vals_a.astype(np.float32))
    w_codes = F.encode(vals_w.astype(np.float32))
    np.testing.assert_array_equal(F.decode(a_codes), vals_a)
    d_a = np.float32([0.5, 2.0, 0.25, 1.0, 8.0])
    d_w = np.float32([1.0, 0.125, 4.0, 2.0, 0.5, 1.0, 0.0625])
    bias = np.float32([0.5, -1.0, 0.0, 2.0, 0.25, -0.5, 1.0])
    got = F.linear_fp8(a_codes, d_a, w_codes, d_w, bias)
    for m in range(5):
        for n in range(7):
            s = sum(Fraction(int(vals_a[m, k])) * int(vals_w[n, k]) for k in range(40))
            ref = s * Fraction(float(d_a[m])) * Fraction(float(d_w[n])) + Fraction(float(bias[n]))
            assert got[m, n] == float(ref)
    g = F.linear_fp8(a_codes, d_a, w_codes, d_w, bias, gelu=True)
    np.testing.assert_array_equal(g, F.gelu_tanh(got))


def test_gelu_tanh_matches_torch():
    z = np.linspace(-12, 12, 4001)
    ref = torch.nn.functional.gelu(torch.from_numpy(z), approximate="tanh").numpy()
    np.testing.assert_allclose(F.gelu_tanh(z), ref, rtol=1e-12, atol=1e-15)
