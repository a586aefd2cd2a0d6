"""Pins of the oracle's number formats against their definitions and library routines.

E2M1 and E4M3 are the element and scale formats of NVFP4 (Sec. 2.1, Eq. 1);
E4M3 is also the P and V format (Sec. 4.1).  The pins are independent of the
oracle's own code: bit-field formulas, torch's float8_e4m3fn / bfloat16
conversions (library routines), and a float rounding construction for E2M1.
"""
import numpy as np
import pytest
import torch


def e2m1_from_bits(code):
    """E2M1 by its bit fields: sign | e1 e0 | m; e == 0 is subnormal (0.5 * m)."""
    s = -1.0 if code & 8 else 1.0
    e = (code >> 1) & 3
    m = code & 1
    return s * (0.5 * m if e == 0 else 2.0 ** (e - 1) * (1 + m / 2))


def test_e2m1_decode_all_codes(orc):
    for c in range(16):
        assert orc.e2m1_value(c) == e2m1_from_bits(c)
    # rho = 6 is the largest E2M1 magnitude (Sec. 2.1)
    assert max(abs(orc.e2m1_value(c)) for c in range(16)) == 6.0


def test_e4m3_decode_all_codes_against_torch(orc):
    codes = torch.arange(256, dtype=torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    for c in range(256):
        v = orc.e4m3_value(c)
        if np.isnan(ref[c]):
            assert np.isnan(v), c
        else:
            assert v == ref[c] and np.signbit(v) == np.signbit(ref[c]), c
    # 448 is the largest normal E4M3 value (Sec. 4.1)
    finite = [abs(orc.e4m3_value(c)) for c in range(256) if not np.isnan(orc.e4m3_value(c))]
    assert max(finite) == 448.0


def _e2m1_round_ref(x):
    """Round to the E2M1 grid by the float construction: quantum 0.5 below 2, 1 in
    [2, 4), 2 from 4 on, round half to even multiple (np.round), saturate at 6."""
    a = np.abs(x.astype(np.float64))
    q = np.where(a < 2.0, 0.5, np.where(a < 4.0, 1.0, 2.0))
    r = np.round(a / q) * q
    r = np.minimum(r, 6.0)
    mag_to_code = {0.0: 0, 0.5: 1, 1.0: 2, 1.5: 3, 2.0: 4, 3.0: 5, 4.0: 6, 6.0: 7}
    code = np.zeros(x.shape, np.uint8)
    for mag, c in mag_to_code.items():
        code[r == mag] = c
    code |= np.where(np.signbit(x), 8, 0).astype(np.uint8)
    return code


def _float_neighbourhoods(points, span=1 << 14):
    """All float32 bit patterns within +-span ulps of each point (both signs)."""
    out = []
    for p in points:
        b = int(np.float32(p).view(np.uint32))
        lo, hi = max(0, b - span), min(0x7F7FFFFF, b + span)
        pats = np.arange(lo, hi + 1, dtype=np.uint32)
        out.append(pats)
        out.append(pats | np.uint32(0x80000000))
    return np.concatenate(out).view(np.float32)


def _strided_all_finite(stride):
    pats = np.arange(0, 1 << 32, stride, dtype=np.uint64).astype(np.uint32)
    x = pats.view(np.float32)
    return x[np.isfinite(x)]


E2M1_POINTS = [0.0, 0.25, 0.5, 0.75, 1.0, 1.25, 1.5, 1.75, 2.0, 2.5, 3.0, 3.5, 4.0, 5.0, 6.0, 7.0]


def test_e2m1_encode_sweep(orc):
    x = np.concatenate([_float_neighbourhoods(E2M1_POINTS), _strided_all_finite(509),
                        np.array([0.0, -0.0, 1e-45, -1e-45, 3.4e38, -3.4e38], np.float32)])
    got = orc.e2m1_encode(x)
    ref = _e2m1_round_ref(x)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, (x[bad[:5]], got[bad[:5]], ref[bad[:5]])


def _e4m3_points():
    vals = sorted({abs(float(v)) for v in torch.arange(0, 127, dtype=torch.uint8)
                   .view(torch.float8_e4m3fn).to(torch.float64).numpy()})
    mids = [(a + b) / 2 for a, b in zip(vals[:-1], vals[1:])]
    return vals + mids + [464.0, 480.0]


def test_e4m3_encode_sweep_against_torch(orc):
    x = np.concatenate([_float_neighbourhoods(_e4m3_points(), span=1 << 10),
                        _strided_all_finite(509)])
    got = orc.e4m3_encode(x)
    inrange = np.abs(x) <= 464.0
    ref = torch.from_numpy(x[inrange]).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    bad = np.nonzero(got[inrange] != ref)[0]
    assert bad.size == 0, (x[inrange][bad[:5]], got[inrange][bad[:5]], ref[bad[:5]])
    # saturation above the largest finite value (the oracle's reading: saturate)
    big = x[~inrange]
    assert np.all((got[~inrange] & 0x7F) == 0x7E)
    assert np.all((got[~inrange] >> 7) == np.signbit(big))


def test_e4m3_encode_p_range_exhaustive(orc):
    """Every FP32 value of 448*P for P in (0, 1] (Sec. 4.1): exhaustive over [2^-12, 448]."""
    lo = int(np.float32(2.0 ** -12).view(np.uint32))
    hi = int(np.float32(448.0).view(np.uint32))
    pats = np.arange(lo, hi + 1, 3, dtype=np.uint32)
    x = pats.view(np.float32)
    got = orc.e4m3_encode(x)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(got, ref)
    # P = 1 maps to the largest code and never saturates (Sec. 4.1)
    assert orc.e4m3_encode(np.array([448.0], np.float32))[0] == 0x7E


def test_bf16_encode_against_torch(orc):
    x = np.concatenate([_strided_all_finite(257),
                        _float_neighbourhoods([1.0, 3.0, 1e-30, 6e4], span=1 << 12)])
    x = x[np.abs(x) < 3.38e38]   # stay clear of rounding up to infinity
    got = orc.bf16_encode(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, ref)


def test_bf16_from_f64_single_rounding(orc):
    # 1 + 2^-8 + 2^-30 is above the BF16 midpoint 1 + 2^-8; a detour through FP32
    # would land on the midpoint and round to even (1.0).
    x = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert orc.bf16_encode_f64(x) == 0x3F81
    assert orc.bf16_encode_f64(1.0 + 2.0 ** -8) == 0x3F80   # exact tie -> even
    assert orc.bf16_encode_f64(-(1.0 + 3 * 2.0 ** -8)) == 0xBF82


def test_signed_zero_kept(orc):
    assert orc.e2m1_encode(np.array([-0.0, -0.1], np.float32)).tolist() == [8, 8]
    assert orc.e4m3_encode(np.array([-0.0, -1e-6], np.float32)).tolist() == [0x80, 0x80]
