"""Hand-worked pins of the online softmax steps that invariants alone cannot
tell apart: the reverse KV-block order (Sec. 4.1), the row sum taken from the
unquantized P (Algorithm 1, the l update), and the direct FP8 write of the
uncentered V (Sec. 4.1 and Sec. 4.2).

The expected values come from tests/golden/online_softmax_cases.json, where
each case is worked out by hand from Algorithm 1 with the arithmetic shown.
"""
import json
import math
import os
import re

import numpy as np
import torch

from paper_2609_33135_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
CASES = json.load(open(os.path.join(GOLDEN, "online_softmax_cases.json")))


def _num(expr):
    """The decimal value after the last '=' of a golden 'formula = value' string."""
    return float(re.findall(r"=\s*([-+0-9.eE]+)", expr)[-1])


def _bf16_bits_f64(x):
    return int(torch.tensor([x], dtype=torch.float64).to(torch.bfloat16).view(torch.int16)) & 0xFFFF


def _unit(c):
    e = np.zeros(128)
    e[c] = 1.0
    return e


def test_golden_arithmetic_is_consistent():
    """The golden numbers follow from their own formulas (exp and the E4M3 grid
    written out, not the oracle)."""
    s = math.sqrt(128.0)
    c = CASES["reverse_sink"]
    p = math.exp(-128.0 / s)
    assert math.isclose(_num(c["p"]), p, rel_tol=1e-15)
    assert 2.5 < 448 * p / 2 ** -9 < 3.5                     # nearest subnormal code: 3 * 2^-9
    assert math.isclose(_num(c["forward"]["out0"]), 3 * 2 ** -9 / (448 * (1 + p)), rel_tol=1e-15)
    assert math.isclose(_num(c["reverse"]["out0"]), p / (1 + p), rel_tol=1e-15)
    for side in ("forward", "reverse"):
        assert int(c[side]["out0_bf16"], 16) == _bf16_bits_f64(_num(c[side]["out0"]))
        assert int(c[side]["out1_bf16"], 16) == _bf16_bits_f64(_num(c[side]["out1"]))
    assert c["forward"]["out0_bf16"] != c["reverse"]["out0_bf16"]
    c = CASES["rowsum_fp32_p"]
    pb = math.exp(-7.5 / s)
    assert math.isclose(_num(c["p"]), pb, rel_tol=1e-15)
    assert 224 < 448 * pb < 232                              # rounds down to 224
    assert math.isclose(_num(c["expected"]["out0"]), 0.5 / (1 + pb), rel_tol=1e-15)
    assert int(c["wrong_if_l_from_p_hat"]["out0_bf16"], 16) == _bf16_bits_f64(0.5 / 1.5)
    assert int(c["wrong_if_p_unquantized"]["out0_bf16"], 16) == _bf16_bits_f64(pb / (1 + pb))
    c = CASES["paged_sink"]
    r = math.exp(-384.0 / s)
    assert math.isclose(_num(c["r"]), r, rel_tol=1e-15)
    assert math.isclose(_num(c["reverse"]["out0"]), p / (1 + p + 127 * r), rel_tol=1e-14)
    assert math.isclose(_num(c["forward"]["out0"]), 3 * 2 ** -9 / (448 * (1 + 127 * r + p)),
                        rel_tol=1e-14)


def test_reverse_order_delays_the_sink(orc):
    """Two KV blocks (tile width 1): a sink key in block 0.  Forward order puts
    the later key's P into the E4M3 subnormal range (3 * 2^-9 instead of
    448 p); reverse order quantizes it at P = 1 and rescales exactly."""
    c = CASES["reverse_sink"]
    q = _unit(0)[None]
    k = np.stack([384.0 * _unit(0), 256.0 * _unit(0)])
    v = np.stack([_unit(1), _unit(0)])
    for flags, side in ((orc.QUANT_P | orc.REVERSE, "reverse"), (orc.QUANT_P, "forward")):
        got = orc.attention_f64(q, k, v, None, None, tile=1, flags=flags)[0]
        assert math.isclose(got[0], _num(c[side]["out0"]), rel_tol=1e-14), side
        assert math.isclose(got[1], _num(c[side]["out1"]), rel_tol=1e-14), side
        assert np.all(got[2:] == 0)
        assert _bf16_bits_f64(got[0]) == int(c[side]["out0_bf16"], 16), side


def test_rowsum_uses_unquantized_p(orc):
    """One block of two keys with 448 p = 230.9: P_hat = 224 enters O, the FP32
    p enters l (Algorithm 1), so out0 = 0.5 / (1 + p), not 0.5 / 1.5."""
    c = CASES["rowsum_fp32_p"]
    q = _unit(0)[None]
    k = np.stack([np.zeros(128), -7.5 * _unit(0)])
    v = np.stack([_unit(1), _unit(0)])
    for tile in (128, 2):
        got = orc.attention_f64(q, k, v, None, None, tile=tile, flags=orc.QUANT_P | orc.REVERSE)[0]
        assert math.isclose(got[0], _num(c["expected"]["out0"]), rel_tol=1e-14)
        assert math.isclose(got[1], _num(c["expected"]["out1"]), rel_tol=1e-14)
        assert _bf16_bits_f64(got[0]) == int(c["expected"]["out0_bf16"], 16)
        assert _bf16_bits_f64(got[1]) == int(c["expected"]["out1_bf16"], 16)


def _paged_sink_cache():
    """The paged_sink case as cache arrays (3 pages of 64 tokens, one head)."""
    n_pages = 3
    k_codes = np.zeros((n_pages, 1, 64, 64), np.uint8)
    k_scales = np.zeros((n_pages, 1, 64, 8), np.uint8)
    v_codes = np.zeros((n_pages, 1, 128, 64), np.uint8)
    ds = np.zeros((n_pages, 1, 64), np.uint16)
    k_codes[0, 0, 0, 0] = 0x07          # key 0, channel 0: E2M1 code 7 (value 6)
    k_scales[0, 0, 0, 0] = 0x58         # E4M3 16
    k_codes[2, 0, 0, 0] = 0x06          # key 128 (page 2, slot 0): code 6 (value 4)
    k_scales[2, 0, 0, 0] = 0x58
    v_codes[0, 0, 1, 0] = 0x38          # key 0: V channel 1 = 1.0
    v_codes[2, 0, 0, 0] = 0x38          # key 128: V channel 0 = 1.0
    cache = dict(k_codes=k_codes, k_scales=k_scales, v_codes=v_codes, ds=ds)
    n = 129
    q_codes = np.zeros((n, 1, 64), np.uint8)
    q_scales = np.zeros((n, 1, 8), np.uint8)
    q_codes[:, 0, 0] = 0x06             # channel 0: value 4
    q_scales[:, 0, 0] = 0x38            # E4M3 1.0
    ones = np.ones((1, 1), np.float32)
    return cache, q_codes, q_scales, ones


def test_paged_sink_reverse_through_prefill_and_decode(orc):
    """The same sink through the product-shaped oracle entry points (128-key
    tiles, 64-token pages): prefill row 128 and the decode query of a 129-key
    context both take the reverse order (one partition of 256 keys)."""
    c = CASES["paged_sink"]["reverse"]
    cache, qc, qs, ones = _paged_sink_cache()
    pt = np.arange(3, dtype=np.int32)[None]
    want = (int(c["out0_bf16"], 16), int(c["out1_bf16"], 16))
    o16, o64 = orc.prefill(cache, pt, [129], ones, qc, qs, ones, [0, 129], [0],
                           np.array([(0, 128, 0)], np.int32), smooth=False)
    assert math.isclose(o64[0, 0], _num(c["out0"]), rel_tol=1e-13)
    assert math.isclose(o64[0, 1], _num(c["out1"]), rel_tol=1e-13)
    assert (int(o16[0, 0]), int(o16[0, 1])) == want and not o16[0, 2:].any()
    for part in (256, 128):   # one partition, or two merged by log-sum-exp: same values
        d16, d64 = orc.decode(cache, pt, [129], ones, qc[128:129], qs[128:129], ones, part,
                              np.array([(0, 0)], np.int32), smooth=False)
        assert math.isclose(d64[0, 0], _num(c["out0"]), rel_tol=1e-13), part
        assert (int(d16[0, 0]), int(d16[0, 1])) == want, part


def test_v_cache_is_direct_e4m3_of_uncentered_v(orc):
    """Algorithm 1 quantizes V itself to FP8 (no centering, no scale; Sec. 4.2
    centers only Q and K).  Every V byte of the channel-major page equals
    torch's float8_e4m3fn encoding of the raw BF16 value, also with smoothing
    on, K offsets present and pages shuffled."""
    n, h_q, h_kv = 200, 4, 2
    q, k, v = W.gen_qkv(41, [n], h_q, h_kv, True, "cpu")
    rng = np.random.default_rng(41)
    vf = v.float()
    vf[:8] *= 2.0 ** -9          # E4M3 subnormal range
    vf[8:16] *= 200.0            # up to the top binade (|v| < 464 keeps torch's cast finite)
    vf = vf.clamp(-460.0, 460.0)
    vf[16, 0, :4] = torch.tensor([0.0, -0.0, 448.0, -2.0 ** -9])
    vb = vf.to(torch.bfloat16)
    perm = rng.permutation(4).astype(np.int64)
    slots = perm[np.arange(n) // 64] * 64 + np.arange(n) % 64
    for flags in (orc.SMOOTH | orc.COMPUTE_STATS, orc.COMPUTE_STATS):
        r = orc.quantize_qk(W.bits(q), W.bits(k), W.bits(vb), [0, n], slots, 4, flags)
        want = vb.float().to(torch.float8_e4m3fn).view(torch.uint8).numpy()   # [n][h_kv][128]
        got = r["cache"]["v_codes"]                                            # [page][h][c][slot]
        for tok in range(n):
            page, off = slots[tok] // 64, slots[tok] % 64
            assert np.array_equal(got[page, :, :, off], want[tok]), (flags, tok)
        assert r["k_mean"].any() == bool(flags & orc.SMOOTH)
