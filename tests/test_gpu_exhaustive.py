"""Exhaustive device checks of the quantizer's element conversions over every
finite FP32 bit pattern (2^32 patterns in chunks of 2^28).

Each fast path the quantization pass uses is compared with a path written out
from the definitions, through mpfa_convert:
  - the gfx950 E4M3 and E2M1 converters (fmt 2, 3) against the software
    encoders (fmt 0, 1);
  - the NVFP4 element path, RN(x / s) from the rounded reciprocal and one
    residual step, then the converter (fmt 0x100 + c), against IEEE division
    and the software encoder (fmt 0x300 + c), for all 126 positive E4M3 scales;
  - the MXFP4 element path, the scaled converter (fmt 0x200 + b), against exact
    power-of-two scaling and the software encoder (fmt 0x400 + b), for all 254
    block exponents.
The definitional paths are tied to the CPU oracle's encoders on a sample of
bit patterns (test_references_match_the_oracle), so the chain reaches the
oracle."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

CHUNK = 1 << 28


@pytest.fixture(scope="module")
def mp():
    import paper_2609_33135_amd as mp
    assert torch.cuda.is_available()
    mp.lib()
    return mp


def _chunks():
    for start in range(0, 1 << 32, CHUNK):
        bits = torch.arange(start, start + CHUNK, dtype=torch.int64, device="cuda").to(torch.int32)
        x = bits.view(torch.float32)
        yield start, x, torch.isfinite(x)


def _pairs_agree(mp, pairs, label):
    """Every (fast fmt, reference fmt) pair gives the same code for every finite x."""
    a = torch.empty(CHUNK, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for start, x, fin in _chunks():
        for f_fast, f_ref in pairs:
            mp.convert(f_fast, x, a)
            mp.convert(f_ref, x, b)
            bad = (a != b) & fin
            if bool(bad.any()):
                i = int(torch.nonzero(bad)[0])
                pytest.fail(f"{label}: fmt {f_fast:#x} vs {f_ref:#x} differ at bit pattern {start + i:#010x}")
        torch.cuda.synchronize()


def test_e4m3_e2m1_converters_exhaustive(mp):
    print("case: exhaustive E4M3 / E2M1 converters", flush=True)
    _pairs_agree(mp, [(2, 0), (3, 1)], "converter")


def test_nvfp4_element_path_exhaustive(mp):
    print("case: exhaustive NVFP4 element division, 126 scales", flush=True)
    _pairs_agree(mp, [(0x100 + c, 0x300 + c) for c in range(1, 0x7F)], "NVFP4 division")


def test_mxfp4_element_path_exhaustive(mp):
    print("case: exhaustive MXFP4 element scaling, 254 exponents", flush=True)
    _pairs_agree(mp, [(0x200 + b, 0x400 + b) for b in range(1, 255)], "MXFP4 scaling")


def test_references_match_the_oracle(orc, mp):
    """The definitional paths (fmt 0x300 + c, 0x400 + b) against the oracle's
    IEEE FP32 division / exact scaling and E2M1 encoder on a stride of the bit
    patterns (the software encoders fmt 0 and 1 are tied to the oracle by
    test_convert_sweep)."""
    print("case: reference paths vs oracle", flush=True)
    pats = np.arange(0, 1 << 32, 7919, dtype=np.uint64).astype(np.uint32)
    x = pats.view(np.float32)
    x = x[np.isfinite(x)]
    xd = torch.from_numpy(x).cuda()
    out = torch.empty(x.size, dtype=torch.uint8, device="cuda")
    for c in range(1, 0x7F, 5):
        s = np.float32(orc.e4m3_value(c))
        mp.convert(0x300 + c, xd, out)
        torch.cuda.synchronize()
        with np.errstate(over="ignore"):
            ref = orc.e2m1_encode(x / s)
        bad = np.nonzero(out.cpu().numpy() != ref)[0]
        assert bad.size == 0, (c, x[bad[:4]])
    for b in list(range(1, 255, 11)) + [254]:
        mp.convert(0x400 + b, xd, out)
        torch.cuda.synchronize()
        with np.errstate(over="ignore"):
            ref = orc.e2m1_encode(np.ldexp(x, -(b - 127)).astype(np.float32))
        bad = np.nonzero(out.cpu().numpy() != ref)[0]
        assert bad.size == 0, (b, x[bad[:4]])
