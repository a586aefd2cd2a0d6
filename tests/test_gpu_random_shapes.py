"""Randomized parity sweep: prefill and paged decode on shapes the fixed cases
do not name (batch size, head grouping, lengths, smoothing, NVFP4 / MXFP4),
each drawn from its seed and compared with the oracle over every output row."""
import numpy as np
import pytest

from tests import helpers as H
from tests.test_gpu_decode import DecodeRun, _cmp
from tests.test_gpu_prefill import _all_items, _check

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mp():
    import torch
    import paper_2609_33135_amd as mp
    assert torch.cuda.is_available()
    mp.lib()
    return mp

HEADS = [(1, 1), (2, 1), (4, 1), (8, 2), (12, 4), (16, 8), (10, 2), (6, 3)]


def _draw(seed):
    rng = np.random.default_rng(1000 + seed)
    b = int(rng.integers(1, 5))
    lens = [int(x) for x in rng.integers(1, 600, b)]
    h_q, h_kv = HEADS[int(rng.integers(0, len(HEADS)))]
    smooth = bool(rng.integers(0, 2))
    mx = bool(rng.integers(0, 2))
    return lens, h_q, h_kv, smooth, mx


@pytest.mark.parametrize("seed", range(24))
def test_prefill_random_shape(orc, mp, seed):
    lens, h_q, h_kv, smooth, mx = _draw(seed)
    print(f"case: prefill seed {seed} lens {lens} {h_q}q/{h_kv}kv smooth={smooth} mx={mx}", flush=True)
    run = H.Run(orc, mp, 200 + seed, lens, h_q, h_kv, outliers=True, smooth=smooth, mxfp4=mx)
    out = run.prefill_gpu()
    _check(run, out, _all_items(lens, h_q), label=f"random {seed}")


@pytest.mark.parametrize("seed", range(24))
def test_decode_random_shape(orc, mp, seed):
    lens, h_q, h_kv, smooth, mx = _draw(seed)
    lens = [n + 1 for n in lens]   # the decode token comes after the context
    part = 128 * int(np.random.default_rng(seed).integers(1, 4))
    print(f"case: decode seed {seed} lens {lens} {h_q}q/{h_kv}kv smooth={smooth} mx={mx} P={part}", flush=True)
    run = DecodeRun(orc, mp, 300 + seed, lens, h_q, h_kv, smooth=smooth, mxfp4=mx)
    _cmp(run, part, f"random {seed}")
