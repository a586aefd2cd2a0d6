"""CPU checks of the benchmark's reporting helpers (no GPU): the FP64 accuracy
reference and the error measure used for the NVFP4 / MXFP4 error report."""
import math
import os
import sys

import numpy as np
import torch

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _inputs(seed, n, h_q, h_kv):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(n, h_q, 128, generator=g).bfloat16()
    k = (torch.randn(n, h_kv, 128, generator=g) + 2.0 * torch.randn(1, h_kv, 128, generator=g)).bfloat16()
    v = torch.randn(n, h_kv, 128, generator=g).bfloat16()
    return dict(q=q, k=k, v=v)


def test_fp64_reference_matches_oracle_textbook(orc):
    st = _inputs(1, 200, 4, 2)
    ref = bench.fp64_reference(np, st, 2, 9)
    assert ref["heads"] == [0, 2]
    assert ref["rows"][0] == 0 and ref["rows"][-1] == 199
    for h in ref["heads"]:
        q = st["q"][:, h].double().numpy()
        k = st["k"][:, h // 2].double().numpy()
        v = st["v"][:, h // 2].double().numpy()
        want = orc.attention_textbook(q[ref["rows"]], k, v, ref["rows"])
        assert np.max(np.abs(ref["o"][h] - want)) < 1e-12


def test_error_measure():
    st = _inputs(2, 130, 2, 1)
    ref = bench.fp64_reference(np, st, 2, 5)
    out = torch.zeros(130, 2, 128, dtype=torch.float64)
    for h in ref["heads"]:
        out[torch.from_numpy(ref["rows"]), h] = torch.from_numpy(ref["o"][h])
    e = bench.error_vs_fp64(np, out, ref)
    assert e["rel_l2"] < 1e-6 and e["max_abs"] < 1e-6          # FP32 rounding of the copy only
    out2 = out * 1.5
    e2 = bench.error_vs_fp64(np, out2, ref)
    assert math.isclose(e2["rel_l2"], 0.5, rel_tol=1e-6)
