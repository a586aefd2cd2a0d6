"""GPU parity of causal QK4PV8 prefill against the oracle (Algorithm 1).

The oracle consumes its own quantized codes (which the quantizer tests show
are byte-identical to the GPU's).  Bar: bf16 vs bf16, max |diff| <= 1e-2 and
mean relative error <= 1e-3.
"""
import numpy as np
import pytest
import torch

from tests import helpers as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mp():
    import paper_2609_33135_amd as mp
    assert torch.cuda.is_available()
    mp.lib()
    return mp


def _check(run, gpu_bits, items, q_start=None, kv_len=None, label=""):
    o16, o64 = run.prefill_oracle(items, q_start, kv_len)
    rows = run.cu[items[:, 0]] + items[:, 1]
    got = gpu_bits[rows, items[:, 2]]
    assert not np.isnan(H.bf16_f64(got)).any(), "NaN in GPU output"
    max_abs, mean_rel, n_bad = H.compare_bf16(got, o16)
    print(f"{label}: rows {len(items)} max|d| {max_abs:.3e} mean rel {mean_rel:.3e} over-bar {n_bad}", flush=True)
    assert mean_rel <= H.TOL_MEAN_REL, mean_rel
    assert n_bad == 0, (n_bad, max_abs)
    return max_abs, mean_rel


def _all_items(seqlens, h_q):
    return np.array([(b, i, h) for b, n in enumerate(seqlens) for i in range(n) for h in range(h_q)],
                    np.int32)


def test_prefill_tiny_full(orc, mp):
    """Tiny workload: 1 head, 256 tokens, every output element."""
    print("case: tiny prefill", flush=True)
    run = H.Run(orc, mp, 1, [256], 1, 1, outliers=False)
    out = run.prefill_gpu()
    _check(run, out, _all_items([256], 1), label="tiny")


@pytest.mark.parametrize("smooth", [True, False])
def test_prefill_ragged_gqa(orc, mp, smooth):
    """Ragged batch (lengths not multiples of the tiles), GQA 4:1, shuffled pages."""
    print(f"case: ragged gqa smooth={smooth}", flush=True)
    seqlens = [1, 130, 300, 513]
    run = H.Run(orc, mp, 17, seqlens, 8, 2, outliers=True, smooth=smooth)
    out = run.prefill_gpu()
    _check(run, out, _all_items(seqlens, 8), label=f"ragged smooth={smooth}")


@pytest.mark.parametrize("mx", [False, True])
def test_prefill_chunked_over_prefix(orc, mp, mx):
    """Chunked prefill: the queries are the last 200 tokens of a 700-token sequence
    (q_start = 500) attending to the whole paged prefix (NVFP4 and MXFP4)."""
    print(f"case: chunked prefill mx={mx}", flush=True)
    seqlens = [700]
    run = H.Run(orc, mp, 23, seqlens, 4, 1, outliers=True, mxfp4=mx)
    # queries: rows 500..699 of the quantized Q, re-based as a 200-token call
    mp_ = mp
    qq = mp_.QuantQ(200, 1, 4, "cuda")
    qq.codes.copy_(run.qq.codes[500:700])
    qq.scales.copy_(run.qq.scales[500:700])
    qq.tscale.copy_(run.qq.tscale)
    cu = torch.tensor([0, 200], dtype=torch.int32, device="cuda")
    out = torch.full((200, 4, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
    mp_.prefill(qq, run.cache, run.stats, cu, torch.tensor([500], dtype=torch.int32, device="cuda"),
                torch.tensor([700], dtype=torch.int32, device="cuda"),
                torch.from_numpy(run.pt).cuda(), out, 200, mp_.SMOOTH | (mp_.MXFP4 if mx else 0))
    torch.cuda.synchronize()
    got = H.bits(out)
    r = run.ref
    items = np.array([(0, i, h) for i in range(200) for h in range(4)], np.int32)
    o16, _ = orc.prefill(r["cache"], run.pt, [700], r["k_tscale"], r["q_codes"][500:700],
                         r["q_scales"][500:700], r["q_tscale"], [0, 200], [500], items,
                         mxfp4=mx)
    max_abs, mean_rel, n_bad = H.compare_bf16(got.reshape(-1, 128), o16)
    print(f"chunked: max|d| {max_abs:.3e} mean rel {mean_rel:.3e}")
    assert mean_rel <= H.TOL_MEAN_REL and n_bad == 0, (n_bad, max_abs)


def test_prefill_llama_sampled(orc, mp):
    """Llama-3.1-8B-shaped workload (16384 tokens, 32q/8kv), the launch the
    benchmark times, checked on sampled rows of every head."""
    print("case: llama 16384 sampled", flush=True)
    n = 16384
    run = H.Run(orc, mp, 2, [n], 32, 8, outliers=True)
    out = run.prefill_gpu()
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([np.arange(0, 300), rng.integers(0, n, 200), [n - 1]]))
    items = np.array([(0, int(i), h) for i in rows for h in range(0, 32, 3)], np.int32)
    _check(run, out, items, label="llama sampled")


def test_prefill_deterministic(orc, mp):
    run = H.Run(orc, mp, 5, [1000], 8, 2)
    a = run.prefill_gpu()
    b = run.prefill_gpu()
    assert np.array_equal(a, b)


def test_prefill_seed_modes_bit_identical(orc, mp):
    """The rank-one BF16 MFMA seed and the accumulator-input seed give the same
    FP32 accumulator start (the BF16 Delta_S value), hence identical outputs."""
    print("case: seed modes", flush=True)
    run = H.Run(orc, mp, 29, [700, 45], 8, 2)
    a = run.prefill_gpu()
    b = run.prefill_gpu(extra_flags=mp.SEED_MFMA)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("mx", [False, True])
def test_prefill_elementwise_placement(orc, mp, mx):
    """The element-wise compensation placement (Fig. 10's comparison arm): every
    output row against the oracle, and within one BF16 step of the seeded
    placement (the two differ only in the FP32 rounding order of the scores)."""
    print(f"case: element-wise placement mx={mx}", flush=True)
    seqlens = [1, 130, 300, 513]
    run = H.Run(orc, mp, 23, seqlens, 8, 2, outliers=True, mxfp4=mx)
    out = run.prefill_gpu(extra_flags=mp.SEED_ELEMWISE)
    _check(run, out, _all_items(seqlens, 8), label=f"elementwise mx={mx}")
    seeded = H.bf16_f64(run.prefill_gpu())
    ew = H.bf16_f64(out)
    assert np.all(np.abs(ew - seeded) <= H.bf16_ulp(np.maximum(np.abs(ew), np.abs(seeded))))
    for _ in range(4):
        assert np.array_equal(run.prefill_gpu(extra_flags=mp.SEED_ELEMWISE), out)


def test_prefill_repeatable_all_modes(orc, mp):
    """Every seed mode gives bit-identical outputs over repeated launches (a
    missing synchronisation or an unsatisfied hardware hazard shows up as
    run-to-run differences), and the two placements of the compensation agree."""
    print("case: repeatability", flush=True)
    run = H.Run(orc, mp, 17, [1, 130, 300, 513], 8, 2, outliers=True, smooth=True)
    first = {}
    for _ in range(12):
        for fl in (0, mp.SEED_MFMA):
            out = run.prefill_gpu(extra_flags=fl)
            if fl in first:
                assert np.array_equal(out, first[fl]), f"flags {fl}: output changed between launches"
            else:
                first[fl] = out
    assert np.array_equal(first[0], first[mp.SEED_MFMA])
    direct = H.Run(orc, mp, 17, [1, 130, 300, 513], 8, 2, outliers=True, smooth=False)
    a = direct.prefill_gpu()
    for _ in range(6):
        assert np.array_equal(direct.prefill_gpu(), a)


@pytest.mark.parametrize("smooth", [True, False])
def test_prefill_mxfp4_ragged(orc, mp, smooth):
    """MXFP4 variant over a ragged GQA batch, every output row."""
    print(f"case: mxfp4 prefill smooth={smooth}", flush=True)
    seqlens = [1, 130, 300, 513]
    run = H.Run(orc, mp, 19, seqlens, 8, 2, outliers=True, smooth=smooth, mxfp4=True)
    out = run.prefill_gpu()
    _check(run, out, _all_items(seqlens, 8), label=f"mxfp4 smooth={smooth}")
    if smooth:
        assert np.array_equal(out, run.prefill_gpu(extra_flags=mp.SEED_MFMA))
    for _ in range(4):
        assert np.array_equal(run.prefill_gpu(), out)


def test_prefill_mxfp4_llama_sampled(orc, mp):
    """MXFP4 variant on the Llama-shaped 16384-token workload, sampled rows."""
    print("case: mxfp4 llama 16384 sampled", flush=True)
    n = 16384
    run = H.Run(orc, mp, 2, [n], 32, 8, outliers=True, mxfp4=True)
    out = run.prefill_gpu()
    rng = np.random.default_rng(1)
    rows = np.unique(np.concatenate([np.arange(0, 200), rng.integers(0, n, 150), [n - 1]]))
    items = np.array([(0, int(i), h) for i in rows for h in range(0, 32, 5)], np.int32)
    _check(run, out, items, label="mxfp4 llama sampled")


@pytest.mark.parametrize("pv,smooth", [("bf16", True), ("bf16", False), ("nvfp4", True), ("nvfp4", False)])
def test_prefill_pv_precisions(orc, mp, pv, smooth):
    """The PV precision assignments compared in Sec. 3.1 (BF16 P and V; NVFP4 P
    with dynamic per-16-key scales and NVFP4 V) over a ragged GQA batch, every
    output row against the oracle; repeated launches give identical bytes."""
    print(f"case: pv={pv} smooth={smooth}", flush=True)
    seqlens = [1, 130, 300, 513]
    run = H.Run(orc, mp, 53, seqlens, 8, 2, outliers=True, smooth=smooth, pv=pv)
    out = run.prefill_gpu()
    _check(run, out, _all_items(seqlens, 8), label=f"pv={pv} smooth={smooth}")
    for _ in range(3):
        assert np.array_equal(run.prefill_gpu(), out)


@pytest.mark.parametrize("pv", ["bf16", "nvfp4"])
def test_prefill_pv_llama_sampled(orc, mp, pv):
    """PV precision assignments on the Llama-shaped 16384-token workload, sampled rows."""
    print(f"case: pv={pv} llama 16384 sampled", flush=True)
    n = 16384
    run = H.Run(orc, mp, 2, [n], 32, 8, outliers=True, pv=pv)
    out = run.prefill_gpu()
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([np.arange(0, 130), rng.integers(0, n, 120), [n - 1]]))
    items = np.array([(0, int(i), h) for i in rows for h in range(0, 32, 7)], np.int32)
    _check(run, out, items, label=f"pv={pv} llama sampled")
