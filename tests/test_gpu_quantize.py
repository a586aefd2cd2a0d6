"""GPU parity of the quantization / cache-write pass: bit-exact against the oracle.

Covers statistics (Eq. 7), NVFP4 Q/K (Eq. 1 + tensor scale), FP8 V, Delta_S
(Eq. 9) on the tiny and the Llama-shaped workloads, ragged multi-sequence
batches, shuffled pages, the direct (unsmoothed) path and the unit tensor
scale.  Also sweeps the device codecs against the oracle's.
"""
import numpy as np
import pytest
import torch

from tests import helpers as H

pytestmark = pytest.mark.gpu

KEYS = ("q_codes", "q_scales", "q_tscale", "q_mean", "k_mean", "k_tscale", "k_codes", "k_scales",
        "v_codes", "ds")


@pytest.fixture(scope="module")
def mp():
    import paper_2609_33135_amd as mp
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    mp.lib()
    return mp


def _assert_quant_equal(run, smooth=True):
    got = run.gpu_quant()
    ref = dict(run.ref)
    ref.update({k: run.ref["cache"][k] for k in ("k_codes", "k_scales", "v_codes", "ds")})
    for key in KEYS:
        if key == "ds" and not smooth:
            continue
        g, r = np.asarray(got[key]), np.asarray(ref[key])
        if key in ("k_codes", "k_scales", "v_codes", "ds"):
            # only the pages this run wrote
            g, r = g[:run.n_pages], r[:run.n_pages]
        assert g.shape == r.shape, (key, g.shape, r.shape)
        if g.dtype.kind == "f":
            eq = np.array_equal(g.view(np.uint32), r.astype(g.dtype).view(np.uint32))
        else:
            eq = np.array_equal(g, r)
        if not eq:
            bad = np.argwhere(g != r)
            raise AssertionError(f"{key}: {len(bad)} mismatches, first at {bad[:3].tolist()}: "
                                 f"gpu {g[tuple(bad[0])]} oracle {r[tuple(bad[0])]}")


def test_quantize_tiny(orc, mp):
    print("case: tiny 1x1 heads 256 tokens seed 1", flush=True)
    run = H.Run(orc, mp, 1, [256], 1, 1, outliers=False)
    _assert_quant_equal(run)


def test_quantize_ragged_batch_shuffled_pages(orc, mp):
    print("case: ragged batch [1, 200, 333, 64] 8q/2kv seed 7", flush=True)
    run = H.Run(orc, mp, 7, [1, 200, 333, 64], 8, 2, outliers=True)
    _assert_quant_equal(run)


@pytest.mark.parametrize("smooth,tunit", [(False, False), (True, True), (False, True)])
def test_quantize_modes(orc, mp, smooth, tunit):
    print(f"case: modes smooth={smooth} tscale_unit={tunit}", flush=True)
    run = H.Run(orc, mp, 9, [300, 129], 4, 4, outliers=True, smooth=smooth, tscale_unit=tunit)
    _assert_quant_equal(run, smooth=smooth)


def test_quantize_statistics_chunk_boundaries(orc, mp):
    """Sequences whose 128-token block counts straddle the 64-block chunks in
    which the statistics finish stages the block partials: 65 blocks (one past
    a chunk, the last block alone in its chunk), 64 (exactly one chunk), 129 (three
    chunks) and 2; means, tensor scales and every code bit-exact."""
    seqlens = [64 * 128 + 1, 64 * 128, 128 * 128 + 37, 129]
    print(f"case: statistics chunk boundaries {seqlens} 4q/2kv seed 23", flush=True)
    run = H.Run(orc, mp, 23, seqlens, 4, 2, outliers=True)
    _assert_quant_equal(run)


def test_quantize_llama_prefill_shape(orc, mp):
    """Full Llama-3.1-8B-shaped prefill workload (16384 tokens, 32q/8kv)."""
    print("case: llama prefill 16384 tokens 32q/8kv seed 2", flush=True)
    run = H.Run(orc, mp, 2, [16384], 32, 8, outliers=True)
    _assert_quant_equal(run)


def test_convert_sweep(orc, mp):
    """Device E4M3 / E2M1 encoders (software and the hardware converters the
    quantization pass uses) against the oracle's over a stride of all FP32 bit
    patterns plus dense neighbourhoods of every rounding boundary."""
    print("case: codec sweep", flush=True)
    pats = np.arange(0, 1 << 32, 61, dtype=np.uint64).astype(np.uint32)
    x = pats.view(np.float32)
    x = x[np.isfinite(x)]
    extra = []
    for p in [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0, 448.0, 464.0, 2.0 ** -6, 2.0 ** -10,
              0.0146484375, 0.9375, 1.0625, 240.0, 232.0]:
        b = int(np.float32(p).view(np.uint32))
        r = np.arange(max(b - 4096, 0), b + 4096, dtype=np.uint32)
        extra += [r, r | np.uint32(0x80000000)]
    x = np.concatenate([x, np.concatenate(extra).view(np.float32)])
    xd = torch.from_numpy(x).cuda()
    for fmt, ref_fn in ((0, orc.e4m3_encode), (1, orc.e2m1_encode), (2, orc.e4m3_encode),
                        (3, orc.e2m1_encode)):
        out = torch.empty(x.size, dtype=torch.uint8, device="cuda")
        mp.convert(fmt, xd, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        ref = ref_fn(x)
        bad = np.nonzero(got != ref)[0]
        assert bad.size == 0, (fmt, x[bad[:5]], got[bad[:5]], ref[bad[:5]])


def test_append_mode_frozen_stats(orc, mp):
    """Second call without statistics reuses the frozen means / K tensor scale
    (decode-time cache write, Sec. 6)."""
    print("case: append mode", flush=True)
    run = H.Run(orc, mp, 13, [500], 8, 2, outliers=True)
    # append 3 new tokens at positions 500..502 of the same sequence
    q, k, v = H.gen_qkv(99, [3], 8, 2, True, "cuda")
    pos = np.arange(500, 503)          # logical page 7 (positions 448..511) already mapped
    assert run.pt.shape[1] * 64 > 502
    slots = H.slots_for(run.pt, 0, pos)
    cu = np.array([0, 3], np.int32)
    qq = mp.QuantQ(3, 1, 8, "cuda")
    mp.quantize_qk(q, k, v, torch.from_numpy(cu).cuda(), torch.from_numpy(slots).cuda(),
                   run.cache, run.stats, qq, mp.SMOOTH, 3)
    torch.cuda.synchronize()
    r = run.ref
    ref = orc.quantize_qk(H.bits(q), H.bits(k), H.bits(v), cu, slots, run.n_pages, orc.SMOOTH,
                          q_mean=r["q_mean"], k_mean=r["k_mean"], k_tscale=r["k_tscale"],
                          cache=r["cache"])
    assert np.array_equal(qq.codes.cpu().numpy(), ref["q_codes"])
    assert np.array_equal(qq.scales.cpu().numpy(), ref["q_scales"])
    assert np.array_equal(qq.tscale.cpu().numpy(), ref["q_tscale"])
    for key in ("k_codes", "k_scales", "v_codes"):
        assert np.array_equal(getattr(run.cache, key).cpu().numpy(), ref["cache"][key]), key
    assert np.array_equal(H.bits(run.cache.ds), ref["cache"]["ds"])


@pytest.mark.parametrize("smooth", [True, False])
def test_quantize_mxfp4(orc, mp, smooth):
    """MXFP4 codes, E8M0 scales (bytes 4..7 zero), unit tensor scales and the
    unchanged means / V / Delta_S, bit for bit."""
    print(f"case: mxfp4 quantize smooth={smooth}", flush=True)
    run = H.Run(orc, mp, 13, [1, 200, 333, 64], 8, 2, outliers=True, smooth=smooth, mxfp4=True)
    _assert_quant_equal(run, smooth=smooth)
    assert np.all(run.stats.k_tscale.cpu().numpy() == 1.0)


def _append_call(orc, mp, run, pos, seed, mx):
    """A later call on sequence 0 of `run` with frozen statistics: tokens at
    positions `pos`, quantized by the HIP path and the oracle from the same
    cache state; compares every output bit."""
    n = len(pos)
    q, k, v = H.gen_qkv(seed, [n], run.h_q, run.h_kv, True, "cuda")
    slots = H.slots_for(run.pt, 0, pos)
    cu = np.array([0, n], np.int32)
    qq = mp.QuantQ(n, 1, run.h_q, "cuda")
    fmt = mp.MXFP4 if mx else 0
    mp.quantize_qk(q, k, v, torch.from_numpy(cu).cuda(), torch.from_numpy(slots).cuda(),
                   run.cache, run.stats, qq, mp.SMOOTH | fmt, n)
    torch.cuda.synchronize()
    r = run.ref
    ref = orc.quantize_qk(H.bits(q), H.bits(k), H.bits(v), cu, slots, run.n_pages,
                          orc.SMOOTH | (orc.MXFP4 if mx else 0), q_mean=r["q_mean"],
                          k_mean=r["k_mean"], k_tscale=r["k_tscale"], cache=r["cache"])
    assert np.array_equal(qq.codes.cpu().numpy(), ref["q_codes"])
    assert np.array_equal(qq.scales.cpu().numpy(), ref["q_scales"])
    assert np.array_equal(qq.tscale.cpu().numpy(), ref["q_tscale"])
    for key in ("k_codes", "k_scales", "v_codes"):
        assert np.array_equal(getattr(run.cache, key).cpu().numpy(), ref["cache"][key]), key
    assert np.array_equal(H.bits(run.cache.ds), ref["cache"]["ds"])
    # the HIP path's cache now equals the oracle's: later calls continue from it
    r["cache"] = ref["cache"]


@pytest.mark.parametrize("mx", [False, True])
def test_chunked_calls_frozen_stats(orc, mp, mx):
    """Chunked prefill: a first 700-token call computes the statistics, then
    300-token chunks with frozen statistics start on a page boundary (whole
    pages written by one chunk) and mid-page (byte-wise page writes); the
    Q tensor scale of each chunk comes from its own tokens over several
    128-token blocks."""
    print(f"case: chunked calls mx={mx}", flush=True)
    run = H.Run(orc, mp, 17, [1400], 8, 2, outliers=True, mxfp4=mx)
    # overwrite positions 704..1003 (page aligned) and 1037..1336 (mid page)
    _append_call(orc, mp, run, np.arange(704, 1004), 71, mx)
    _append_call(orc, mp, run, np.arange(1037, 1337), 72, mx)


def test_quantize_empty_and_short_sequences(orc, mp):
    """Sequences with 0 tokens (means 0, tensor scale 1), one short block, and a
    last block of a single token after a full one."""
    print("case: ragged batch [0, 5, 129, 0, 256]", flush=True)
    run = H.Run(orc, mp, 19, [0, 5, 129, 0, 256], 4, 2, outliers=True)
    _assert_quant_equal(run)


@pytest.mark.parametrize("pv", ["bf16", "nvfp4"])
def test_quantize_pv_copies(orc, mp, pv):
    """The V copies of the PV precision characterization (BF16 rows, or NVFP4
    16-key groups per channel in two planes) bit for bit, next to the unchanged
    FP8 cache, over a ragged batch with shuffled pages and partial last pages."""
    print(f"case: quantize pv={pv}", flush=True)
    run = H.Run(orc, mp, 47, [1, 200, 333, 64, 130], 8, 2, outliers=True, pv=pv)
    _assert_quant_equal(run)
    got = run.cache.v_aux
    got = (H.bits(got) if got.dtype == torch.bfloat16 else got.cpu().numpy()).reshape(-1)
    ref = np.asarray(run.ref["cache"]["v_aux"]).reshape(-1)
    assert got.shape == ref.shape
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, (bad[:5], got[bad[:5]], ref[bad[:5]])


def test_quantizer_division_sweep(orc, mp):
    """The NVFP4 quantizer's element path (correctly rounded x / scale from the
    rounded reciprocal and one residual step, then the FP4 converter) for all
    126 positive E4M3 scales, and the MXFP4 power-of-two path for a spread of
    exponents, against the oracle's IEEE FP32 division and E2M1 encoder, over a
    stride of all FP32 bit patterns plus the neighbourhoods of every decision
    threshold times the scale."""
    print("case: quantizer division sweep", flush=True)
    pats = np.arange(0, 1 << 32, 9973, dtype=np.uint64).astype(np.uint32)
    base = pats.view(np.float32)
    base = base[np.isfinite(base)]
    xd_base = torch.from_numpy(base).cuda()
    out = torch.empty(base.size, dtype=torch.uint8, device="cuda")
    thresholds = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0], np.float32)
    for c in range(1, 0x7F):
        s = np.float32(orc.e4m3_value(c))
        mp.convert(0x100 + c, xd_base, out)
        torch.cuda.synchronize()
        with np.errstate(over="ignore"):   # quotients past FP32 saturate like +-inf
            ref = orc.e2m1_encode(base / s)
        bad = np.nonzero(out.cpu().numpy() != ref)[0]
        assert bad.size == 0, (c, base[bad[:4]])
        # dense neighbourhoods of threshold * scale (the rounding decisions)
        cen = (thresholds * s).astype(np.float32).view(np.uint32).astype(np.int64)
        nb = (cen[:, None] + np.arange(-300, 301)[None, :]).reshape(-1)
        nb = nb[(nb > 0) & (nb < 0x7F800000)].astype(np.uint32)
        x = np.concatenate([nb, nb | np.uint32(0x80000000)]).view(np.float32)
        o2 = torch.empty(x.size, dtype=torch.uint8, device="cuda")
        mp.convert(0x100 + c, torch.from_numpy(x).cuda(), o2)
        torch.cuda.synchronize()
        ref = orc.e2m1_encode(x / s)
        bad = np.nonzero(o2.cpu().numpy() != ref)[0]
        assert bad.size == 0, (c, x[bad[:4]])
    for b in list(range(1, 255, 17)) + [1, 127, 254]:
        mp.convert(0x200 + b, xd_base, out)
        torch.cuda.synchronize()
        with np.errstate(over="ignore"):
            ref = orc.e2m1_encode(np.ldexp(base, -(b - 127)).astype(np.float32))
        bad = np.nonzero(out.cpu().numpy() != ref)[0]
        assert bad.size == 0, (b, base[bad[:4]])
