"""The C-ABI library loads without a GPU, exports every entry point declared in
include/*.h, and rejects bad arguments on the host before any HIP call."""
import ctypes as C
import glob
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared(header="mpfa.h"):
    text = open(os.path.join(ROOT, "include", header)).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return set(re.findall(r"\b(mpfa_[a-z0-9_]+)\s*\(", text))


@pytest.fixture(scope="module")
def mp():
    import paper_2609_33135_amd as mp
    if not os.path.exists(mp.LIB_PATH):
        from paper_2609_33135_amd import build
        build.build()
    mp.lib()
    return mp


def test_headers_are_covered():
    assert sorted(os.path.basename(h) for h in glob.glob(os.path.join(ROOT, "include", "*.h"))) == \
        ["mpfa.h", "mpfa_ablate.h", "mpfa_probe.h"]


def test_exports_every_declared_symbol(mp):
    names = _declared()
    assert {"mpfa_quantize_qk", "mpfa_prefill", "mpfa_decode_paged"} <= names
    L = C.CDLL(mp.LIB_PATH)
    for n in sorted(names):
        assert hasattr(L, n), f"{n} declared in include/mpfa.h but not exported"
    assert set(mp.EXPORTED) == names


def test_probe_library_is_separate(mp):
    """The measurement probes live in the benchmark's libmpfa_probe.so, which
    exports what include/mpfa_probe.h declares; the product library has none."""
    from paper_2609_33135_amd import probe
    names = _declared("mpfa_probe.h")
    assert set(probe.EXPORTED) == names
    P = C.CDLL(probe.PROBE_LIB_PATH)
    L = C.CDLL(mp.LIB_PATH)
    for n in sorted(names):
        assert hasattr(P, n), f"{n} missing from libmpfa_probe.so"
        assert not hasattr(L, n), f"{n} still exported by the product library"


def test_ablation_library_is_separate(mp):
    """The softmax ablation levels live in libmpfa_ablate.so (the product entry
    points plus what include/mpfa_ablate.h declares); the product library has
    no trace of them, and the level setter validates its argument."""
    names = _declared("mpfa_ablate.h")
    assert names == {"mpfa_ablation_set_level"}
    A = C.CDLL(os.path.join(os.path.dirname(mp.LIB_PATH), "libmpfa_ablate.so"))
    L = C.CDLL(mp.LIB_PATH)
    for n in sorted(_declared()):
        assert hasattr(A, n), f"{n} missing from libmpfa_ablate.so"
    assert hasattr(A, "mpfa_ablation_set_level") and not hasattr(L, "mpfa_ablation_set_level")
    A.mpfa_ablation_set_level.restype = C.c_int
    assert A.mpfa_ablation_set_level(3) == 1 and A.mpfa_ablation_set_level(-1) == 1
    assert A.mpfa_ablation_set_level(2) == 0 and A.mpfa_ablation_set_level(0) == 0


def test_debug_library_exports_the_same_symbols(mp):
    names = _declared()
    L = C.CDLL(mp.DEBUG_LIB_PATH)
    for n in sorted(names):
        assert hasattr(L, n), f"{n} missing from the debug library"
    assert mp.debug_lib().mpfa_version().decode() == mp.lib().mpfa_version().decode()
    # host validation is shared: bad arguments fail the same way without a GPU
    a = _prefill_args(mp, h_q=7)
    assert mp.debug_lib().mpfa_prefill(C.byref(a), None) == 1


def test_status_strings(mp):
    for s in range(6):
        assert mp.status_string(s)
    assert "data" in mp.status_string(mp.MPFA_ERR_DATA)
    assert mp.lib().mpfa_version().decode().startswith("mpfa")


def _prefill_args(mp, **kw):
    a = mp.PrefillArgs(batch=1, h_q=8, h_kv=2, head_dim=128, max_seqlen_q=16, max_pages=1, flags=1)
    for f in ("cu_seqlens_q", "q_start", "kv_len", "page_table", "q_codes", "q_scales", "q_tscale",
              "k_codes", "k_scales", "v_codes", "ds", "k_tscale", "out"):
        setattr(a, f, 0x1000)   # never dereferenced: validation fails before any launch
    for k, v in kw.items():
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 64, 2), ("head_dim", 0, 1), ("h_q", 7, 1), ("h_kv", 0, 1), ("batch", 0, 1),
    ("max_pages", 0, 1), ("flags", 64, 1), ("flags", 1 | 8 | 32, 1), ("q_codes", None, 1), ("ds", None, 1),
    ("max_seqlen_q", -1, 1), ("h_kv", 64, 1),
])
def test_prefill_validation(mp, field, value, status):
    a = _prefill_args(mp, **{field: value})
    assert mp.lib().mpfa_prefill(C.byref(a), None) == status


def test_prefill_direct_needs_no_side_cache(mp):
    # without MPFA_SMOOTH a null ds is accepted by validation; use an invalid
    # head count as well so that nothing is launched
    a = _prefill_args(mp, flags=0, ds=None, h_q=7)
    assert mp.lib().mpfa_prefill(C.byref(a), None) == 1


def _decode_args(mp, **kw):
    a = mp.DecodeArgs(batch=2, h_q=32, h_kv=8, head_dim=128, max_pages=4, partition_tokens=256,
                      max_partitions=2, flags=1)
    for f in ("kv_len", "page_table", "q_codes", "q_scales", "q_tscale", "k_codes", "k_scales",
              "v_codes", "ds", "k_tscale", "out"):
        setattr(a, f, 0x1000)
    for k, v in kw.items():
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("field,value,status", [
    ("partition_tokens", 100, 1), ("partition_tokens", 0, 1), ("max_partitions", 0, 1),
    ("h_q", 72, 2), ("head_dim", 256, 2), ("kv_len", None, 1), ("flags", 2, 1),
])
def test_decode_validation(mp, field, value, status):
    a = _decode_args(mp, **{field: value})
    assert mp.lib().mpfa_decode_paged(C.byref(a), 0x1000, 1 << 40, None) == status


def test_decode_workspace_checks(mp):
    a = _decode_args(mp)
    need = mp.decode_workspace_size(2, 32, 2)
    assert need == 2 * 32 * 2 * 130 * 4
    assert mp.lib().mpfa_decode_paged(C.byref(a), None, need, None) == 3
    assert mp.lib().mpfa_decode_paged(C.byref(a), 0x1000, need - 1, None) == 3


def test_decode_static_validation(mp):
    """The allocation-free decode rejects bad arguments like mpfa_decode_paged,
    and states larger than the static scratch with MPFA_ERR_WORKSPACE, all on
    the host before any HIP call (this runs without a GPU)."""
    L = mp.lib()
    for field, value, status in (("partition_tokens", 100, 1), ("h_q", 72, 2), ("kv_len", None, 1)):
        a = _decode_args(mp, **{field: value})
        assert L.mpfa_decode_paged_static(C.byref(a), None) == status
    limit = mp.STATIC_SCRATCH_BYTES
    per_partition = 32 * 130 * 4                 # one partition state of every query head
    fits = limit // (2 * per_partition)          # batch 2
    assert mp.decode_workspace_size(2, 32, fits) <= limit < mp.decode_workspace_size(2, 32, fits + 1)
    a = _decode_args(mp, max_partitions=fits + 1)
    assert L.mpfa_decode_paged_static(C.byref(a), None) == mp.MPFA_ERR_WORKSPACE
    assert mp.debug_lib().mpfa_decode_paged_static(C.byref(a), None) == mp.MPFA_ERR_WORKSPACE


def test_choose_partition(mp):
    lens = np.array([16384, 131072, 50000, 8000] * 8, np.int32)
    p = mp.decode_choose_partition(lens, 8, 256)
    assert p % 128 == 0 and 256 <= p <= 16384
    items = sum(-(-int(n) // p) for n in lens) * 8
    assert items >= 256          # enough partition waves to cover the chip
    with pytest.raises(mp.MpfaError):
        mp.decode_choose_partition(np.array([0], np.int32), 8, 256)


def test_quantize_validation(mp):
    a = mp.QuantArgs(batch=1, total_tokens=4, max_seqlen=4, h_q=4, h_kv=2, head_dim=128, flags=3,
                     num_pages=1)
    for f in ("cu_seqlens", "q", "k", "v", "slot_mapping", "q_mean", "k_mean", "k_tscale",
              "q_codes", "q_scales", "q_tscale", "k_codes", "k_scales", "v_codes", "ds"):
        setattr(a, f, 0x1000)
    a.ds = None
    assert mp.lib().mpfa_quantize_qk(C.byref(a), None) == 1      # smoothing needs the side cache
    a.ds = 0x1000
    a.flags = 32
    assert mp.lib().mpfa_quantize_qk(C.byref(a), None) == 1
    a.flags = 3
    a.head_dim = 96
    assert mp.lib().mpfa_quantize_qk(C.byref(a), None) == 2
    a.head_dim = 128
    a.h_kv = 3
    assert mp.lib().mpfa_quantize_qk(C.byref(a), None) == 1


def test_convert_validation(mp):
    for bad in (4, -1, 0x100, 0x17F, 0x200, 0x2FF, 0x300, 0x37F, 0x400, 0x4FF, 0x500):
        assert mp.lib().mpfa_convert(bad, None, 0, None, None) == 1, bad
    assert mp.lib().mpfa_convert(0, None, 5, None, None) == 1


def test_mixed_step_validation(mp):
    """Host validation of the fused step: workspace size, flag consistency,
    unsupported prefill placements; nothing is launched on these paths."""
    n = C.c_size_t(0)
    assert mp.lib().mpfa_mixed_workspace_size(2, 32, 8, 3, C.byref(n)) == 0
    states = 2 * 32 * 3 * 130 * 4
    assert n.value == (states + 255) // 256 * 256 + 2 * 8 * 4
    assert mp.lib().mpfa_mixed_workspace_size(2, 32, 0, 3, C.byref(n)) == 1
    pa = _prefill_args(mp, h_q=32, h_kv=8)
    da = _decode_args(mp, max_partitions=3)
    # smoothing differs between the parts
    pa.flags, da.flags = 1, 0
    assert mp.lib().mpfa_mixed_step(C.byref(pa), C.byref(da), 0x1000, 1 << 30, None) == 1
    # placements the fused kernel does not run
    for f in (1 | 8, 1 | 32, 1 | 64):
        pa.flags, da.flags = f, 1
        assert mp.lib().mpfa_mixed_step(C.byref(pa), C.byref(da), 0x1000, 1 << 30, None) == 2
    # workspace too small for states + counters
    pa.flags, da.flags = 1, 1
    assert mp.lib().mpfa_mixed_step(C.byref(pa), C.byref(da), 0x1000, states, None) == 3
    assert mp.lib().mpfa_mixed_step(None, C.byref(da), 0x1000, 1 << 30, None) == 1


def test_probe_validation(mp):
    """The measurement probes reject bad arguments on the host; the fake device
    addresses below are never dereferenced."""
    from paper_2609_33135_amd import probe
    L = probe.lib()
    sink = 0x1000
    for kind, iters, blocks, s in ((3, 1, 1, sink), (-1, 1, 1, sink), (0, 0, 1, sink), (0, 1, 0, sink),
                                   (0, 1, (1 << 20) + 1, sink), (0, 1, 1, None)):
        assert L.mpfa_probe_mfma(kind, iters, blocks, 0, 0, s, None) == 1, (kind, iters, blocks)
    per_round = 4 * 256 * 8 * 16
    for mode, src, nbytes, blocks, s in ((2, 0x1000, per_round, 4, sink), (0, None, per_round, 4, sink),
                                         (0, 0x1008, per_round, 4, sink), (0, 0x1000, per_round + 16, 4, sink),
                                         (0, 0x1000, 0, 4, sink), (0, 0x1000, per_round, 0, sink),
                                         (1, 0x1000, per_round, 4, None)):
        assert L.mpfa_probe_read(mode, src, nbytes, blocks, s, None) == 1, (mode, src, nbytes, blocks)
