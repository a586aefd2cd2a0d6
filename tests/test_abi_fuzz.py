"""Host validation under random arguments (no GPU needed).

Every device pointer is NULL, so no call may get past validation to a launch:
whatever the sizes and flags, each entry point must return OK (nothing to do),
MPFA_ERR_INVALID, MPFA_ERR_UNSUPPORTED or MPFA_ERR_WORKSPACE, never
MPFA_ERR_HIP (which would mean it tried to launch) and never crash."""
import ctypes as C
import os

import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

ALLOWED = {0, 1, 2, 3}
INTS = st.sampled_from([-2 ** 31, -1, 0, 1, 2, 3, 5, 7, 8, 16, 32, 40, 63, 64, 65, 127, 128, 129, 256, 4096,
                        65535, 65536, 2 ** 31 - 1])
FLAGS = st.one_of(st.integers(0, 2 ** 32 - 1), st.integers(0, 255))
I64 = st.sampled_from([-1, 0, 1, 64, 1 << 20, 1 << 40])
SET = settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])


@pytest.fixture(scope="module")
def mp():
    import paper_2609_33135_amd as mp
    if not os.path.exists(mp.LIB_PATH):
        from paper_2609_33135_amd import build
        build.build()
    mp.lib()
    return mp


def _ints(struct, values):
    a = struct()
    for (name, ctype), v in zip([f for f in struct._fields_ if f[1] is not C.c_void_p], values):
        if ctype is C.c_uint32:
            v &= 0xFFFFFFFF
        setattr(a, name, v)
    return a


@SET
@given(data=st.data())
def test_prefill_null_pointers(mp, data):
    vals = [data.draw(FLAGS if f[0] == "flags" else (I64 if f[1] is C.c_int64 else INTS))
            for f in mp.PrefillArgs._fields_ if f[1] is not C.c_void_p]
    a = _ints(mp.PrefillArgs, vals)
    assert mp.lib().mpfa_prefill(C.byref(a), None) in ALLOWED


@SET
@given(data=st.data())
def test_decode_null_pointers(mp, data):
    vals = [data.draw(FLAGS if f[0] == "flags" else (I64 if f[1] is C.c_int64 else INTS))
            for f in mp.DecodeArgs._fields_ if f[1] is not C.c_void_p]
    a = _ints(mp.DecodeArgs, vals)
    ws_bytes = data.draw(st.sampled_from([0, 1, 1 << 20, 1 << 40]))
    L = mp.lib()
    assert L.mpfa_decode_paged(C.byref(a), None, ws_bytes, None) in ALLOWED
    assert L.mpfa_decode_paged_static(C.byref(a), None) in ALLOWED


@SET
@given(data=st.data())
def test_quantize_null_pointers(mp, data):
    vals = [data.draw(FLAGS if f[0] == "flags" else (I64 if f[1] is C.c_int64 else INTS))
            for f in mp.QuantArgs._fields_ if f[1] is not C.c_void_p]
    a = _ints(mp.QuantArgs, vals)
    assert mp.lib().mpfa_quantize_qk(C.byref(a), None) in ALLOWED


@SET
@given(data=st.data())
def test_mixed_step_null_pointers(mp, data):
    pv = [data.draw(FLAGS if f[0] == "flags" else (I64 if f[1] is C.c_int64 else INTS))
          for f in mp.PrefillArgs._fields_ if f[1] is not C.c_void_p]
    dv = [data.draw(FLAGS if f[0] == "flags" else (I64 if f[1] is C.c_int64 else INTS))
          for f in mp.DecodeArgs._fields_ if f[1] is not C.c_void_p]
    pa, da = _ints(mp.PrefillArgs, pv), _ints(mp.DecodeArgs, dv)
    ws_bytes = data.draw(st.sampled_from([0, 1 << 20, 1 << 40]))
    assert mp.lib().mpfa_mixed_step(C.byref(pa), C.byref(da), None, ws_bytes, None) in ALLOWED


@SET
@given(fmt=st.integers(-2 ** 31, 2 ** 31 - 1), n=st.sampled_from([-1, 1, 100, 1 << 40]))
def test_convert_null_pointers(mp, fmt, n):
    assert mp.lib().mpfa_convert(fmt, None, n, None, None) in ALLOWED


@SET
@given(batch=INTS, h_q=INTS, maxp=INTS)
def test_workspace_sizes(mp, batch, h_q, maxp):
    out = C.c_size_t(0)
    rc = mp.lib().mpfa_decode_workspace_size(batch, h_q, maxp, C.byref(out))
    assert rc in (0, 1)
    if rc == 0:
        assert out.value > 0
    assert mp.lib().mpfa_decode_workspace_size(batch, h_q, maxp, None) == 1
