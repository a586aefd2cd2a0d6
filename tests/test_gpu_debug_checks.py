"""The debug library (libmpfa_debug.so): same kernels, entry points that check
the data they are handed.  On valid inputs its results equal the product
library's bit for bit; on inputs that break an entry point's data contract it
returns MPFA_ERR_DATA before launching anything.

Every invalid input used here stays inside the buffers that were allocated
(page indices past a declared capacity that is smaller than the allocation,
a query range past kv_len inside an allocated page, a NaN value), so that the
kernels would not read outside memory even if a check let them through.
"""
import numpy as np
import pytest
import torch

from tests import helpers as H

pytestmark = pytest.mark.gpu

SEQ = [200, 77]


@pytest.fixture(scope="module")
def mp():
    import paper_2609_33135_amd as mp
    assert torch.cuda.is_available()
    mp.lib()
    mp.debug_lib()
    return mp


@pytest.fixture
def debug(mp, monkeypatch):
    monkeypatch.setattr(mp, "lib", mp.debug_lib)
    return mp


def _decode(mp, run, kv_len, partition=128):
    maxp = -(-int(max(kv_len)) // partition)
    ws = torch.empty(mp.decode_workspace_size(run.B, run.h_q, maxp) // 4, dtype=torch.float32,
                     device="cuda")
    out = torch.full((run.B, run.h_q, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    mp.decode_paged(run.qq, run.cache, run.stats, dev(np.asarray(kv_len, np.int32)), dev(run.pt),
                    out, partition, maxp, ws, mp.SMOOTH)
    torch.cuda.synchronize()
    return H.bits(out)


def test_valid_inputs_match_product_library(orc, mp, monkeypatch):
    ref = H.Run(orc, mp, 71, SEQ, 8, 2)
    p_ref = ref.prefill_gpu()
    d_ref = _decode(mp, ref, SEQ)
    monkeypatch.setattr(mp, "lib", mp.debug_lib)
    run = H.Run(orc, mp, 71, SEQ, 8, 2)
    got = run.gpu_quant()
    for k, v in ref.gpu_quant().items():
        np.testing.assert_array_equal(got[k], v, err_msg=k)
    np.testing.assert_array_equal(run.prefill_gpu(), p_ref)
    np.testing.assert_array_equal(_decode(mp, run, SEQ), d_ref)


def test_nonfinite_input_rejected(orc, debug):
    mp = debug
    run = H.Run(orc, mp, 72, SEQ, 8, 2)
    for which in ("q", "k", "v"):
        x = {"q": run.q, "k": run.k, "v": run.v}
        bad = x[which].clone()
        bad[150, 1, 99] = float("inf") if which == "k" else float("nan")
        x[which] = bad
        with pytest.raises(mp.MpfaError) as e:
            mp.quantize_qk(x["q"], x["k"], x["v"], run.cu_d, run.slots_d, run.cache, run.stats,
                           run.qq, run.flags, max(SEQ))
        assert e.value.status == mp.MPFA_ERR_DATA, which


def test_slot_beyond_capacity_rejected(orc, debug):
    mp = debug
    run = H.Run(orc, mp, 73, SEQ, 8, 2)
    run.cache.num_pages = run.n_pages - 1     # the last allocated page is now past the capacity
    with pytest.raises(mp.MpfaError) as e:
        mp.quantize_qk(run.q, run.k, run.v, run.cu_d, run.slots_d, run.cache, run.stats, run.qq,
                       run.flags, max(SEQ))
    assert e.value.status == mp.MPFA_ERR_DATA


def test_sequence_longer_than_max_seqlen_rejected(orc, debug):
    mp = debug
    run = H.Run(orc, mp, 74, SEQ, 8, 2)
    with pytest.raises(mp.MpfaError) as e:
        mp.quantize_qk(run.q, run.k, run.v, run.cu_d, run.slots_d, run.cache, run.stats, run.qq,
                       run.flags, max(SEQ) - 1)
    assert e.value.status == mp.MPFA_ERR_DATA


def test_prefill_query_range_past_kv_len_rejected(orc, debug):
    mp = debug
    run = H.Run(orc, mp, 75, SEQ, 8, 2)
    with pytest.raises(mp.MpfaError) as e:
        run.prefill_gpu(q_start=[1, 0])        # 200 queries from position 1 over 200 keys
    assert e.value.status == mp.MPFA_ERR_DATA


def test_prefill_page_beyond_capacity_rejected(orc, debug):
    mp = debug
    run = H.Run(orc, mp, 76, SEQ, 8, 2)
    run.cache.num_pages = run.n_pages - 1
    with pytest.raises(mp.MpfaError) as e:
        run.prefill_gpu()
    assert e.value.status == mp.MPFA_ERR_DATA


def test_decode_page_beyond_capacity_rejected(orc, debug):
    mp = debug
    run = H.Run(orc, mp, 77, SEQ, 8, 2)
    assert _decode(mp, run, SEQ).shape == (2, 8, 128)
    run.cache.num_pages = run.n_pages - 1
    with pytest.raises(mp.MpfaError) as e:
        _decode(mp, run, SEQ)
    assert e.value.status == mp.MPFA_ERR_DATA
