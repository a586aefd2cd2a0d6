"""GPU tests of the one-launch mixed serving step (mpfa_mixed_step): a chunked
prefill and a split-KV decode batch in one kernel, merge included.  The fused
launch must give exactly the bytes of mpfa_prefill followed by
mpfa_decode_paged (which the prefill and decode parity tests check against
the oracle), and it must leave its partition counters at zero."""
import numpy as np
import pytest
import torch

from tests import helpers as H
from tests.test_gpu_decode import DecodeRun

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mp():
    import paper_2609_33135_amd as mp
    assert torch.cuda.is_available()
    mp.lib()
    return mp


@pytest.mark.parametrize("smooth,mx,partition", [(True, False, 128), (True, False, 1024),
                                                 (False, False, 256), (True, True, 256)])
def test_mixed_step_matches_separate_launches(orc, mp, smooth, mx, partition):
    print(f"case: mixed step smooth={smooth} mx={mx} P={partition}", flush=True)
    seqlens = [130, 300, 513]
    pre = H.Run(orc, mp, 61, seqlens, 8, 2, outliers=True, smooth=smooth, mxfp4=mx)
    dec = DecodeRun(orc, mp, 67, [1, 129, 700, 1500, 64], 8, 2, smooth=smooth, mxfp4=mx)
    flags = (mp.SMOOTH if smooth else 0) | (mp.MXFP4 if mx else 0)
    ref_pre = pre.prefill_gpu()
    ref_dec = dec.gpu(partition)
    maxp = int(max((dec.kv + partition - 1) // partition))
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    ws = torch.zeros(mp.mixed_workspace_size(dec.B, 8, 2, maxp) // 4, dtype=torch.float32, device="cuda")
    n_states = mp.decode_workspace_size(dec.B, 8, maxp) // 4
    T = int(pre.cu[-1])
    for rep in range(3):
        o_pre = torch.full((T, 8, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
        o_dec = torch.full((dec.B, 8, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
        mp.mixed_step(dict(qq=pre.qq, cache=pre.cache, stats=pre.stats, cu_seqlens_q=pre.cu_d,
                           q_start=d(np.zeros(len(seqlens), np.int32)),
                           kv_len=d(np.asarray(seqlens, np.int32)), page_table=d(pre.pt), out=o_pre,
                           max_seqlen_q=max(seqlens)),
                      dict(qq=dec.qq, cache=dec.cache, stats=dec.stats, kv_len=d(dec.kv),
                           page_table=d(dec.pt), out=o_dec, partition_tokens=partition,
                           max_partitions=maxp),
                      ws, flags)
        torch.cuda.synchronize()
        assert np.array_equal(H.bits(o_pre), ref_pre), f"prefill part differs (call {rep})"
        assert np.array_equal(H.bits(o_dec), ref_dec), f"decode part differs (call {rep})"
        counters = ws[(n_states + 63) // 64 * 64:].view(torch.int32).cpu().numpy()
        assert np.all(counters[:dec.B * 2] == 0), "partition counters not reset"
