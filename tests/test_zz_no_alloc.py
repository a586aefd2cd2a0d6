"""mpfa_decode_paged_static (the decode entry point for callers that cannot
allocate) against mpfa_decode_paged on the same inputs: identical bytes on two
calls in a row, the second with a smaller batch and shorter contexts, both
within the oracle bar; and the host-side rejection of states larger than the
static scratch."""
import ctypes as C

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


def _decode_both(mp, run, seqs, kv, part):
    """Decode of the last query token of sequences `seqs` over kv keys each,
    through the workspace entry point and through the static one."""
    B = len(seqs)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    last = torch.from_numpy((run.cu[1:][seqs] - 1).astype(np.int64)).cuda()
    qq = mp.QuantQ(B, B, run.h_q, "cuda")
    qq.codes.copy_(run.qq.codes.index_select(0, last))
    qq.scales.copy_(run.qq.scales.index_select(0, last))
    qq.tscale.copy_(run.qq.tscale[torch.as_tensor(seqs).cuda()])
    stats = mp.SeqStats(B, run.h_q, run.h_kv, "cuda")
    idx = torch.as_tensor(seqs).cuda()
    stats.q_mean.copy_(run.stats.q_mean[idx])
    stats.k_mean.copy_(run.stats.k_mean[idx])
    stats.k_tscale.copy_(run.stats.k_tscale[idx])
    kv = np.asarray(kv, np.int32)
    kv_d, pt_d = dev(kv), dev(run.pt[seqs])
    maxp = int(max((kv + part - 1) // part))
    ws = torch.empty(mp.decode_workspace_size(B, run.h_q, maxp) // 4, dtype=torch.float32, device="cuda")
    ref = torch.full((B, run.h_q, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
    got = torch.full((B, run.h_q, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    mp.decode_paged(qq, run.cache, stats, kv_d, pt_d, ref, part, maxp, ws, mp.SMOOTH)
    mp.decode_paged_static(qq, run.cache, stats, kv_d, pt_d, got, part, maxp, mp.SMOOTH)
    torch.cuda.synchronize()
    return H.bits(got), H.bits(ref)


def test_decode_static_matches_workspace_entry(orc, mp):
    print("case: decode static scratch vs workspace, two calls", flush=True)
    seqlens = [700, 300, 129, 1000]
    run = H.Run(orc, mp, 103, seqlens, 8, 2)
    # first call: all four sequences, whole contexts, partition 128
    got, ref = _decode_both(mp, run, [0, 1, 2, 3], seqlens, 128)
    assert np.array_equal(got, ref), "static decode differs from the workspace decode (call 1)"
    oref = run.decode_last_oracle(128)
    max_abs, mean_rel, n_bad = H.compare_bf16(got, oref)
    print(f"call 1: max|d| {max_abs:.3e} mean rel {mean_rel:.3e}", flush=True)
    assert n_bad == 0 and mean_rel <= H.TOL_MEAN_REL
    # second call: a smaller input (two sequences, shorter visible contexts,
    # fewer partitions); the scratch still holds the first call's states
    kv2 = [250, 100]
    got2, ref2 = _decode_both(mp, run, [1, 2], kv2, 256)
    assert np.array_equal(got2, ref2), "static decode differs from the workspace decode (call 2)"
    assert not np.isnan(H.bf16_f64(got2)).any()


def test_decode_static_rejects_oversized_states(mp):
    print("case: decode static oversized request", flush=True)
    a = mp.DecodeArgs(batch=2, h_q=32, h_kv=8, head_dim=128, max_pages=4, partition_tokens=256,
                      max_partitions=1 << 14, flags=1)
    for f in ("kv_len", "page_table", "q_codes", "q_scales", "q_tscale", "k_codes", "k_scales",
              "v_codes", "ds", "k_tscale", "out"):
        setattr(a, f, 0x1000)   # never dereferenced: rejected on the host
    assert mp.decode_workspace_size(2, 32, 1 << 14) > mp.STATIC_SCRATCH_BYTES
    assert mp.lib().mpfa_decode_paged_static(C.byref(a), None) == mp.MPFA_ERR_WORKSPACE
