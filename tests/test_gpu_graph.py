"""HIP-graph capture of the attention entry points (Sec. 5.3 and Sec. 6: the
split-KV workspaces are preallocated so that decode can be captured into a
graph and replayed).

prefill, paged decode and the one-launch mixed step are captured together
through torch.cuda.CUDAGraph on one stream (and, in a second graph, the whole
path: quantization with statistics, prefill, the decode step's cache write and
the decode), with every buffer (workspaces
included) allocated and initialised before the capture; the graph is then
replayed several times, with the program's own eager launches and host
synchronisations between the replays, and every replay must reproduce the
bytes of the direct launches.
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


def test_graph_capture_and_replay(orc, mp):
    print("case: graph capture of prefill + decode + mixed step", flush=True)
    seqlens = [300, 129, 77]
    run = H.Run(orc, mp, 101, seqlens, 8, 2)
    part = 128
    B, h_q, h_kv = run.B, run.h_q, run.h_kv
    T = int(run.cu[-1])
    want_pre = run.prefill_gpu()
    want_dec = run.decode_last_gpu(part)
    # parity of the direct launches themselves
    items = np.array([(b, i, h) for b, n in enumerate(seqlens) for i in range(0, n, 11)
                      for h in range(h_q)], np.int32)
    ref, _ = run.prefill_oracle(items)
    max_abs, mean_rel, n_bad = H.compare_bf16(want_pre[run.cu[items[:, 0]] + items[:, 1], items[:, 2]], ref)
    assert n_bad == 0 and mean_rel <= H.TOL_MEAN_REL
    max_abs, mean_rel, n_bad = H.compare_bf16(want_dec, run.decode_last_oracle(part))
    assert n_bad == 0 and mean_rel <= H.TOL_MEAN_REL

    # every argument buffer exists before the capture
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    kv = dev(np.asarray(seqlens, np.int32))
    q_start = dev(np.zeros(B, np.int32))
    pt = dev(run.pt)
    last = torch.from_numpy((run.cu[1:] - 1).astype(np.int64)).cuda()
    qd = mp.QuantQ(B, B, h_q, "cuda")
    qd.codes.copy_(run.qq.codes.index_select(0, last))
    qd.scales.copy_(run.qq.scales.index_select(0, last))
    qd.tscale.copy_(run.qq.tscale)
    maxp = int(max((np.asarray(seqlens) + part - 1) // part))
    ws = torch.zeros(mp.decode_workspace_size(B, h_q, maxp) // 4, dtype=torch.float32, device="cuda")
    wsm = torch.zeros(mp.mixed_workspace_size(B, h_q, h_kv, maxp) // 4, dtype=torch.float32,
                      device="cuda")
    outs = {k: torch.full(shape, float("nan"), dtype=torch.bfloat16, device="cuda")
            for k, shape in (("pre", (T, h_q, 128)), ("dec", (B, h_q, 128)),
                             ("mpre", (T, h_q, 128)), ("mdec", (B, h_q, 128)))}
    torch.cuda.synchronize()

    def step():
        mp.prefill(run.qq, run.cache, run.stats, run.cu_d, q_start, kv, pt, outs["pre"], max(seqlens),
                   mp.SMOOTH)
        mp.decode_paged(qd, run.cache, run.stats, kv, pt, outs["dec"], part, maxp, ws, mp.SMOOTH)
        mp.mixed_step(dict(qq=run.qq, cache=run.cache, stats=run.stats, cu_seqlens_q=run.cu_d,
                           q_start=q_start, kv_len=kv, page_table=pt, out=outs["mpre"],
                           max_seqlen_q=max(seqlens)),
                      dict(qq=qd, cache=run.cache, stats=run.stats, kv_len=kv, page_table=pt,
                           out=outs["mdec"], partition_tokens=part, max_partitions=maxp),
                      wsm, mp.SMOOTH)

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    print("graph captured", flush=True)
    eager_out = torch.empty((B, h_q, 128), dtype=torch.bfloat16, device="cuda")
    for rep in range(4):
        for t in outs.values():
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(H.bits(outs["pre"]), want_pre), f"replay {rep}: prefill"
        assert np.array_equal(H.bits(outs["dec"]), want_dec), f"replay {rep}: decode"
        assert np.array_equal(H.bits(outs["mpre"]), want_pre), f"replay {rep}: mixed prefill"
        assert np.array_equal(H.bits(outs["mdec"]), want_dec), f"replay {rep}: mixed decode"
        # eager work of the program between replays, on the same buffers' inputs
        mp.decode_paged(qd, run.cache, run.stats, kv, pt, eager_out, part, maxp, ws, mp.SMOOTH)
        torch.cuda.synchronize()
        assert np.array_equal(H.bits(eager_out), want_dec), f"eager decode after replay {rep}"
    print("graph replays identical", flush=True)


def test_graph_whole_path(orc, mp):
    """The whole path in one graph: the first quantization call (statistics
    computed, cache written), the causal prefill over that cache, then a decode
    step: the cache write of one new token per sequence with the frozen
    statistics (Sec. 6) and the paged decode.  Before every replay the graph's
    cache, statistics and outputs are cleared by eager fills, so each replay
    must rewrite them; all of them must match the eager run byte for byte."""
    print("case: graph capture of quantize + prefill + append + decode", flush=True)
    seqlens = [200, 65, 130]
    h_q, h_kv, part = 8, 2, 128
    run = H.Run(orc, mp, 103, seqlens, h_q, h_kv)
    B = run.B
    T = int(run.cu[-1])
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    pos = np.asarray(seqlens)                       # the new token of each sequence
    assert all(int(p) // 64 < (n + 63) // 64 for p, n in zip(pos, seqlens))
    slots1 = dev(np.concatenate([H.slots_for(run.pt, b, [int(pos[b])]) for b in range(B)]))
    cu1 = dev(np.arange(B + 1, dtype=np.int32))
    q1, k1, v1 = H.gen_qkv(104, [1] * B, h_q, h_kv, True, "cuda")
    kv = dev((pos + 1).astype(np.int32))
    kv0 = dev(np.asarray(seqlens, np.int32))
    q_start = dev(np.zeros(B, np.int32))
    pt = dev(run.pt)
    maxp = int(max((pos + 1 + part - 1) // part))
    ws = torch.zeros(mp.decode_workspace_size(B, h_q, maxp) // 4, dtype=torch.float32, device="cuda")

    # eager reference on the Run's buffers (its first quantization call already ran)
    want_pre = run.prefill_gpu()
    qd = mp.QuantQ(B, B, h_q, "cuda")
    mp.quantize_qk(q1, k1, v1, cu1, slots1, run.cache, run.stats, qd, mp.SMOOTH, 1)
    dec = torch.empty((B, h_q, 128), dtype=torch.bfloat16, device="cuda")
    mp.decode_paged(qd, run.cache, run.stats, kv, pt, dec, part, maxp, ws, mp.SMOOTH)
    torch.cuda.synchronize()
    want_dec = H.bits(dec)
    planes = lambda c, s, qq, qd_: [c.k_codes, c.k_scales, c.v_codes, c.ds, s.q_mean, s.k_mean, s.k_tscale,
                                    qq.codes, qq.scales, qq.tscale, qd_.codes, qd_.scales, qd_.tscale]
    want = [t.detach().clone() for t in planes(run.cache, run.stats, run.qq, qd)]

    # graph buffers: all allocated before the capture
    cache = mp.PagedCache(run.cache.num_pages, h_q, h_kv, "cuda", smooth=True)
    stats = mp.SeqStats(B, h_q, h_kv, "cuda")
    qq = mp.QuantQ(T, B, h_q, "cuda")
    qd2 = mp.QuantQ(B, B, h_q, "cuda")
    pre = torch.empty((T, h_q, 128), dtype=torch.bfloat16, device="cuda")
    dec2 = torch.empty((B, h_q, 128), dtype=torch.bfloat16, device="cuda")
    ws2 = torch.zeros_like(ws)
    torch.cuda.synchronize()

    def step():
        mp.quantize_qk(run.q, run.k, run.v, run.cu_d, run.slots_d, cache, stats, qq, run.flags, max(seqlens))
        mp.prefill(qq, cache, stats, run.cu_d, q_start, kv0, pt, pre, max(seqlens), mp.SMOOTH)
        mp.quantize_qk(q1, k1, v1, cu1, slots1, cache, stats, qd2, mp.SMOOTH, 1)
        mp.decode_paged(qd2, cache, stats, kv, pt, dec2, part, maxp, ws2, mp.SMOOTH)

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    print("graph captured", flush=True)
    for rep in range(3):
        for t in planes(cache, stats, qq, qd2):
            t.zero_()
        pre.fill_(float("nan"))
        dec2.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(planes(cache, stats, qq, qd2), want)):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"replay {rep}: plane {i}"
        assert np.array_equal(H.bits(pre), want_pre), f"replay {rep}: prefill"
        assert np.array_equal(H.bits(dec2), want_dec), f"replay {rep}: decode"
    print("graph replays identical", flush=True)
