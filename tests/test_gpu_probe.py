"""The measurement probes compute what they claim: every MFMA of the issue-rate
probe runs (the accumulators reach exactly 32 * K * iters with all-ones
operands), and the read probe reads every word of the buffer exactly once (the
XOR of its per-thread results equals the XOR of the buffer)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mp():
    import torch
    from paper_2609_33135_amd import probe as mp
    assert torch.cuda.is_available()
    mp.lib()
    return mp


@pytest.mark.parametrize("kind,k", [(0, 32), (1, 128), (2, 128)])
def test_mfma_probe_counts_every_mfma(mp, kind, k):
    import torch
    print(f"case: mfma probe kind {kind}", flush=True)
    blocks, iters = 12, 300
    sink = torch.full((blocks * 256,), -1.0, dtype=torch.float32, device="cuda")
    fl = mp.probe_mfma(kind, iters, blocks, sink)
    torch.cuda.synchronize()
    assert fl == blocks * 4 * iters * 8 * 2 * 16 * 16 * k
    assert torch.all(sink == float(32 * k * iters)).item()


def test_mfma_probe_operands_reach_the_product(mp):
    """A = 2, B = 1.5 (FP16): each MFMA adds 32 * 3 to every accumulator."""
    import torch
    print("case: mfma probe operands", flush=True)
    sink = torch.zeros(256 * 2, dtype=torch.float32, device="cuda")
    mp.probe_mfma(0, 7, 2, sink, pa=0x40004000, pb=0x3E003E00)
    torch.cuda.synchronize()
    assert torch.all(sink == float(32 * 32 * 3 * 7)).item()


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("blocks,rounds", [(8, 1), (24, 5)])
def test_read_probe_reads_every_word_once(mp, mode, blocks, rounds):
    import torch
    print(f"case: read probe mode {mode} blocks {blocks} rounds {rounds}", flush=True)
    n_words = blocks * 256 * 8 * 4 * rounds
    g = torch.Generator().manual_seed(5 + mode + blocks)
    host = torch.randint(-2 ** 31, 2 ** 31 - 1, (n_words,), dtype=torch.int32, generator=g)
    buf = host.cuda()
    sink = torch.zeros(blocks * 256, dtype=torch.int32, device="cuda")
    mp.probe_read(mode, buf, blocks, sink)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(host.numpy().view(np.uint32))
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == want
    # a word read twice or skipped would show in the XOR of a buffer with one word changed
    host2 = host.clone()
    host2[n_words // 3] ^= 0x10203
    buf.copy_(host2)
    mp.probe_read(mode, buf, blocks, sink)
    torch.cuda.synchronize()
    assert np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32)) == want ^ np.uint32(0x10203)
