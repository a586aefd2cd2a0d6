"""Seeded synthetic inputs for the QK4PV8 attention path.

This module holds only random-number generation and workload shapes; none of
the method's arithmetic.  It serves both the HIP path and the oracle: inputs
are generated once (on the CPU or on the GPU) and the same bits are handed to
both sides.

Generator (counter based, so any slice can be regenerated without storing
the rest): every element has a 64-bit counter built from (batch, token, head,
channel); the SplitMix64 finaliser applied to (stream key + counter * golden
gamma) yields 64 random bits; the upper and lower 32 bits are two uniforms
and Box-Muller (FP64) turns them into one standard normal, which is rounded
to FP32 and then to BF16.

Value structure: the paper's Q/K activations show stable per-channel outlier
ridges (Sec. 4.2, Fig. 4); with no trained weights available, synthetic K gets
one N(0, 4) offset per (KV head, channel), shared by all tokens, and in the
outlier recipe a 0.001 fraction of Q and K entries is multiplied by 20 (before
the offset is added).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB

STREAM_Q, STREAM_K, STREAM_V, STREAM_KOFF, STREAM_OUT_Q, STREAM_OUT_K = 1, 2, 3, 4, 5, 6
OUTLIER_FRACTION = 0.001
OUTLIER_GAIN = 20.0
K_OFFSET_STD = 2.0   # variance 4


def _s64(x: int) -> int:
    """Python int -> the int64 with the same 64-bit pattern."""
    x &= MASK64
    return x - (1 << 64) if x >= (1 << 63) else x


def _mix_py(z: int) -> int:
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX1) & MASK64
    z = ((z ^ (z >> 27)) * MIX2) & MASK64
    return z ^ (z >> 31)


def stream_key(seed: int, stream: int) -> int:
    return _mix_py(_mix_py(seed * GAMMA + stream) + stream * GAMMA)


def _lsr(z: torch.Tensor, k: int) -> torch.Tensor:
    return (z >> k) & ((1 << (64 - k)) - 1)


def _mix_t(z: torch.Tensor) -> torch.Tensor:
    z = (z ^ _lsr(z, 30)) * _s64(MIX1)
    z = (z ^ _lsr(z, 27)) * _s64(MIX2)
    return z ^ _lsr(z, 31)


def random_bits(key: int, ctr: torch.Tensor) -> torch.Tensor:
    """64 random bits (as int64) per counter."""
    return _mix_t(ctr * _s64(GAMMA) + _s64(key))


def normal_from_bits(z: torch.Tensor) -> torch.Tensor:
    hi = _lsr(z, 32).to(torch.float64)
    lo = (z & 0xFFFFFFFF).to(torch.float64)
    u1 = (hi + 0.5) * (1.0 / 4294967296.0)
    u2 = lo * (1.0 / 4294967296.0)
    return torch.sqrt(-2.0 * torch.log(u1)) * torch.cos((2.0 * math.pi) * u2)


def counters(b: int, tok0: int, ntok: int, heads: int, device) -> torch.Tensor:
    """Counter of element (b, token, head, channel): b<<48 | token<<15 | head<<7 | channel."""
    t = torch.arange(tok0, tok0 + ntok, dtype=torch.int64, device=device).view(-1, 1, 1)
    h = torch.arange(heads, dtype=torch.int64, device=device).view(1, -1, 1)
    c = torch.arange(128, dtype=torch.int64, device=device).view(1, 1, -1)
    return (int(b) << 48) + (t << 15) + (h << 7) + c


def k_offsets(seed: int, h_kv: int, device="cpu") -> torch.Tensor:
    """FP32 [h_kv][128] per-channel offsets, N(0, 4)."""
    ctr = torch.arange(h_kv * 128, dtype=torch.int64, device=device).view(h_kv, 128)
    z = random_bits(stream_key(seed, STREAM_KOFF), ctr)
    return (K_OFFSET_STD * normal_from_bits(z)).to(torch.float32)


def gen_tensor(seed: int, stream: int, b: int, tok0: int, ntok: int, heads: int, device="cpu",
               outliers: bool = False, out_stream: int = 0, offset: torch.Tensor | None = None,
               chunk_tokens: int = 4096) -> torch.Tensor:
    """bf16 [ntok][heads][128] for tokens tok0..tok0+ntok-1 of sequence b."""
    out = torch.empty((ntok, heads, 128), dtype=torch.bfloat16, device=device)
    key = stream_key(seed, stream)
    okey = stream_key(seed, out_stream) if outliers else 0
    thresh = int(OUTLIER_FRACTION * (1 << 53))
    for s in range(0, ntok, chunk_tokens):
        n = min(chunk_tokens, ntok - s)
        ctr = counters(b, tok0 + s, n, heads, device)
        x = normal_from_bits(random_bits(key, ctr))
        if outliers:
            zo = random_bits(okey, ctr)
            x = torch.where(_lsr(zo, 11) < thresh, x * OUTLIER_GAIN, x)
        x = x.to(torch.float32)
        if offset is not None:
            x = x + offset.to(device=device, dtype=torch.float32).view(1, heads, 128)
        out[s:s + n] = x.to(torch.bfloat16)
    return out


@dataclass
class PrefillWorkload:
    name: str
    batch: int
    h_q: int
    h_kv: int
    seqlens: list
    q_start: list
    kv_len: list
    outliers: bool
    seed: int
    smooth: bool = True

    @property
    def total_q(self) -> int:
        return int(sum(self.seqlens))

    def causal_pairs(self) -> int:
        """(query, key) pairs with key <= query, summed over sequences and q heads."""
        tot = 0
        for n, s in zip(self.seqlens, self.q_start):
            # query i (absolute s+i) sees s+i+1 keys
            tot += n * s + n * (n + 1) // 2
        return tot * self.h_q


@dataclass
class DecodeWorkload:
    name: str
    batch: int
    h_q: int
    h_kv: int
    kv_len: list
    seed: int
    outliers: bool = True
    smooth: bool = True
    qstat_tokens: int = 4096
    extra: dict = field(default_factory=dict)


def draw_lengths(seed: int, n: int, lo: int, hi: int) -> list:
    rng = np.random.default_rng(seed)
    return [int(x) for x in rng.integers(lo, hi + 1, size=n)]


def page_permutation(seed: int, n_pages: int) -> np.ndarray:
    return np.random.default_rng(seed + 7919).permutation(n_pages).astype(np.int32)


# The five workloads of the evaluation: shapes of Llama-3.1-8B (GQA 32:8) and
# Qwen3-14B (GQA 40:8), head_dim 128 (Sec. 7.1), contexts 16K-128K (Sec. 7.2).
def tiny_prefill() -> PrefillWorkload:
    return PrefillWorkload("tiny causal prefill 1x1 heads, 256 tokens", 1, 1, 1, [256], [0],
                           [256], outliers=False, seed=1)


def llama_prefill(seq: int = 16384) -> PrefillWorkload:
    return PrefillWorkload(f"llama-3.1-8b-shaped causal prefill, {seq} tokens, 32q/8kv heads",
                           1, 32, 8, [seq], [0], [seq], outliers=True, seed=2)


def qwen_prefill(seq: int = 131072) -> PrefillWorkload:
    return PrefillWorkload(f"qwen3-14b-shaped causal prefill, {seq} tokens, 40q/8kv heads",
                           1, 40, 8, [seq], [0], [seq], outliers=True, seed=3)


def llama_decode(batch: int = 32, lo: int = 16384, hi: int = 131072) -> DecodeWorkload:
    return DecodeWorkload(f"llama-3.1-8b-shaped paged decode, batch {batch}, contexts U[{lo},{hi}]",
                          batch, 32, 8, draw_lengths(4, batch, lo, hi), seed=4)


def mixed_step(n_decode: int = 64) -> tuple:
    pre = PrefillWorkload("qwen3-14b-shaped chunked prefill 32768 over a 65536 prefix", 1, 40, 8,
                          [32768], [65536], [98304], outliers=True, seed=5)
    dec = DecodeWorkload(f"qwen3-14b-shaped paged decode, batch {n_decode}, contexts U[8192,131072]",
                         n_decode, 40, 8, draw_lengths(55, n_decode, 8192, 131072), seed=55)
    return pre, dec


def gen_qkv(seed, seqlens, h_q, h_kv, outliers, device, tok_offsets=None, seq_ids=None):
    """Concatenated bf16 Q, K, V for sequences of the given lengths.  Entry i is
    sequence seq_ids[i] (default i) of the seeded stream, starting at its token
    tok_offsets[i] (default 0)."""
    qs, ks, vs = [], [], []
    off = k_offsets(seed, h_kv, device=device)
    for i, n in enumerate(seqlens):
        b = i if seq_ids is None else int(seq_ids[i])
        t0 = 0 if tok_offsets is None else int(tok_offsets[i])
        qs.append(gen_tensor(seed, STREAM_Q, b, t0, n, h_q, device, outliers, STREAM_OUT_Q))
        ks.append(gen_tensor(seed, STREAM_K, b, t0, n, h_kv, device, outliers, STREAM_OUT_K,
                             offset=off))
        vs.append(gen_tensor(seed, STREAM_V, b, t0, n, h_kv, device))
    return torch.cat(qs), torch.cat(ks), torch.cat(vs)


def make_pages(seed, kv_lens, shuffle=True):
    """Page table [B][max_pages] over a shared pool of 64-token pages, physical
    pages permuted.  Returns (page_table int32, pages used)."""
    need = [(int(n) + 63) // 64 for n in kv_lens]
    total = int(sum(need))
    perm = page_permutation(seed, total) if shuffle else np.arange(total, dtype=np.int32)
    maxp = max(need) if need else 1
    pt = np.zeros((len(kv_lens), max(maxp, 1)), np.int32)
    i = 0
    for b, n in enumerate(need):
        pt[b, :n] = perm[i:i + n]
        i += n
    return pt, total


def slots_for(page_table, b, positions):
    """Cache slots (page * 64 + offset) of key positions of sequence b."""
    positions = np.asarray(positions, np.int64)
    return page_table[b, positions // 64].astype(np.int64) * 64 + positions % 64


def bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> uint16 numpy bit patterns (CPU copy)."""
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
