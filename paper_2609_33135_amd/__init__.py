"""MI355X-native QK4PV8 FlashAttention (MpFA): thin Python binding of libmpfa.so.

Argument marshalling only: torch tensors provide device memory and the current
stream; every step of the attention path runs in the library's HIP kernels.
The binding raises if the compiled library is missing — there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
DEBUG_LIB_PATH = os.path.join(PKG_DIR, "libmpfa_debug.so")
# MPFA_DEBUG=1 loads the twin library whose entry points also check the data
# they are handed (index ranges, non-finite inputs) before launching
LIB_PATH = DEBUG_LIB_PATH if os.environ.get("MPFA_DEBUG") == "1" else os.path.join(PKG_DIR, "libmpfa.so")

(MPFA_OK, MPFA_ERR_INVALID, MPFA_ERR_UNSUPPORTED, MPFA_ERR_WORKSPACE, MPFA_ERR_HIP,
 MPFA_ERR_DATA) = range(6)
SMOOTH, COMPUTE_STATS, TSCALE_UNIT, SEED_MFMA, MXFP4, SEED_ELEMWISE = 1, 2, 4, 8, 16, 32
PV_BF16, PV_NVFP4 = 64, 128
HEAD_DIM, PAGE, TILE = 128, 64, 128
STATIC_SCRATCH_BYTES = 64 << 20   # MPFA_STATIC_SCRATCH_BYTES

EXPORTED = ("mpfa_quantize_qk", "mpfa_prefill", "mpfa_decode_workspace_size",
            "mpfa_decode_choose_partition", "mpfa_decode_paged", "mpfa_decode_paged_static",
            "mpfa_mixed_workspace_size",
            "mpfa_mixed_step", "mpfa_convert", "mpfa_status_string", "mpfa_version")


class MpfaError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} ({status})")
        self.status = status


class QuantArgs(C.Structure):
    _fields_ = [("batch", C.c_int32), ("total_tokens", C.c_int32), ("max_seqlen", C.c_int32),
                ("h_q", C.c_int32), ("h_kv", C.c_int32), ("head_dim", C.c_int32),
                ("flags", C.c_uint32), ("num_pages", C.c_int64),
                ("cu_seqlens", C.c_void_p), ("q", C.c_void_p), ("k", C.c_void_p),
                ("v", C.c_void_p), ("slot_mapping", C.c_void_p), ("q_mean", C.c_void_p),
                ("k_mean", C.c_void_p), ("k_tscale", C.c_void_p), ("q_codes", C.c_void_p),
                ("q_scales", C.c_void_p), ("q_tscale", C.c_void_p), ("k_codes", C.c_void_p),
                ("k_scales", C.c_void_p), ("v_codes", C.c_void_p), ("ds", C.c_void_p),
                ("v_aux", C.c_void_p)]


class PrefillArgs(C.Structure):
    _fields_ = [("batch", C.c_int32), ("h_q", C.c_int32), ("h_kv", C.c_int32),
                ("head_dim", C.c_int32), ("max_seqlen_q", C.c_int32), ("max_pages", C.c_int32),
                ("flags", C.c_uint32), ("cu_seqlens_q", C.c_void_p), ("q_start", C.c_void_p),
                ("kv_len", C.c_void_p), ("page_table", C.c_void_p), ("q_codes", C.c_void_p),
                ("q_scales", C.c_void_p), ("q_tscale", C.c_void_p), ("k_codes", C.c_void_p),
                ("k_scales", C.c_void_p), ("v_codes", C.c_void_p), ("ds", C.c_void_p),
                ("k_tscale", C.c_void_p), ("out", C.c_void_p), ("v_aux", C.c_void_p),
                ("num_pages", C.c_int64)]


class DecodeArgs(C.Structure):
    _fields_ = [("batch", C.c_int32), ("h_q", C.c_int32), ("h_kv", C.c_int32),
                ("head_dim", C.c_int32), ("max_pages", C.c_int32),
                ("partition_tokens", C.c_int32), ("max_partitions", C.c_int32),
                ("flags", C.c_uint32), ("kv_len", C.c_void_p), ("page_table", C.c_void_p),
                ("q_codes", C.c_void_p), ("q_scales", C.c_void_p), ("q_tscale", C.c_void_p),
                ("k_codes", C.c_void_p), ("k_scales", C.c_void_p), ("v_codes", C.c_void_p),
                ("ds", C.c_void_p), ("k_tscale", C.c_void_p), ("out", C.c_void_p),
                ("num_pages", C.c_int64)]


_libs: dict = {}


def lib():
    """Load libmpfa.so (built in-tree by build.py); raise if it is missing."""
    return _load(LIB_PATH)


def debug_lib():
    """Load libmpfa_debug.so: the same kernels behind entry points that also
    check the data (index ranges, non-finite inputs) and return MPFA_ERR_DATA."""
    return _load(DEBUG_LIB_PATH)


def _load(path):
    if path not in _libs:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run paper_2609_33135_amd/build.py")
        L = C.CDLL(path)
        L.mpfa_quantize_qk.restype = C.c_int
        L.mpfa_quantize_qk.argtypes = [C.POINTER(QuantArgs), C.c_void_p]
        L.mpfa_prefill.restype = C.c_int
        L.mpfa_prefill.argtypes = [C.POINTER(PrefillArgs), C.c_void_p]
        L.mpfa_decode_workspace_size.restype = C.c_int
        L.mpfa_decode_workspace_size.argtypes = [C.c_int32, C.c_int32, C.c_int32,
                                                 C.POINTER(C.c_size_t)]
        L.mpfa_decode_choose_partition.restype = C.c_int
        L.mpfa_decode_choose_partition.argtypes = [C.c_int32, C.c_void_p, C.c_int32, C.c_int32,
                                                   C.POINTER(C.c_int32)]
        L.mpfa_decode_paged.restype = C.c_int
        L.mpfa_decode_paged.argtypes = [C.POINTER(DecodeArgs), C.c_void_p, C.c_size_t, C.c_void_p]
        L.mpfa_decode_paged_static.restype = C.c_int
        L.mpfa_decode_paged_static.argtypes = [C.POINTER(DecodeArgs), C.c_void_p]
        L.mpfa_mixed_workspace_size.restype = C.c_int
        L.mpfa_mixed_workspace_size.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                                C.POINTER(C.c_size_t)]
        L.mpfa_mixed_step.restype = C.c_int
        L.mpfa_mixed_step.argtypes = [C.POINTER(PrefillArgs), C.POINTER(DecodeArgs), C.c_void_p,
                                      C.c_size_t, C.c_void_p]
        L.mpfa_convert.restype = C.c_int
        L.mpfa_convert.argtypes = [C.c_int32, C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p]
        L.mpfa_status_string.restype = C.c_char_p
        L.mpfa_status_string.argtypes = [C.c_int]
        L.mpfa_version.restype = C.c_char_p
        _libs[path] = L
    return _libs[path]


def status_string(s: int) -> str:
    return lib().mpfa_status_string(s).decode()


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _check(rc: int, what: str):
    if rc != MPFA_OK:
        raise MpfaError(rc, what)


class PagedCache:
    """Device buffers of the paged NVFP4/FP8 KV cache and the Delta_S side cache."""

    def __init__(self, num_pages: int, h_q: int, h_kv: int, device="cuda", smooth=True, pv=0):
        """pv: 0, PV_BF16 or PV_NVFP4 (adds the V copy of that precision, v_aux)."""
        import torch
        self.num_pages, self.h_q, self.h_kv = num_pages, h_q, h_kv
        u8 = dict(dtype=torch.uint8, device=device)
        self.k_codes = torch.zeros((num_pages, h_kv, PAGE, 64), **u8)
        self.k_scales = torch.zeros((num_pages, h_kv, PAGE, 8), **u8)
        self.v_codes = torch.zeros((num_pages, h_kv, HEAD_DIM, PAGE), **u8)
        self.ds = torch.zeros((num_pages, h_q, PAGE), dtype=torch.bfloat16, device=device) \
            if smooth else None
        self.v_aux = None
        if pv == PV_BF16:
            self.v_aux = torch.zeros((num_pages, h_kv, HEAD_DIM, PAGE), dtype=torch.bfloat16,
                                     device=device)
        elif pv == PV_NVFP4:   # code plane [P][H][128][32], then scale plane [P][H][128][4]
            self.v_aux = torch.zeros(num_pages * h_kv * HEAD_DIM * 36, **u8)


class SeqStats:
    """Per-sequence statistics frozen after the first prefill (means, K tensor scale)."""

    def __init__(self, batch: int, h_q: int, h_kv: int, device="cuda"):
        import torch
        self.q_mean = torch.zeros((batch, h_q, HEAD_DIM), dtype=torch.bfloat16, device=device)
        self.k_mean = torch.zeros((batch, h_kv, HEAD_DIM), dtype=torch.bfloat16, device=device)
        self.k_tscale = torch.ones((batch, h_kv), dtype=torch.float32, device=device)


class QuantQ:
    """NVFP4 queries of one call: codes [T][H][64], scales [T][H][8], tensor scale [B][H]."""

    def __init__(self, total: int, batch: int, h_q: int, device="cuda"):
        import torch
        self.codes = torch.zeros((total, h_q, 64), dtype=torch.uint8, device=device)
        self.scales = torch.zeros((total, h_q, 8), dtype=torch.uint8, device=device)
        self.tscale = torch.zeros((batch, h_q), dtype=torch.float32, device=device)


def quantize_qk(q, k, v, cu_seqlens, slot_mapping, cache: PagedCache, stats: SeqStats,
                qout: QuantQ, flags: int, max_seqlen: int, stream=None):
    """mpfa_quantize_qk: q bf16 [T][Hq][128], k/v bf16 [T][Hkv][128] on the device."""
    T, h_q, d = q.shape
    a = QuantArgs(batch=cu_seqlens.numel() - 1, total_tokens=T, max_seqlen=max_seqlen, h_q=h_q,
                  h_kv=k.shape[1], head_dim=d, flags=flags, num_pages=cache.num_pages,
                  cu_seqlens=_ptr(cu_seqlens), q=_ptr(q), k=_ptr(k), v=_ptr(v),
                  slot_mapping=_ptr(slot_mapping), q_mean=_ptr(stats.q_mean),
                  k_mean=_ptr(stats.k_mean), k_tscale=_ptr(stats.k_tscale),
                  q_codes=_ptr(qout.codes), q_scales=_ptr(qout.scales),
                  q_tscale=_ptr(qout.tscale), k_codes=_ptr(cache.k_codes),
                  k_scales=_ptr(cache.k_scales), v_codes=_ptr(cache.v_codes), ds=_ptr(cache.ds),
                  v_aux=_ptr(cache.v_aux))
    _check(lib().mpfa_quantize_qk(C.byref(a), _stream(stream)), "mpfa_quantize_qk")


def prefill(qq: QuantQ, cache: PagedCache, stats: SeqStats, cu_seqlens_q, q_start, kv_len,
            page_table, out, max_seqlen_q: int, flags: int, stream=None):
    """mpfa_prefill: causal attention of the quantized queries over the paged cache."""
    a = PrefillArgs(batch=cu_seqlens_q.numel() - 1, h_q=qq.codes.shape[1], h_kv=cache.h_kv,
                    head_dim=HEAD_DIM, max_seqlen_q=max_seqlen_q, max_pages=page_table.shape[1],
                    flags=flags, cu_seqlens_q=_ptr(cu_seqlens_q), q_start=_ptr(q_start),
                    kv_len=_ptr(kv_len), page_table=_ptr(page_table), q_codes=_ptr(qq.codes),
                    q_scales=_ptr(qq.scales), q_tscale=_ptr(qq.tscale),
                    k_codes=_ptr(cache.k_codes), k_scales=_ptr(cache.k_scales),
                    v_codes=_ptr(cache.v_codes), ds=_ptr(cache.ds),
                    k_tscale=_ptr(stats.k_tscale), out=_ptr(out), v_aux=_ptr(cache.v_aux),
                    num_pages=cache.num_pages)
    _check(lib().mpfa_prefill(C.byref(a), _stream(stream)), "mpfa_prefill")


def decode_workspace_size(batch: int, h_q: int, max_partitions: int) -> int:
    n = C.c_size_t(0)
    _check(lib().mpfa_decode_workspace_size(batch, h_q, max_partitions, C.byref(n)),
           "mpfa_decode_workspace_size")
    return n.value


def decode_choose_partition(kv_len_host, h_kv: int, num_cus: int) -> int:
    import numpy as np
    kl = np.ascontiguousarray(kv_len_host, dtype=np.int32)
    out = C.c_int32(0)
    _check(lib().mpfa_decode_choose_partition(kl.size, kl.ctypes.data, h_kv, num_cus,
                                              C.byref(out)), "mpfa_decode_choose_partition")
    return out.value


def decode_paged(qq: QuantQ, cache: PagedCache, stats: SeqStats, kv_len, page_table, out,
                 partition_tokens: int, max_partitions: int, workspace, flags: int, stream=None):
    """mpfa_decode_paged: one query per sequence (qq rows indexed by sequence)."""
    a = DecodeArgs(batch=kv_len.numel(), h_q=qq.codes.shape[1], h_kv=cache.h_kv,
                   head_dim=HEAD_DIM, max_pages=page_table.shape[1],
                   partition_tokens=partition_tokens, max_partitions=max_partitions, flags=flags,
                   kv_len=_ptr(kv_len), page_table=_ptr(page_table), q_codes=_ptr(qq.codes),
                   q_scales=_ptr(qq.scales), q_tscale=_ptr(qq.tscale),
                   k_codes=_ptr(cache.k_codes), k_scales=_ptr(cache.k_scales),
                   v_codes=_ptr(cache.v_codes), ds=_ptr(cache.ds),
                   k_tscale=_ptr(stats.k_tscale), out=_ptr(out), num_pages=cache.num_pages)
    _check(lib().mpfa_decode_paged(C.byref(a), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream)),
           "mpfa_decode_paged")


def _decode_args(qq, cache, stats, kv_len, page_table, out, partition_tokens, max_partitions, flags):
    return DecodeArgs(batch=kv_len.numel(), h_q=qq.codes.shape[1], h_kv=cache.h_kv,
                      head_dim=HEAD_DIM, max_pages=page_table.shape[1],
                      partition_tokens=partition_tokens, max_partitions=max_partitions, flags=flags,
                      kv_len=_ptr(kv_len), page_table=_ptr(page_table), q_codes=_ptr(qq.codes),
                      q_scales=_ptr(qq.scales), q_tscale=_ptr(qq.tscale),
                      k_codes=_ptr(cache.k_codes), k_scales=_ptr(cache.k_scales),
                      v_codes=_ptr(cache.v_codes), ds=_ptr(cache.ds),
                      k_tscale=_ptr(stats.k_tscale), out=_ptr(out), num_pages=cache.num_pages)


def decode_paged_static(qq: QuantQ, cache: PagedCache, stats: SeqStats, kv_len, page_table, out,
                        partition_tokens: int, max_partitions: int, flags: int, stream=None):
    """mpfa_decode_paged_static: decode_paged with the partition states in the
    library's per-GPU scratch array instead of a caller workspace (for callers
    that cannot allocate; calls on one GPU must not overlap)."""
    a = _decode_args(qq, cache, stats, kv_len, page_table, out, partition_tokens, max_partitions, flags)
    _check(lib().mpfa_decode_paged_static(C.byref(a), _stream(stream)), "mpfa_decode_paged_static")


def mixed_workspace_size(batch: int, h_q: int, h_kv: int, max_partitions: int) -> int:
    n = C.c_size_t(0)
    _check(lib().mpfa_mixed_workspace_size(batch, h_q, h_kv, max_partitions, C.byref(n)),
           "mpfa_mixed_workspace_size")
    return n.value


def mixed_step(pre: dict, dec: dict, workspace, flags: int, stream=None):
    """mpfa_mixed_step: one launch for a prefill (keyword arguments of prefill())
    and a decode (keyword arguments of decode_paged() without the workspace and
    flags); the workspace must start zeroed (torch.zeros) and stays zeroed."""
    qq, cache, stats = pre["qq"], pre["cache"], pre["stats"]
    pa = PrefillArgs(batch=pre["cu_seqlens_q"].numel() - 1, h_q=qq.codes.shape[1], h_kv=cache.h_kv,
                     head_dim=HEAD_DIM, max_seqlen_q=pre["max_seqlen_q"],
                     max_pages=pre["page_table"].shape[1], flags=flags,
                     cu_seqlens_q=_ptr(pre["cu_seqlens_q"]), q_start=_ptr(pre["q_start"]),
                     kv_len=_ptr(pre["kv_len"]), page_table=_ptr(pre["page_table"]),
                     q_codes=_ptr(qq.codes), q_scales=_ptr(qq.scales), q_tscale=_ptr(qq.tscale),
                     k_codes=_ptr(cache.k_codes), k_scales=_ptr(cache.k_scales),
                     v_codes=_ptr(cache.v_codes), ds=_ptr(cache.ds), k_tscale=_ptr(stats.k_tscale),
                     out=_ptr(pre["out"]), v_aux=None, num_pages=cache.num_pages)
    qd, dcache, dstats = dec["qq"], dec["cache"], dec["stats"]
    da = DecodeArgs(batch=dec["kv_len"].numel(), h_q=qd.codes.shape[1], h_kv=dcache.h_kv,
                    head_dim=HEAD_DIM, max_pages=dec["page_table"].shape[1],
                    partition_tokens=dec["partition_tokens"], max_partitions=dec["max_partitions"],
                    flags=flags, kv_len=_ptr(dec["kv_len"]), page_table=_ptr(dec["page_table"]),
                    q_codes=_ptr(qd.codes), q_scales=_ptr(qd.scales), q_tscale=_ptr(qd.tscale),
                    k_codes=_ptr(dcache.k_codes), k_scales=_ptr(dcache.k_scales),
                    v_codes=_ptr(dcache.v_codes), ds=_ptr(dcache.ds), k_tscale=_ptr(dstats.k_tscale),
                    out=_ptr(dec["out"]), num_pages=dcache.num_pages)
    _check(lib().mpfa_mixed_step(C.byref(pa), C.byref(da), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _stream(stream)),
           "mpfa_mixed_step")


def convert(fmt: int, x, out, stream=None):
    """mpfa_convert: fmt 0 FP32 -> E4M3, fmt 1 FP32 -> E2M1 (one code per byte),
    written from the format definitions; fmt 2 / 3 the same through the hardware
    converters the quantization pass uses; 0x100 + c: E2M1 of x / e4m3(c) by the
    NVFP4 quantizer's division; 0x200 + b: E2M1 of x / 2^(b-127) (MXFP4);
    0x300 + c / 0x400 + b: the same quotients from their definitions (IEEE
    division, exact scaling) through the fmt 1 encoder."""
    _check(lib().mpfa_convert(fmt, _ptr(x), x.numel(), _ptr(out), _stream(stream)), "mpfa_convert")
