"""ctypes binding of the CPU oracle (liboracle.so).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the CPU
baseline leg of the benchmark.  The product package never imports it.

Arrays are numpy; bf16 data travels as uint16 bit patterns.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")
SRC = os.path.join(HERE, "mpfa_oracle.c")

SMOOTH = 1
COMPUTE_STATS = 2
TSCALE_UNIT = 4
MXFP4 = 8
PV_BF16 = 16        # V in BF16 (v_aux), P rounded to BF16
PV_NVFP4 = 32       # V as NVFP4 along keys (v_aux), P as NVFP4 per 16 keys
QUANT_P = 1
REVERSE = 2
P_BF16 = 4
P_NVFP4 = 8

D = 128
PAGE = 64


def build(force: bool = False) -> str:
    """Compile liboracle.so with gcc (IEEE semantics: no fast-math, no FP contraction)."""
    if force or not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC):
        cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
               "-Wall", "-o", LIB_PATH + ".tmp", SRC, "-lm"]
        subprocess.check_call(cmd, cwd=HERE)
        os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


_lib = None


class _QuantArgs(C.Structure):
    _fields_ = [("batch", C.c_int32), ("total_tokens", C.c_int32), ("h_q", C.c_int32),
                ("h_kv", C.c_int32), ("flags", C.c_int32),
                ("cu_seqlens", C.c_void_p), ("q", C.c_void_p), ("k", C.c_void_p),
                ("v", C.c_void_p), ("slot_mapping", C.c_void_p),
                ("q_mean", C.c_void_p), ("k_mean", C.c_void_p), ("k_tscale", C.c_void_p),
                ("q_codes", C.c_void_p), ("q_scales", C.c_void_p), ("q_tscale", C.c_void_p),
                ("k_codes", C.c_void_p), ("k_scales", C.c_void_p), ("v_codes", C.c_void_p),
                ("ds", C.c_void_p), ("v_aux", C.c_void_p), ("num_pages", C.c_int64)]


class _Cache(C.Structure):
    _fields_ = [("batch", C.c_int32), ("h_q", C.c_int32), ("h_kv", C.c_int32),
                ("max_pages", C.c_int32), ("flags", C.c_int32),
                ("page_table", C.c_void_p), ("kv_len", C.c_void_p),
                ("k_codes", C.c_void_p), ("k_scales", C.c_void_p), ("v_codes", C.c_void_p),
                ("ds", C.c_void_p), ("k_tscale", C.c_void_p),
                ("q_codes", C.c_void_p), ("q_scales", C.c_void_p), ("q_tscale", C.c_void_p),
                ("v_aux", C.c_void_p), ("num_pages", C.c_int64)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = C.CDLL(LIB_PATH)
        L.orc_e2m1_value.restype = C.c_double
        L.orc_e2m1_value.argtypes = [C.c_uint8]
        L.orc_e2m1_encode.restype = C.c_uint8
        L.orc_e2m1_encode.argtypes = [C.c_double]
        L.orc_e4m3_value.restype = C.c_double
        L.orc_e4m3_value.argtypes = [C.c_uint8]
        L.orc_e4m3_encode.restype = C.c_uint8
        L.orc_e4m3_encode.argtypes = [C.c_double]
        L.orc_bf16_encode_f64.restype = C.c_uint16
        L.orc_bf16_encode_f64.argtypes = [C.c_double]
        L.orc_tensor_scale.restype = C.c_float
        L.orc_tensor_scale.argtypes = [C.c_float]
        for name in ("orc_e4m3_encode_f32_array", "orc_e2m1_encode_f32_array",
                     "orc_bf16_encode_f32_array"):
            getattr(L, name).restype = None
            getattr(L, name).argtypes = [C.c_void_p, C.c_int64, C.c_void_p]
        L.orc_nvfp4_row.restype = None
        L.orc_nvfp4_row.argtypes = [C.c_void_p, C.c_float, C.c_void_p, C.c_void_p]
        L.orc_nvfp4_dequant_row.restype = None
        L.orc_nvfp4_dequant_row.argtypes = [C.c_void_p, C.c_void_p, C.c_double, C.c_void_p]
        L.orc_mxfp4_row.restype = None
        L.orc_mxfp4_row.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
        L.orc_mxfp4_dequant_row.restype = None
        L.orc_mxfp4_dequant_row.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
        L.orc_stats_one.restype = None
        L.orc_stats_one.argtypes = [C.c_void_p, C.c_int64, C.c_int64, C.c_int, C.c_int,
                                    C.c_void_p, C.c_void_p]
        L.orc_quantize_qk.restype = C.c_int
        L.orc_quantize_qk.argtypes = [C.POINTER(_QuantArgs)]
        L.orc_attention_f64.restype = None
        L.orc_attention_f64.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                        C.c_void_p, C.c_int64, C.c_int64, C.c_int, C.c_int64,
                                        C.c_int, C.c_void_p]
        L.orc_attention_textbook.restype = None
        L.orc_attention_textbook.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                             C.c_int64, C.c_int64, C.c_void_p]
        L.orc_prefill.restype = C.c_int
        L.orc_prefill.argtypes = [C.POINTER(_Cache), C.c_void_p, C.c_void_p, C.c_int64,
                                  C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.orc_decode.restype = C.c_int
        L.orc_decode.argtypes = [C.POINTER(_Cache), C.c_int32, C.c_int64, C.c_void_p,
                                 C.c_void_p, C.c_void_p, C.c_void_p]
        L.orc_num_threads.restype = C.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ---- number formats ---------------------------------------------------------

def e2m1_value(code: int) -> float:
    return lib().orc_e2m1_value(code)


def e4m3_value(code: int) -> float:
    return lib().orc_e4m3_value(code)


def e2m1_encode(x) -> np.ndarray:
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint8)
    lib().orc_e2m1_encode_f32_array(_p(x), x.size, _p(out))
    return out


def e4m3_encode(x) -> np.ndarray:
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint8)
    lib().orc_e4m3_encode_f32_array(_p(x), x.size, _p(out))
    return out


def e4m3_encode_f64(x: float) -> int:
    return lib().orc_e4m3_encode(float(x))


def bf16_encode(x) -> np.ndarray:
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().orc_bf16_encode_f32_array(_p(x), x.size, _p(out))
    return out


def bf16_encode_f64(x: float) -> int:
    return lib().orc_bf16_encode_f64(float(x))


def bf16_to_f32(bits) -> np.ndarray:
    bits = _c(bits, np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32)


def tensor_scale(amax: float) -> float:
    return float(lib().orc_tensor_scale(float(amax)))


def nvfp4_row(xc, t: float):
    xc = _c(xc, np.float32)
    assert xc.shape == (D,)
    codes = np.empty(64, np.uint8)
    scales = np.empty(8, np.uint8)
    lib().orc_nvfp4_row(_p(xc), float(t), _p(codes), _p(scales))
    return codes, scales


def mxfp4_row(xc):
    """MXFP4 codes (64 bytes) and scale bytes (8; 0..3 used) of one centered row."""
    xc = _c(xc, np.float32)
    assert xc.shape == (D,)
    codes = np.empty(64, np.uint8)
    scales = np.empty(8, np.uint8)
    lib().orc_mxfp4_row(_p(xc), _p(codes), _p(scales))
    return codes, scales


def mxfp4_dequant_row(codes, scales) -> np.ndarray:
    codes = _c(codes, np.uint8)
    scales = _c(scales, np.uint8)
    out = np.empty(D, np.float64)
    lib().orc_mxfp4_dequant_row(_p(codes), _p(scales), _p(out))
    return out


def nvfp4_dequant_row(codes, scales, t: float) -> np.ndarray:
    codes = _c(codes, np.uint8)
    scales = _c(scales, np.uint8)
    out = np.empty(D, np.float64)
    lib().orc_nvfp4_dequant_row(_p(codes), _p(scales), float(t), _p(out))
    return out


def stats_one(x_bf16, smooth=True, tscale_unit=False):
    """x_bf16: uint16 [n][128]."""
    x = _c(x_bf16, np.uint16)
    n = x.shape[0]
    mean = np.empty(D, np.uint16)
    t = np.empty(1, np.float32)
    lib().orc_stats_one(_p(x), n, D, int(smooth), int(tscale_unit), _p(mean), _p(t))
    return mean, float(t[0])


# ---- quantization pass --------------------------------------------------------

def v_aux_nvfp4_planes(aux, n_pages, h_kv):
    """Views of an NVFP4 v_aux buffer: codes [pages][h_kv][128][32] and
    E4M3 scales [pages][h_kv][128][4]."""
    n = n_pages * h_kv * D
    return aux[:n * 32].reshape(n_pages, h_kv, D, 32), aux[n * 32:n * 36].reshape(n_pages, h_kv, D, 4)


def quantize_qk(q, k, v, cu_seqlens, slot_mapping, n_pages, flags,
                q_mean=None, k_mean=None, k_tscale=None, cache=None):
    """q: uint16 [T][Hq][128], k/v: uint16 [T][Hkv][128] (bf16 bits).

    Returns a dict with the quantized query, the cache arrays and the statistics.
    `cache` (a dict from a previous call) is updated in place when given, so that
    appended tokens land in the same pages.
    """
    q = _c(q, np.uint16)
    k = _c(k, np.uint16)
    v = _c(v, np.uint16)
    T, Hq, _ = q.shape
    Hkv = k.shape[1]
    cu = _c(cu_seqlens, np.int32)
    B = cu.shape[0] - 1
    sm = _c(slot_mapping, np.int64)
    if cache is None:
        cache = {
            "k_codes": np.zeros((n_pages, Hkv, PAGE, 64), np.uint8),
            "k_scales": np.zeros((n_pages, Hkv, PAGE, 8), np.uint8),
            "v_codes": np.zeros((n_pages, Hkv, D, PAGE), np.uint8),
            "ds": np.zeros((n_pages, Hq, PAGE), np.uint16),
        }
    if (flags & PV_BF16) and "v_aux" not in cache:
        cache["v_aux"] = np.zeros((n_pages, Hkv, D, PAGE), np.uint16)
    if (flags & PV_NVFP4) and "v_aux" not in cache:
        # code plane [pages][Hkv][128][32], then scale plane [pages][Hkv][128][4]
        cache["v_aux"] = np.zeros(n_pages * Hkv * D * 36, np.uint8)
    stats = flags & COMPUTE_STATS
    if stats:
        q_mean = np.zeros((B, Hq, D), np.uint16)
        k_mean = np.zeros((B, Hkv, D), np.uint16)
        k_tscale = np.zeros((B, Hkv), np.float32)
    else:
        q_mean = _c(q_mean, np.uint16).copy()
        k_mean = _c(k_mean, np.uint16).copy()
        k_tscale = _c(k_tscale, np.float32).copy()
    out = {
        "q_codes": np.zeros((T, Hq, 64), np.uint8),
        "q_scales": np.zeros((T, Hq, 8), np.uint8),
        "q_tscale": np.zeros((B, Hq), np.float32),
    }
    a = _QuantArgs(B, T, Hq, Hkv, flags, _p(cu), _p(q), _p(k), _p(v), _p(sm),
                   _p(q_mean), _p(k_mean), _p(k_tscale),
                   _p(out["q_codes"]), _p(out["q_scales"]), _p(out["q_tscale"]),
                   _p(cache["k_codes"]), _p(cache["k_scales"]), _p(cache["v_codes"]),
                   _p(cache["ds"]), _p(cache.get("v_aux")), cache["k_codes"].shape[0])
    rc = lib().orc_quantize_qk(C.byref(a))
    if rc != 0:
        raise ValueError("orc_quantize_qk rejected its arguments")
    out.update(cache=cache, q_mean=q_mean, k_mean=k_mean, k_tscale=k_tscale)
    return out


# ---- attention ------------------------------------------------------------------

def attention_f64(q, k, v, ds=None, q_pos=None, tile=128, partition=0, flags=REVERSE):
    q = _c(q, np.float64)
    k = _c(k, np.float64)
    v = _c(v, np.float64)
    nq, nk = q.shape[0], k.shape[0]
    if q_pos is None:
        q_pos = np.full(nq, nk - 1, np.int64)
    q_pos = _c(q_pos, np.int64)
    if ds is not None:
        ds = _c(ds, np.float64)
        assert ds.shape == (nq, nk)
    out = np.empty((nq, D), np.float64)
    lib().orc_attention_f64(_p(q), _p(k), _p(v), _p(ds), _p(q_pos), nq, nk, int(tile),
                            int(partition), int(flags), _p(out))
    return out


def attention_textbook(q, k, v, q_pos=None):
    q = _c(q, np.float64)
    k = _c(k, np.float64)
    v = _c(v, np.float64)
    nq, nk = q.shape[0], k.shape[0]
    if q_pos is None:
        q_pos = np.full(nq, nk - 1, np.int64)
    q_pos = _c(q_pos, np.int64)
    out = np.empty((nq, D), np.float64)
    lib().orc_attention_textbook(_p(q), _p(k), _p(v), _p(q_pos), nq, nk, _p(out))
    return out


def _cache_struct(cache, page_table, kv_len, k_tscale, q_codes, q_scales, q_tscale, h_q,
                  flags, keep):
    pt = _c(page_table, np.int32)
    kl = _c(kv_len, np.int32)
    arrs = dict(k_codes=_c(cache["k_codes"], np.uint8), k_scales=_c(cache["k_scales"], np.uint8),
                v_codes=_c(cache["v_codes"], np.uint8), ds=_c(cache["ds"], np.uint16),
                k_tscale=_c(k_tscale, np.float32), q_codes=_c(q_codes, np.uint8),
                q_scales=_c(q_scales, np.uint8), q_tscale=_c(q_tscale, np.float32), pt=pt, kl=kl)
    if flags & (PV_BF16 | PV_NVFP4):
        arrs["v_aux"] = np.ascontiguousarray(cache["v_aux"])
    keep.append(arrs)
    h_kv = arrs["k_codes"].shape[1]
    return _Cache(pt.shape[0], h_q, h_kv, pt.shape[1], flags, _p(pt), _p(kl),
                  _p(arrs["k_codes"]), _p(arrs["k_scales"]), _p(arrs["v_codes"]),
                  _p(arrs["ds"]), _p(arrs["k_tscale"]), _p(arrs["q_codes"]),
                  _p(arrs["q_scales"]), _p(arrs["q_tscale"]), _p(arrs.get("v_aux")),
                  arrs["k_codes"].shape[0])


def prefill(cache, page_table, kv_len, k_tscale, q_codes, q_scales, q_tscale, cu_seqlens,
            q_start, items, smooth=True, mxfp4=False, pv=0):
    """items: int32 [n][3] rows of (sequence, row within sequence, q head).
    pv: 0 (FP8 P and V), PV_BF16 or PV_NVFP4 (precision assignments of the PV
    product compared in Sec. 3.1; the cache then carries v_aux).
    Returns (bf16 bits [n][128], float64 [n][128])."""
    keep = []
    h_q = q_codes.shape[1]
    cs = _cache_struct(cache, page_table, kv_len, k_tscale, q_codes, q_scales, q_tscale, h_q,
                       (SMOOTH if smooth else 0) | (MXFP4 if mxfp4 else 0) | pv, keep)
    items = _c(items, np.int32).reshape(-1, 3)
    ib, ir, ih = (np.ascontiguousarray(items[:, i]) for i in range(3))
    cu = _c(cu_seqlens, np.int32)
    qs = _c(q_start, np.int32)
    n = items.shape[0]
    o16 = np.empty((n, D), np.uint16)
    o64 = np.empty((n, D), np.float64)
    rc = lib().orc_prefill(C.byref(cs), _p(cu), _p(qs), n, _p(ib), _p(ir), _p(ih), _p(o16),
                           _p(o64))
    assert rc == 0
    return o16, o64


def decode(cache, page_table, kv_len, k_tscale, q_codes, q_scales, q_tscale, partition_tokens,
           items, smooth=True, mxfp4=False):
    """items: int32 [n][2] rows of (sequence, q head); q_codes indexed by sequence."""
    keep = []
    h_q = q_codes.shape[1]
    cs = _cache_struct(cache, page_table, kv_len, k_tscale, q_codes, q_scales, q_tscale, h_q,
                       (SMOOTH if smooth else 0) | (MXFP4 if mxfp4 else 0), keep)
    items = _c(items, np.int32).reshape(-1, 2)
    ib, ih = (np.ascontiguousarray(items[:, i]) for i in range(2))
    n = items.shape[0]
    o16 = np.empty((n, D), np.uint16)
    o64 = np.empty((n, D), np.float64)
    rc = lib().orc_decode(C.byref(cs), int(partition_tokens), n, _p(ib), _p(ih), _p(o16), _p(o64))
    if rc != 0:
        raise ValueError("orc_decode rejected its arguments")
    return o16, o64


def num_threads() -> int:
    return lib().orc_num_threads()
