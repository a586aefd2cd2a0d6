"""Binding of libmpfa_probe.so, the measurement probes of include/mpfa_probe.h:
the achievable issue rate of each MFMA form the attention kernels use and the
achievable HBM read rate, measured on the device.  The benchmark loads it for
the second denominators of its roofline fractions; the product library does
not contain these kernels."""
from __future__ import annotations

import ctypes as C
import os

from . import MPFA_OK, PKG_DIR, MpfaError, _ptr, _stream

PROBE_LIB_PATH = os.path.join(PKG_DIR, "libmpfa_probe.so")
EXPORTED = ("mpfa_probe_mfma", "mpfa_probe_read")
PROBE_MFMA_F16, PROBE_MFMA_FP8, PROBE_MFMA_FP4 = 0, 1, 2
PROBE_READ_VGPR, PROBE_READ_LDS = 0, 1

_lib = None


def lib():
    """Load libmpfa_probe.so (built in-tree by build.py); raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(PROBE_LIB_PATH):
            raise RuntimeError(f"{PROBE_LIB_PATH} is not built; run paper_2609_33135_amd/build.py")
        L = C.CDLL(PROBE_LIB_PATH)
        L.mpfa_probe_mfma.restype = C.c_int
        L.mpfa_probe_mfma.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_uint32, C.c_uint32, C.c_void_p,
                                      C.c_void_p]
        L.mpfa_probe_read.restype = C.c_int
        L.mpfa_probe_read.argtypes = [C.c_int32, C.c_void_p, C.c_int64, C.c_int32, C.c_void_p, C.c_void_p]
        _lib = L
    return _lib


def _check(rc: int, what: str):
    if rc != MPFA_OK:
        raise MpfaError(rc, what)


# Operand words that make every A and B element 1.0 in each probe form.
PROBE_ONES = {PROBE_MFMA_F16: 0x3C003C00, PROBE_MFMA_FP8: 0x38383838, PROBE_MFMA_FP4: 0x22222222}


def probe_mfma(kind: int, iters: int, blocks: int, sink, pa=None, pb=None, stream=None):
    """mpfa_probe_mfma: `blocks` x 4 waves, each `iters` rounds of 8 MFMAs of
    form `kind`; sink is a float32 tensor of blocks * 256 elements.  Returns the
    FLOP count of the launch."""
    pa = PROBE_ONES[kind] if pa is None else pa
    pb = PROBE_ONES[kind] if pb is None else pb
    _check(lib().mpfa_probe_mfma(kind, iters, blocks, pa, pb, _ptr(sink), _stream(stream)), "mpfa_probe_mfma")
    k = 32 if kind == PROBE_MFMA_F16 else 128
    return blocks * 4 * iters * 8 * (2 * 16 * 16 * k)


def probe_read(mode: int, buf, blocks: int, sink, stream=None):
    """mpfa_probe_read: read every byte of the device tensor `buf` once; sink is
    an int32 tensor of blocks * 256 elements (XOR of each thread's words)."""
    nbytes = buf.numel() * buf.element_size()
    _check(lib().mpfa_probe_read(mode, _ptr(buf), nbytes, blocks, _ptr(sink), _stream(stream)),
           "mpfa_probe_read")
    return nbytes
