"""Python binding of the ps_lda C ABI (include/ps_lda.h): argument marshalling only.

Collapsed Gibbs sampling for LDA under clocked SSP / ESSP runs in the HIP kernels of
``libps_mf.so``; this module converts numpy arrays and torch streams into the plain
pointers the C functions take.  The functions keep the C names; ``PsLda`` wraps a handle.
The library is required: importing this module raises if it is not built.
"""
from __future__ import annotations

import ctypes

import numpy as np

from paper_1410_8043_amd import ps_mf as _mf

LIB_PATH = _mf.LIB_PATH
OK, EINVAL, ENOMEM, EDEVICE, ESTATE = 0, -1, -2, -3, -4
OPT_POLICY, OPT_MB_BLOCKS, OPT_SEED, OPT_HOST_ONLY, OPT_TIMING, OPT_FLAT_ADDRESSING = range(1, 7)
SSP_LAZY, SSP_WORST, ESSP = 0, 1, 2
X_Z, X_NDK, X_NWK, X_VERSION_LOG, X_BLOCK_ORDER = range(5)

SYMBOLS = ("ps_lda_create", "ps_lda_set_option", "ps_lda_set_stream", "ps_lda_load", "ps_lda_clock", "ps_lda_loglik",
           "ps_lda_get_clock", "ps_lda_export", "ps_lda_kernel_time", "ps_lda_last_error", "ps_lda_destroy")


def _bind():
    lib = ctypes.CDLL(LIB_PATH)
    i64, i32, dbl, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_void_p
    sig = {
        "ps_lda_create": [i64, i64, i32, i32, i32, dbl, dbl, ctypes.POINTER(vp)],
        "ps_lda_set_option": [vp, i32, i64],
        "ps_lda_set_stream": [vp, vp],
        "ps_lda_load": [vp, vp, vp, vp, i64],
        "ps_lda_clock": [vp, i32],
        "ps_lda_loglik": [vp, ctypes.POINTER(dbl)],
        "ps_lda_get_clock": [vp, ctypes.POINTER(i64)],
        "ps_lda_export": [vp, i32, i32, vp, i64, ctypes.POINTER(i64)],
        "ps_lda_kernel_time": [vp, ctypes.POINTER(dbl), ctypes.POINTER(i64)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.ps_lda_last_error.argtypes = [vp]
    lib.ps_lda_last_error.restype = ctypes.c_char_p
    lib.ps_lda_destroy.argtypes = [vp]
    lib.ps_lda_destroy.restype = None
    return lib


_lib = _bind()


class PsLdaError(RuntimeError):
    def __init__(self, func, code, msg):
        super().__init__(f"{func} failed ({code}): {msg}")
        self.code = code


def _check(h, func, rc):
    if rc != OK:
        msg = _lib.ps_lda_last_error(h) if h else b""
        raise PsLdaError(func, rc, (msg or b"").decode(errors="replace"))


def ps_lda_create(D, V, K, P, s, alpha, beta):
    h = ctypes.c_void_p()
    _check(None, "ps_lda_create", _lib.ps_lda_create(int(D), int(V), int(K), int(P), int(s), float(alpha),
                                                      float(beta), ctypes.byref(h)))
    return h


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


class PsLda:
    """One handle: create, set options, load tokens, run clocks, read the state back."""

    def __init__(self, D, V, K, P, s, alpha, beta, policy=ESSP, B=2, seed=0, host_only=False, timing=False,
                 stream=None, flat=False):
        self.D, self.V, self.K, self.P, self.s, self.B = int(D), int(V), int(K), int(P), int(s), int(B)
        self._h = ps_lda_create(D, V, K, P, s, alpha, beta)
        for key, val in ((OPT_POLICY, policy), (OPT_MB_BLOCKS, B), (OPT_SEED, int(seed) & (2**64 - 1)),
                         (OPT_HOST_ONLY, int(host_only)), (OPT_TIMING, int(timing)), (OPT_FLAT_ADDRESSING, int(flat))):
            if key == OPT_SEED and val >= 2**63:
                val -= 2**64  # the C side takes the 64 bits as int64_t
            _check(self._h, "ps_lda_set_option", _lib.ps_lda_set_option(self._h, key, int(val)))
        if stream is not None:
            self.set_stream(stream)

    def close(self):
        if self._h:
            _lib.ps_lda_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_stream(self, stream):
        ptr = getattr(stream, "cuda_stream", stream)
        _check(self._h, "ps_lda_set_stream", _lib.ps_lda_set_stream(self._h, ctypes.c_void_p(int(ptr or 0))))

    def load(self, doc, word, z0):
        doc, word, z0 = _i32(doc), _i32(word), _i32(z0)
        n = doc.shape[0]
        if word.shape[0] != n or z0.shape[0] != n:
            raise ValueError("doc, word and z0 must have one entry per token")
        ptr = (lambda a: a.ctypes.data if n else None)
        _check(self._h, "ps_lda_load", _lib.ps_lda_load(self._h, ptr(doc), ptr(word), ptr(z0), n))

    def clock(self, n=1):
        _check(self._h, "ps_lda_clock", _lib.ps_lda_clock(self._h, int(n)))

    def loglik(self) -> float:
        out = ctypes.c_double()
        _check(self._h, "ps_lda_loglik", _lib.ps_lda_loglik(self._h, ctypes.byref(out)))
        return out.value

    def get_clock(self) -> int:
        out = ctypes.c_int64()
        _check(self._h, "ps_lda_get_clock", _lib.ps_lda_get_clock(self._h, ctypes.byref(out)))
        return out.value

    def export(self, kind, block=0):
        n = ctypes.c_int64()
        _check(self._h, "ps_lda_export", _lib.ps_lda_export(self._h, kind, block, None, 0, ctypes.byref(n)))
        buf = np.empty(n.value, dtype=np.int32 if kind in (X_Z, X_NDK, X_NWK) else np.int64)
        _check(self._h, "ps_lda_export", _lib.ps_lda_export(self._h, kind, block, buf.ctypes.data if n.value else None,
                                                            n.value, ctypes.byref(n)))
        return buf

    def z(self):
        return self.export(X_Z)

    def ndk(self):
        return self.export(X_NDK).reshape(self.D, self.K)

    def nwk(self):
        """Latest version: [V+1, K], row V the topic totals."""
        return self.export(X_NWK).reshape(self.V + 1, self.K)

    def kernel_time(self):
        ms, cnt = ctypes.c_double(), ctypes.c_int64()
        _check(self._h, "ps_lda_kernel_time", _lib.ps_lda_kernel_time(self._h, ctypes.byref(ms), ctypes.byref(cnt)))
        return ms.value, cnt.value
