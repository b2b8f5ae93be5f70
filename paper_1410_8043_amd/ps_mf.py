"""Python binding of the ps_mf C ABI (include/ps_mf.h): argument marshalling only.

Every step of the clocked SSP/ESSP matrix-factorization sweep runs in the HIP kernels of
``libps_mf.so``; this module only converts numpy arrays and torch streams into the plain
pointers the C functions take.  The functions keep the C names; ``PsMf`` wraps a handle.

torch is imported first so that the library binds to the same HIP runtime that torch
loaded (both name it libamdhip64.so.7); the library is required: importing this module
raises if it is not built.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

try:  # share torch's HIP runtime when torch is present
    import torch  # noqa: F401
except Exception:  # pragma: no cover - torch is part of the image
    torch = None

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libps_mf.so")

OK, EINVAL, ENOMEM, EDEVICE, ESTATE, EINTERNAL = 0, -1, -2, -3, -4, -5
(OPT_POLICY, OPT_STEP, OPT_MB_BLOCKS, OPT_MB_SEED, OPT_HOST_ONLY, OPT_TIMING, OPT_TILE_BYTES, OPT_UNIT_MAX, OPT_CELLS,
 OPT_HEAVY_MIN, OPT_TWO_STREAMS, OPT_HOT_STEPS, OPT_DENSE_MIN, OPT_SEQ_STRATA, OPT_ETA_DECAY,
 OPT_SEQ_GRAPHS, OPT_ITEM_TILE_BYTES, OPT_DEVICE, OPT_POISON, OPT_SWEEP_GRAPHS, OPT_UNIT_COMMIT) = range(1, 22)
SSP_LAZY, SSP_WORST, ESSP, SSP_ROW, ESSP_ROW, VAP = 0, 1, 2, 3, 4, 5
STEP_ROWMEAN, STEP_SUM, STEP_SEQ = 0, 1, 2
(IDX_OWNER, IDX_ROW_PTR, IDX_COL, IDX_PERM, IDX_USER_COUNT, IDX_ITEM_COUNT, IDX_VERSION_LOG, IDX_SPLIT, IDX_STALENESS,
 IDX_ROW_VERSIONS, IDX_SEQ_ORDER, IDX_VAP_NORMS) = range(12)
KERNEL_SWEEP, KERNEL_COMMIT = 0, 1

SYMBOLS = ("ps_mf_create", "ps_mf_set_option", "ps_mf_set_value_bound", "ps_mf_set_owner_map", "ps_mf_set_stream",
           "ps_mf_load_ratings",
           "ps_mf_set_factors", "ps_mf_clock", "ps_mf_loss", "ps_mf_loss_noalloc", "ps_mf_get_factors", "ps_mf_get_version",
           "ps_mf_get_clock", "ps_mf_export_index", "ps_mf_kernel_time", "ps_mf_last_error", "ps_mf_destroy")


def _load_lib():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(the HIP library is required; there is no fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    i64, i32, f32, dbl, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_double, ctypes.c_void_p
    sig = {
        "ps_mf_create": [i64, i64, i32, i32, i32, f32, f32, ctypes.POINTER(vp)],
        "ps_mf_set_option": [vp, i32, i64],
        "ps_mf_set_value_bound": [vp, dbl],
        "ps_mf_set_owner_map": [vp, vp],
        "ps_mf_set_stream": [vp, vp],
        "ps_mf_load_ratings": [vp, vp, vp, vp, i64],
        "ps_mf_set_factors": [vp, vp, vp],
        "ps_mf_clock": [vp, i32],
        "ps_mf_loss": [vp, ctypes.POINTER(dbl)],
        "ps_mf_loss_noalloc": [vp, ctypes.POINTER(dbl)],
        "ps_mf_get_factors": [vp, vp, vp],
        "ps_mf_get_version": [vp, i64, vp, vp],
        "ps_mf_get_clock": [vp, ctypes.POINTER(i64)],
        "ps_mf_export_index": [vp, i32, i32, vp, i64, ctypes.POINTER(i64)],
        "ps_mf_kernel_time": [vp, i32, ctypes.POINTER(dbl), ctypes.POINTER(i64)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.ps_mf_last_error.argtypes = [vp]
    lib.ps_mf_last_error.restype = ctypes.c_char_p
    lib.ps_mf_destroy.argtypes = [vp]
    lib.ps_mf_destroy.restype = None
    return lib


_lib = _load_lib()


class PsMfError(RuntimeError):
    def __init__(self, func, code, msg):
        super().__init__(f"{func} failed ({code}): {msg}")
        self.code = code


def _check(h, func, rc):
    if rc != 0:
        msg = _lib.ps_mf_last_error(h).decode() if h else ""
        raise PsMfError(func, rc, msg)


def _arr(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ---- the C functions, one Python function each (same names)
def ps_mf_create(users, items, K, P, s, eta, lam):
    h = ctypes.c_void_p()
    _check(None, "ps_mf_create", _lib.ps_mf_create(int(users), int(items), int(K), int(P), int(s), float(eta),
                                                   float(lam), ctypes.byref(h)))
    return h


def ps_mf_set_option(h, key, value):
    _check(h, "ps_mf_set_option", _lib.ps_mf_set_option(h, int(key), int(value)))


def ps_mf_set_value_bound(h, v0):
    _check(h, "ps_mf_set_value_bound", _lib.ps_mf_set_value_bound(h, float(v0)))


def ps_mf_set_owner_map(h, owner):
    owner = _arr(owner, np.int32)
    _check(h, "ps_mf_set_owner_map", _lib.ps_mf_set_owner_map(h, owner.ctypes.data))


def ps_mf_set_stream(h, stream):
    """stream: a torch.cuda.Stream, an integer hipStream_t, or None for the handle's own."""
    if stream is not None and hasattr(stream, "cuda_stream"):
        stream = stream.cuda_stream
    _check(h, "ps_mf_set_stream", _lib.ps_mf_set_stream(h, ctypes.c_void_p(stream) if stream else None))


def ps_mf_load_ratings(h, user, item, value):
    user, item, value = _arr(user, np.int32), _arr(item, np.int32), _arr(value, np.float32)
    n = user.shape[0]
    if item.shape[0] != n or value.shape[0] != n:
        raise ValueError("user, item and value must have the same length")
    _check(h, "ps_mf_load_ratings", _lib.ps_mf_load_ratings(h, user.ctypes.data, item.ctypes.data,
                                                            value.ctypes.data, n))


def ps_mf_set_factors(h, L, R):
    L, R = _arr(L, np.float32), _arr(R, np.float32)
    _check(h, "ps_mf_set_factors", _lib.ps_mf_set_factors(h, L.ctypes.data, R.ctypes.data))


def ps_mf_clock(h, n=1):
    _check(h, "ps_mf_clock", _lib.ps_mf_clock(h, int(n)))


def ps_mf_loss(h):
    out = ctypes.c_double()
    _check(h, "ps_mf_loss", _lib.ps_mf_loss(h, ctypes.byref(out)))
    return out.value


def ps_mf_loss_noalloc(h):
    out = ctypes.c_double()
    _check(h, "ps_mf_loss_noalloc", _lib.ps_mf_loss_noalloc(h, ctypes.byref(out)))
    return out.value


def ps_mf_get_factors(h, users, items, K):
    L = np.empty((users, K), np.float32)
    R = np.empty((items, K), np.float32)
    _check(h, "ps_mf_get_factors", _lib.ps_mf_get_factors(h, L.ctypes.data, R.ctypes.data))
    return L, R


def ps_mf_get_version(h, v, users, items, K):
    L = np.empty((users, K), np.float32)
    R = np.empty((items, K), np.float32)
    _check(h, "ps_mf_get_version", _lib.ps_mf_get_version(h, int(v), L.ctypes.data, R.ctypes.data))
    return L, R


def ps_mf_get_clock(h):
    c = ctypes.c_int64()
    _check(h, "ps_mf_get_clock", _lib.ps_mf_get_clock(h, ctypes.byref(c)))
    return c.value


def ps_mf_export_index(h, kind, block=0):
    n = ctypes.c_int64()
    _check(h, "ps_mf_export_index", _lib.ps_mf_export_index(h, int(kind), int(block), None, 0, ctypes.byref(n)))
    dt = (np.int32 if kind in (IDX_OWNER, IDX_COL, IDX_USER_COUNT, IDX_ITEM_COUNT) else
          np.float64 if kind == IDX_VAP_NORMS else np.int64)
    buf = np.empty(n.value, dtype=dt)
    _check(h, "ps_mf_export_index", _lib.ps_mf_export_index(h, int(kind), int(block),
                                                            buf.ctypes.data if n.value else None, n.value,
                                                            ctypes.byref(n)))
    return buf


def ps_mf_kernel_time(h, kernel):
    ms = ctypes.c_double()
    cnt = ctypes.c_int64()
    _check(h, "ps_mf_kernel_time", _lib.ps_mf_kernel_time(h, int(kernel), ctypes.byref(ms), ctypes.byref(cnt)))
    return ms.value, cnt.value


def ps_mf_last_error(h):
    return _lib.ps_mf_last_error(h).decode()


def ps_mf_destroy(h):
    _lib.ps_mf_destroy(h)


class PsMf:
    """A ps_mf handle: create -> options -> load_ratings -> set_factors -> clock/loss/get."""

    def __init__(self, users, items, K, P, s, eta, lam, *, policy=SSP_LAZY, step=STEP_ROWMEAN, B=1, mb_seed=0,
                 owner=None, host_only=False, timing=False, stream=None, tile_bytes=None, unit_max=None,
                 cells=None, heavy_min=None, two_streams=None, hot_steps=None, dense_min=None, strata=None,
                 value_bound=None, eta_decay=False, seq_graphs=None, item_tile_bytes=None, device=None,
                 poison=False, sweep_graphs=None, unit_commit=None):
        self.N, self.M, self.K, self.P, self.s = int(users), int(items), int(K), int(P), int(s)
        self.h = ps_mf_create(users, items, K, P, s, eta, lam)
        try:
            ps_mf_set_option(self.h, OPT_POLICY, policy)
            ps_mf_set_option(self.h, OPT_STEP, step)
            ps_mf_set_option(self.h, OPT_MB_BLOCKS, B)
            ps_mf_set_option(self.h, OPT_MB_SEED, mb_seed if mb_seed < 2**63 else mb_seed - 2**64)
            if host_only:
                ps_mf_set_option(self.h, OPT_HOST_ONLY, 1)
            if timing:
                ps_mf_set_option(self.h, OPT_TIMING, 1)
            if tile_bytes is not None:
                ps_mf_set_option(self.h, OPT_TILE_BYTES, tile_bytes)
            if unit_max is not None:
                ps_mf_set_option(self.h, OPT_UNIT_MAX, unit_max)
            if cells is not None:
                ps_mf_set_option(self.h, OPT_CELLS, int(bool(cells)))
            if heavy_min is not None:
                ps_mf_set_option(self.h, OPT_HEAVY_MIN, heavy_min)
            if two_streams is not None:
                ps_mf_set_option(self.h, OPT_TWO_STREAMS, int(bool(two_streams)))
            if hot_steps is not None:
                ps_mf_set_option(self.h, OPT_HOT_STEPS, hot_steps)
            if dense_min is not None:
                ps_mf_set_option(self.h, OPT_DENSE_MIN, dense_min)
            if strata is not None:
                ps_mf_set_option(self.h, OPT_SEQ_STRATA, strata)
            if value_bound is not None:
                ps_mf_set_value_bound(self.h, value_bound)
            if eta_decay:
                ps_mf_set_option(self.h, OPT_ETA_DECAY, 1)
            if seq_graphs is not None:
                ps_mf_set_option(self.h, OPT_SEQ_GRAPHS, int(bool(seq_graphs)))
            if item_tile_bytes is not None:
                ps_mf_set_option(self.h, OPT_ITEM_TILE_BYTES, item_tile_bytes)
            if device is not None:
                ps_mf_set_option(self.h, OPT_DEVICE, device)
            if poison:
                ps_mf_set_option(self.h, OPT_POISON, 1)
            if sweep_graphs is not None:
                ps_mf_set_option(self.h, OPT_SWEEP_GRAPHS, int(bool(sweep_graphs)))
            if unit_commit is not None:
                ps_mf_set_option(self.h, OPT_UNIT_COMMIT, int(bool(unit_commit)))
            if owner is not None:
                ps_mf_set_owner_map(self.h, owner)
            if stream is not None:
                ps_mf_set_stream(self.h, stream)
        except Exception:
            self.close()
            raise

    def close(self):
        if getattr(self, "h", None):
            ps_mf_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def load_ratings(self, user, item, value):
        ps_mf_load_ratings(self.h, user, item, value)

    def set_factors(self, L, R):
        ps_mf_set_factors(self.h, L, R)

    def clock(self, n=1):
        ps_mf_clock(self.h, n)

    def loss(self):
        return ps_mf_loss(self.h)

    def get_factors(self):
        return ps_mf_get_factors(self.h, self.N, self.M, self.K)

    def get_version(self, v):
        return ps_mf_get_version(self.h, v, self.N, self.M, self.K)

    @property
    def clock_value(self):
        return ps_mf_get_clock(self.h)

    def export_index(self, kind, block=0):
        return ps_mf_export_index(self.h, kind, block)

    def kernel_time(self, kernel):
        return ps_mf_kernel_time(self.h, kernel)
