"""ORACLE (test infrastructure only): ctypes wrapper of libps_mf_oracle.so.

A plain single-threaded CPU implementation of the clocked SSP/ESSP matrix-factorization
SGD of arXiv 1410.8043 (Section 3.1 update rule, Section 3.2 SSP condition, Section 4
coalesced updates).  Versions are stored in fp32, all arithmetic is fp64.  Only the tests,
the package smoke check and the benchmark's CPU-baseline leg use this module; the
product path (``paper_1410_8043_amd``) never imports it, and it imports nothing from
the product.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libps_mf_oracle.so")

SSP_LAZY, SSP_WORST, ESSP, SSP_ROW, ESSP_ROW, VAP = 0, 1, 2, 3, 4, 5
ROWMEAN, SUM, SEQ = 0, 1, 2
(X_OWNER, X_ROW_PTR, X_COL, X_PERM, X_USER_COUNT, X_ITEM_COUNT, X_VERSION_LOG, X_STALENESS, X_ROW_VERSIONS,
 X_SEQ_ORDER, X_VAP_NORMS) = range(11)

_lib = None


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc (no fast-math: fp64 evaluation order is kept)."""
    srcs = [os.path.join(_HERE, f) for f in ("ps_mf_oracle.c", "ps_lda_oracle.c")]
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-std=gnu11", *srcs, "-lm", "-o", tmp]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    i64, i32, u64, dbl, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p
    sig = {
        "oracle_create": [i64, i64, i32, i32, i32, dbl, dbl, i32, i32, i32, u64, vp, ctypes.POINTER(vp)],
        "oracle_load": [vp, vp, vp, vp, i64],
        "oracle_set_factors": [vp, vp, vp],
        "oracle_clock": [vp, i32],
        "oracle_get_clock": [vp, ctypes.POINTER(i64)],
        "oracle_get_version": [vp, i64, vp, vp],
        "oracle_loss": [vp, ctypes.POINTER(dbl)],
        "oracle_rows_from_v0": [vp, i32, i64, vp, i64, vp, vp, vp],
        "oracle_export": [vp, i32, i32, vp, i64, ctypes.POINTER(i64)],
        "oracle_view_version": [vp, i64, i64, ctypes.POINTER(i64)],
        "oracle_splitmix64": [u64, ctypes.POINTER(u64)],
        "oracle_set_strata": [vp, i32],
        "oracle_set_value_bound": [vp, dbl],
        "oracle_set_eta_decay": [vp, i32],
        "lda_create": [i64, i64, i32, i32, i32, dbl, dbl, i32, i32, u64, ctypes.POINTER(vp)],
        "lda_load": [vp, vp, vp, vp, i64],
        "lda_clock": [vp, i32],
        "lda_loglik": [vp, ctypes.POINTER(dbl)],
        "lda_export": [vp, i32, i32, vp, i64, ctypes.POINTER(i64)],
        "lda_token_draw": [vp, vp, vp, vp, i32, u64, vp, ctypes.POINTER(u64), ctypes.POINTER(i32)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.oracle_destroy.argtypes = [vp]
    lib.oracle_destroy.restype = None
    lib.lda_destroy.argtypes = [vp]
    lib.lda_destroy.restype = None
    _lib = lib
    return lib


class OracleError(RuntimeError):
    def __init__(self, what, code):
        super().__init__(f"{what} returned {code}")
        self.code = code


def _chk(rc, what):
    if rc != 0:
        raise OracleError(what, rc)


def splitmix64(state: int) -> int:
    out = ctypes.c_uint64(0)
    _chk(_load().oracle_splitmix64(state, ctypes.byref(out)), "oracle_splitmix64")
    return out.value


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


class Oracle:
    """Clocked SSP/ESSP MF-SGD on the CPU; mirrors the library's call sequence."""

    def __init__(self, N, M, K, P, s, eta, lam, policy=SSP_LAZY, step=ROWMEAN, B=1, seed=0, owner=None, strata=None,
                 value_bound=None, eta_decay=False):
        self._lib = _load()
        self.N, self.M, self.K, self.P, self.s = int(N), int(M), int(K), int(P), int(s)
        self._owner = None if owner is None else _c(owner, np.int32)
        h = ctypes.c_void_p()
        _chk(self._lib.oracle_create(self.N, self.M, self.K, self.P, self.s, float(eta), float(lam), int(policy),
                                     int(step), int(B), int(seed) & (2**64 - 1),
                                     None if self._owner is None else self._owner.ctypes.data, ctypes.byref(h)),
             "oracle_create")
        self._h = h
        if strata is not None:
            _chk(self._lib.oracle_set_strata(self._h, int(strata)), "oracle_set_strata")
        if value_bound is not None:
            _chk(self._lib.oracle_set_value_bound(self._h, float(value_bound)), "oracle_set_value_bound")
        if eta_decay:
            _chk(self._lib.oracle_set_eta_decay(self._h, 1), "oracle_set_eta_decay")

    def close(self):
        if self._h:
            self._lib.oracle_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def load(self, user, item, val):
        self._u, self._i, self._v = _c(user, np.int32), _c(item, np.int32), _c(val, np.float32)
        n = self._u.shape[0]
        if not (self._i.shape[0] == n and self._v.shape[0] == n):
            raise ValueError("COO arrays differ in length")
        _chk(self._lib.oracle_load(self._h, self._u.ctypes.data, self._i.ctypes.data, self._v.ctypes.data, n),
             "oracle_load")

    def set_factors(self, L0, R0):
        L0 = _c(L0, np.float32).reshape(self.N, self.K)
        R0 = _c(R0, np.float32).reshape(self.M, self.K)
        _chk(self._lib.oracle_set_factors(self._h, L0.ctypes.data, R0.ctypes.data), "oracle_set_factors")

    def clock(self, n=1):
        _chk(self._lib.oracle_clock(self._h, int(n)), "oracle_clock")

    @property
    def clock_value(self) -> int:
        c = ctypes.c_int64()
        _chk(self._lib.oracle_get_clock(self._h, ctypes.byref(c)), "oracle_get_clock")
        return c.value

    def get_version(self, v):
        L = np.empty((self.N, self.K), np.float32)
        R = np.empty((self.M, self.K), np.float32)
        _chk(self._lib.oracle_get_version(self._h, int(v), L.ctypes.data, R.ctypes.data), "oracle_get_version")
        return L, R

    def get_factors(self):
        return self.get_version(self.clock_value)

    def loss(self) -> float:
        out = ctypes.c_double()
        _chk(self._lib.oracle_loss(self._h, ctypes.byref(out)), "oracle_loss")
        return out.value

    def rows_from_v0(self, nclocks, users, items):
        users = _c(users, np.int64)
        items = _c(items, np.int64)
        L = np.empty((users.shape[0], self.K), np.float32)
        R = np.empty((items.shape[0], self.K), np.float32)
        _chk(self._lib.oracle_rows_from_v0(self._h, int(nclocks), users.shape[0], users.ctypes.data, items.shape[0],
                                           items.ctypes.data, L.ctypes.data, R.ctypes.data), "oracle_rows_from_v0")
        return L, R

    def view_version(self, p, c) -> int:
        v = ctypes.c_int64()
        _chk(self._lib.oracle_view_version(self._h, int(p), int(c), ctypes.byref(v)), "oracle_view_version")
        return v.value

    def export(self, kind, block=0):
        n = ctypes.c_int64()
        _chk(self._lib.oracle_export(self._h, kind, block, None, 0, ctypes.byref(n)), "oracle_export")
        dt = (np.int32 if kind in (X_OWNER, X_COL, X_USER_COUNT, X_ITEM_COUNT) else
              np.float64 if kind == X_VAP_NORMS else np.int64)
        buf = np.empty(n.value, dtype=dt)
        _chk(self._lib.oracle_export(self._h, kind, block, buf.ctypes.data if n.value else None, n.value,
                                     ctypes.byref(n)), "oracle_export")
        return buf


def run(user, item, val, L0, R0, *, N, M, K, P, s, eta, lam, clocks, policy=SSP_LAZY, step=ROWMEAN, B=1, seed=0,
        owner=None):
    """Convenience: load, set factors, run `clocks` clocks; returns (L, R, loss, oracle)."""
    o = Oracle(N, M, K, P, s, eta, lam, policy, step, B, seed, owner)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(clocks)
    L, R = o.get_factors()
    return L, R, o.loss(), o


# ---- LDA by collapsed Gibbs sampling under SSP / ESSP (Section 5's topic-model workload) ----
LDA_Z, LDA_NDK, LDA_NWK, LDA_VERSION_LOG, LDA_BLOCK_ORDER = range(5)


class LdaOracle:
    """Clocked SSP/ESSP collapsed Gibbs sampling for LDA on the CPU.

    The shared word-topic counts (and topic totals, row V) are versioned per clock; the
    doc-topic counts and the assignments stay with the worker that owns the document
    (d mod P).  Policies: SSP_LAZY, SSP_WORST, ESSP.
    """

    def __init__(self, D, V, K, P, s, alpha, beta, policy=ESSP, B=2, seed=0):
        self._lib = _load()
        self.D, self.V, self.K, self.P, self.s, self.B = int(D), int(V), int(K), int(P), int(s), int(B)
        h = ctypes.c_void_p()
        _chk(self._lib.lda_create(self.D, self.V, self.K, self.P, self.s, float(alpha), float(beta), int(policy),
                                  self.B, int(seed) & (2**64 - 1), ctypes.byref(h)), "lda_create")
        self._h = h

    def close(self):
        if self._h:
            self._lib.lda_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def load(self, doc, word, z0):
        self._keep = (_c(doc, np.int32), _c(word, np.int32), _c(z0, np.int32))
        n = self._keep[0].shape[0]
        _chk(self._lib.lda_load(self._h, *(a.ctypes.data if n else None for a in self._keep), n), "lda_load")
        self._keep = None

    def clock(self, n=1):
        _chk(self._lib.lda_clock(self._h, int(n)), "lda_clock")

    def loglik(self) -> float:
        out = ctypes.c_double()
        _chk(self._lib.lda_loglik(self._h, ctypes.byref(out)), "lda_loglik")
        return out.value

    def export(self, kind, block=0):
        n = ctypes.c_int64()
        _chk(self._lib.lda_export(self._h, kind, block, None, 0, ctypes.byref(n)), "lda_export")
        dt = np.int32 if kind in (LDA_Z, LDA_NDK, LDA_NWK) else np.int64
        buf = np.empty(n.value, dtype=dt)
        _chk(self._lib.lda_export(self._h, kind, block, buf.ctypes.data if n.value else None, n.value,
                                  ctypes.byref(n)), "lda_export")
        return buf

    def token_draw(self, nd, nw, nk, k0, r):
        """One token's draw from its counts n_dk, n_wk, n_k (each including the token, which
        is in topic k0) and the random number r: (weights [K] as Python ints, their sum, topic)."""
        nd, nw, nk = _c(nd, np.int32), _c(nw, np.int32), _c(nk, np.int32)
        assert nd.shape == nw.shape == nk.shape == (self.K,)
        w = np.zeros(self.K, np.uint64)
        total, k = ctypes.c_uint64(), ctypes.c_int32()
        _chk(self._lib.lda_token_draw(self._h, nd.ctypes.data, nw.ctypes.data, nk.ctypes.data, int(k0),
                                      int(r) & (2**64 - 1), w.ctypes.data, ctypes.byref(total), ctypes.byref(k)),
             "lda_token_draw")
        return [int(x) for x in w], total.value, k.value

    def z(self):
        return self.export(LDA_Z)

    def ndk(self):
        return self.export(LDA_NDK).reshape(self.D, self.K)

    def nwk(self):
        """Latest version: [V+1, K], row V the topic totals."""
        return self.export(LDA_NWK).reshape(self.V + 1, self.K)
