"""Seeded synthetic workloads shaped like the paper's matrix-factorization experiment.

Section 5 of arXiv 1410.8043 runs MF-by-SGD on the Netflix matrix (480k users x 18k
items, 100M ratings, integer 1..5).  That dataset is not available, so these generators
stand in for it: heavy-tailed (Zipf) user and item degrees, distinct (user, item) pairs
and integer ratings from planted low-rank factors plus Gaussian noise.

This module produces inputs only and holds none of the method's arithmetic; the C part
(``synth.c``) is compiled into ``libps_mf_synth.so`` next to this file.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libps_mf_synth.so")
BASE_SEED = 0x14108043

_lib = None


def build(verbose: bool = False) -> str:
    """Compile synth.c into libps_mf_synth.so (gcc, host code only)."""
    import subprocess

    src = os.path.join(_HERE, "synth.c")
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-pthread", "-std=gnu11", src, "-lm", "-o", tmp]
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
    i64, i32, u64, dbl = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_double
    vp = ctypes.c_void_p
    lib.synth_rank_weights.argtypes = [i64, dbl, u64, i32, vp]
    lib.synth_degrees.argtypes = [i64, vp, i64, i64, vp]
    lib.synth_pairs.argtypes = [i64, i64, vp, vp, u64, i32, vp, vp]
    lib.synth_uniform_cells.argtypes = [i64, i64, i64, u64, vp, vp]
    lib.synth_normal.argtypes = [i64, dbl, u64, u64, i32, vp]
    lib.synth_ratings.argtypes = [i64, i64, i64, vp, vp, i32, dbl, dbl, dbl, dbl, u64, i32, vp]
    lib.synth_splitmix64_next.argtypes = [ctypes.POINTER(u64), ctypes.POINTER(u64)]
    for f in (lib.synth_rank_weights, lib.synth_degrees, lib.synth_pairs, lib.synth_uniform_cells,
              lib.synth_normal, lib.synth_ratings, lib.synth_splitmix64_next):
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise RuntimeError(f"{what} failed with code {rc}")


def _threads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(16, n))


def splitmix64_sequence(state: int, n: int) -> list:
    """First n outputs of sequential SplitMix64 from `state` (for pinning the generator)."""
    lib = _load()
    st = ctypes.c_uint64(state)
    out = ctypes.c_uint64(0)
    res = []
    for _ in range(n):
        lib.synth_splitmix64_next(ctypes.byref(st), ctypes.byref(out))
        res.append(out.value)
    return res


def rank_weights(n: int, a: float, seed: int, which: int) -> np.ndarray:
    w = np.empty(n, dtype=np.float64)
    _check(_load().synth_rank_weights(n, a, seed, which, _ptr(w)), "synth_rank_weights")
    return w


def degrees(weights: np.ndarray, nnz: int, cap: int) -> np.ndarray:
    w = np.ascontiguousarray(weights, dtype=np.float64)
    d = np.empty(w.shape[0], dtype=np.int64)
    _check(_load().synth_degrees(w.shape[0], _ptr(w), nnz, cap, _ptr(d)), "synth_degrees")
    return d


def pairs(N: int, M: int, deg: np.ndarray, item_w: np.ndarray, seed: int):
    deg = np.ascontiguousarray(deg, dtype=np.int64)
    item_w = np.ascontiguousarray(item_w, dtype=np.float64)
    nnz = int(deg.sum())
    u = np.empty(nnz, dtype=np.int32)
    i = np.empty(nnz, dtype=np.int32)
    _check(_load().synth_pairs(N, M, _ptr(deg), _ptr(item_w), seed, _threads(), _ptr(u), _ptr(i)), "synth_pairs")
    return u, i


def uniform_cells(N: int, M: int, nnz: int, seed: int):
    u = np.empty(nnz, dtype=np.int32)
    i = np.empty(nnz, dtype=np.int32)
    _check(_load().synth_uniform_cells(N, M, nnz, seed, _ptr(u), _ptr(i)), "synth_uniform_cells")
    return u, i


def normal(shape, sd: float, seed: int, stream: int) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    _check(_load().synth_normal(out.size, sd, seed, stream, _threads(), _ptr(out)), "synth_normal")
    return out


def planted_ratings(N, M, user, item, rank, factor_sd, noise_sd, seed, lo=1.0, hi=5.0) -> np.ndarray:
    val = np.empty(user.shape[0], dtype=np.float32)
    _check(_load().synth_ratings(N, M, user.shape[0], _ptr(user), _ptr(item), rank, factor_sd, noise_sd,
                                 lo, hi, seed, _threads(), _ptr(val)), "synth_ratings")
    return val


@dataclasses.dataclass
class ConfigSpec:
    """One workload: matrix shape, degree laws, planted model and the SGD/SSP settings."""
    name: str
    index: int
    N: int
    M: int
    nnz: int
    user_zipf: Optional[float]   # None: uniform cells without replacement; 0.0: equal degrees
    item_zipf: float
    planted_rank: int
    noise_sd: float
    K: int
    P: int
    s_values: Sequence[int]
    eta: float
    lam: float
    clocks: int
    B: int
    factor_sd: float = 0.5
    init_sd: float = 0.1

    @property
    def seed(self) -> int:
        return BASE_SEED + self.index


CONFIGS = {
    "tiny": ConfigSpec("tiny", 1, 1000, 500, 20_000, None, 0.0, 8, 0.5, 16, 4, (0, 2), 0.01, 0.05, 10, 1),
    "medium": ConfigSpec("medium", 2, 100_000, 20_000, 10_000_000, 1.1, 1.1, 16, 0.5, 64, 32, (3,), 0.005, 0.05, 20, 4),
    "full": ConfigSpec("full", 3, 480_189, 17_770, 100_000_000, 1.1, 0.9, 32, 0.7, 128, 64, (0, 1, 3, 7),
                       0.002, 0.05, 30, 1),
    "large": ConfigSpec("large", 4, 2_000_000, 200_000, 500_000_000, 1.0, 1.0, 64, 0.7, 256, 128, (3,),
                        0.001, 0.05, 10, 1),
    "contention": ConfigSpec("contention", 5, 1_000_000, 10_000, 100_000_000, 0.0, 1.5, 16, 0.5, 32, 256, (15,),
                             0.002, 0.1, 20, 1),
}


@dataclasses.dataclass
class Workload:
    spec: ConfigSpec
    user: np.ndarray   # int32 [nnz]
    item: np.ndarray   # int32 [nnz]
    val: np.ndarray    # float32 [nnz]
    L0: np.ndarray     # float32 [N, K]
    R0: np.ndarray     # float32 [M, K]

    @property
    def nnz(self) -> int:
        return int(self.user.shape[0])


def scaled(spec: ConfigSpec, factor: float, **overrides) -> ConfigSpec:
    """The same degree laws at a smaller size: N, M and nnz multiplied by `factor`."""
    N = max(1, int(round(spec.N * factor)))
    M = max(1, int(round(spec.M * factor)))
    nnz = max(1, int(round(spec.nnz * factor * factor)))
    nnz = min(nnz, N * M // 2)
    s = dataclasses.replace(spec, N=N, M=M, nnz=nnz, name=f"{spec.name}@{factor:g}")
    return dataclasses.replace(s, **overrides) if overrides else s


def generate(spec, K: Optional[int] = None) -> Workload:
    """Build the workload for a ConfigSpec (or a config name)."""
    if isinstance(spec, str):
        spec = CONFIGS[spec]
    K = spec.K if K is None else K
    seed = spec.seed
    if spec.user_zipf is None:
        user, item = uniform_cells(spec.N, spec.M, spec.nnz, seed)
    else:
        uw = rank_weights(spec.N, spec.user_zipf, seed, 0)
        deg = degrees(uw, spec.nnz, spec.M)
        iw = rank_weights(spec.M, spec.item_zipf, seed, 1)
        user, item = pairs(spec.N, spec.M, deg, iw, seed)
    val = planted_ratings(spec.N, spec.M, user, item, spec.planted_rank, spec.factor_sd, spec.noise_sd, seed)
    L0 = normal((spec.N, K), spec.init_sd, seed, 1)
    R0 = normal((spec.M, K), spec.init_sd, seed, 2)
    return Workload(spec, user, item, val, L0, R0)
