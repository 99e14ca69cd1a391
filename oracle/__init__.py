"""Mutual Pair Merging CPU oracle: float64 brute force.

TEST INFRASTRUCTURE ONLY. Callers are the tests, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``. The product path never imports this
package; it shares no code with the HIP library.

Python wrapper over ``libmpm_oracle.so`` (plain C in ``mpm_oracle.c``).
Arrays are numpy; storage values are converted exactly to float64 before the C
code sees them. Every function works on one image; ``merge`` and ``schedule``
chain the steps the way the paper does:

* ``nearest``  -- Eq. 1 and the nearest-neighbour rule of Sec. 3.2.
* ``pairs``    -- mutual pairs, RepMask and the left-to-right compact ids (Alg. 1).
* ``average``  -- cluster means (Eq. 2), rounded once to the storage dtype.
* ``compose``  -- r*(i) = r2(r1(i)) (Eq. 3).
* ``unmerge``  -- gather reconstruction Z_up[i] = Z[r*(i)] (Eq. 4).
* the locality constraint of Sec. 5 (also Sec. 4.3): ``nearest``, ``merge`` and
  ``schedule`` take token positions on the grid and a window radius; candidates
  are restricted to the window, and a merged token takes its representative's
  position.

Parity status of each function is recorded in the tests: every function here is
pinned by hand-derived cases and properties (see ``tests/test_oracle_*.py``).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

from .build import library_path, build_oracle

_F64P = ctypes.POINTER(ctypes.c_double)
_I32P = ctypes.POINTER(ctypes.c_int32)

DTYPES = {"f32": 0, "bf16": 1}

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        build_oracle()
    lib = ctypes.CDLL(path)
    lib.mpm_oracle_nearest.argtypes = [_F64P, ctypes.c_int, ctypes.c_int, ctypes.c_int, _I32P, _F64P, _F64P]
    lib.mpm_oracle_nearest.restype = ctypes.c_int
    lib.mpm_oracle_nearest_window.argtypes = [_F64P, ctypes.c_int, ctypes.c_int, _I32P, ctypes.c_int, ctypes.c_int,
                                              ctypes.c_int, _I32P, _F64P, _F64P]
    lib.mpm_oracle_nearest_window.restype = ctypes.c_int
    lib.mpm_oracle_nearest_from_affinity.argtypes = [_F64P, ctypes.c_int, _I32P]
    lib.mpm_oracle_nearest_from_affinity.restype = ctypes.c_int
    lib.mpm_oracle_pairs.argtypes = [_I32P, ctypes.c_int, _I32P, _I32P, _I32P]
    lib.mpm_oracle_pairs.restype = ctypes.c_int
    lib.mpm_oracle_average.argtypes = [_F64P, ctypes.c_int, _I32P, _I32P, ctypes.c_int, ctypes.c_int, _F64P]
    lib.mpm_oracle_average.restype = None
    lib.mpm_oracle_compose.argtypes = [_I32P, ctypes.c_int, _I32P, _I32P]
    lib.mpm_oracle_compose.restype = None
    lib.mpm_oracle_unmerge.argtypes = [_F64P, ctypes.c_int, _I32P, ctypes.c_int, _F64P]
    lib.mpm_oracle_unmerge.restype = None
    lib.mpm_oracle_cosine.argtypes = [_F64P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]
    lib.mpm_oracle_cosine.restype = ctypes.c_double
    lib.mpm_oracle_round.argtypes = [_F64P, ctypes.c_int64, ctypes.c_int, _F64P]
    lib.mpm_oracle_round.restype = None
    _lib = lib
    return lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _p(a: np.ndarray, t):
    return a.ctypes.data_as(t)


def as_f64(x) -> np.ndarray:
    """Exact float64 copy of a storage tensor/array (torch float32/bfloat16 or numpy)."""
    try:
        import torch

        if isinstance(x, torch.Tensor):
            return x.detach().to("cpu", torch.float64).numpy()
    except ImportError:  # pragma: no cover
        pass
    return _f64(x)


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return max(1, os.cpu_count() or 1)


@dataclass
class Nearest:
    nb: np.ndarray      # int32 [n]; b(i), -1 when n == 1
    top1: np.ndarray    # float64 [n]; max_{j != i} S_ij
    top2: np.ndarray    # float64 [n]; second largest S_ij over j != i

    @property
    def gap(self) -> np.ndarray:
        return self.top1 - self.top2


def nearest(x, threads: int | None = None, pos=None, grid_w: int | None = None, window: int | None = None) -> Nearest:
    """b(i) = argmax_{j != i} cos(x_i, x_j), lowest j on equal values (Eq. 1, Sec. 3.2).
    With ``window`` (the locality constraint of Sec. 5): only tokens j whose grid
    positions (``pos``: raster indices on a grid of ``grid_w`` columns; default the
    raster order 0..n-1) lie within ``window`` rows and columns of token i's are
    candidates; b(i) = -1 (top1 = top2 = -inf) when there is none."""
    lib = _load()
    x = _f64(x)
    n, D = x.shape
    if not np.isfinite(x).all():
        raise ValueError("oracle: input holds NaN or Inf")
    nb = np.empty(n, np.int32)
    t1 = np.empty(n, np.float64)
    t2 = np.empty(n, np.float64)
    if window is not None:
        p = _i32(np.arange(n) if pos is None else pos)
        rc = lib.mpm_oracle_nearest_window(_p(x, _F64P), n, D, _p(p, _I32P), int(grid_w), int(window),
                                           threads or default_threads(), _p(nb, _I32P), _p(t1, _F64P),
                                           _p(t2, _F64P))
        if rc != 0:
            raise RuntimeError("mpm_oracle_nearest_window failed")
        return Nearest(nb, t1, t2)
    rc = lib.mpm_oracle_nearest(_p(x, _F64P), n, D, threads or default_threads(),
                                _p(nb, _I32P), _p(t1, _F64P), _p(t2, _F64P))
    if rc != 0:
        raise RuntimeError("mpm_oracle_nearest failed")
    return Nearest(nb, t1, t2)


def nearest_from_affinity(S) -> np.ndarray:
    """Same argmax rule on a given affinity matrix (diagonal ignored)."""
    lib = _load()
    S = _f64(S)
    n = S.shape[0]
    nb = np.empty(n, np.int32)
    if lib.mpm_oracle_nearest_from_affinity(_p(S, _F64P), n, _p(nb, _I32P)) != 0:
        raise RuntimeError("mpm_oracle_nearest_from_affinity failed")
    return nb


def cosine(x, i: int, j: int) -> float:
    """S_ij exactly as ``nearest`` evaluates it."""
    x = _f64(x)
    n, D = x.shape
    return float(_load().mpm_oracle_cosine(_p(x, _F64P), n, D, int(i), int(j)))


@dataclass
class Pairs:
    map: np.ndarray     # int32 [n]; r(i)
    src_a: np.ndarray   # int32 [n']; representative of cluster k
    src_b: np.ndarray   # int32 [n']; partner of cluster k (== src_a for singletons)

    @property
    def count(self) -> int:
        return int(self.src_a.shape[0])


def pairs(nb) -> Pairs:
    """Mutual pairs, RepMask and compact ids (Sec. 3.2, Alg. 1)."""
    lib = _load()
    nb = _i32(nb)
    n = nb.shape[0]
    m = np.empty(n, np.int32)
    a = np.empty(n, np.int32)
    b = np.empty(n, np.int32)
    cnt = lib.mpm_oracle_pairs(_p(nb, _I32P), n, _p(m, _I32P), _p(a, _I32P), _p(b, _I32P))
    if cnt < 0:
        raise RuntimeError("mpm_oracle_pairs failed")
    return Pairs(m, a[:cnt].copy(), b[:cnt].copy())


def average(x, src_a, src_b, dtype: str) -> np.ndarray:
    """Cluster means (Eq. 2) rounded once to ``dtype`` ('f32' or 'bf16')."""
    lib = _load()
    x = _f64(x)
    a = _i32(src_a)
    b = _i32(src_b)
    m = a.shape[0]
    D = x.shape[1]
    y = np.empty((m, D), np.float64)
    lib.mpm_oracle_average(_p(x, _F64P), D, _p(a, _I32P), _p(b, _I32P), m, DTYPES[dtype], _p(y, _F64P))
    return y


def round_to(v, dtype: str) -> np.ndarray:
    """Round float64 values to the storage dtype (nearest even), as float64."""
    v = _f64(v)
    out = np.empty_like(v)
    _load().mpm_oracle_round(_p(v, _F64P), v.size, DTYPES[dtype], _p(out, _F64P))
    return out


def compose(r1, r2) -> np.ndarray:
    """r*(i) = r2(r1(i)) (Eq. 3)."""
    r1 = _i32(r1)
    r2 = _i32(r2)
    out = np.empty_like(r1)
    _load().mpm_oracle_compose(_p(r1, _I32P), r1.shape[0], _p(r2, _I32P), _p(out, _I32P))
    return out


def unmerge(z, rstar) -> np.ndarray:
    """Z_up[i] = Z[r*(i)] (Eq. 4); a plain row copy."""
    z = _f64(z)
    r = _i32(rstar)
    n = r.shape[0]
    out = np.empty((n, z.shape[1]), np.float64)
    _load().mpm_oracle_unmerge(_p(z, _F64P), z.shape[1], _p(r, _I32P), n, _p(out, _F64P))
    return out


@dataclass
class MergeResult:
    nearest: Nearest
    pairs: Pairs
    y: np.ndarray       # float64 [n', D], values exactly representable in the storage dtype
    y_pos: np.ndarray | None = None  # int32 [n']: grid position of each cluster (its representative's)

    @property
    def map(self) -> np.ndarray:
        return self.pairs.map

    @property
    def count(self) -> int:
        return self.pairs.count


def merge(x, dtype: str, threads: int | None = None, nb=None, pos=None, grid_w: int | None = None,
          window: int | None = None) -> MergeResult:
    """One MPM call on one image (Alg. 1). ``nb`` replaces the nearest-neighbour
    step (used to re-seed the later steps with another implementation's choice).
    With ``window``: the locality-constrained neighbour of ``nearest``; the merged
    tokens' positions are their representatives' (``y_pos``)."""
    x = _f64(x)
    if nb is not None:
        nn = Nearest(_i32(nb), np.full(len(nb), np.nan), np.full(len(nb), np.nan))
    else:
        nn = nearest(x, threads, pos=pos, grid_w=grid_w, window=window)
    pr = pairs(nn.nb)
    y = average(x, pr.src_a, pr.src_b, dtype)
    y_pos = None
    if window is not None:
        p = np.arange(x.shape[0], dtype=np.int32) if pos is None else _i32(pos)
        y_pos = p[pr.src_a].copy()
    return MergeResult(nn, pr, y, y_pos)


def schedule(x, dtype: str, insertions: int = 2, threads: int | None = None, grid_w: int | None = None,
             window: int | None = None):
    """Insertions with identity blocks in between, then composition and
    reconstruction (Sec. 3.3, Eq. 3, Eq. 4). With ``window``, every insertion is
    locality-constrained (Sec. 5) on a grid of ``grid_w`` columns, the first on the
    raster positions. Returns (stages, rstar, x_up)."""
    cur = _f64(x)
    stages = []
    rstar = None
    pos = None
    for _ in range(insertions):
        res = merge(cur, dtype, threads, pos=pos, grid_w=grid_w, window=window)
        stages.append(res)
        rstar = res.map.copy() if rstar is None else compose(rstar, res.map)
        cur, pos = res.y, res.y_pos
    return stages, rstar, unmerge(cur, rstar)
