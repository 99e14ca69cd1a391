"""Torch-facing binding of the MPM C ABI.

Argument marshalling only: every step runs in the HIP kernels of libmpm.so,
on ``torch.cuda.current_stream()``. PyTorch provides device memory and the
stream. Outputs are allocated at capacity with ``torch.empty``.

Token layouts (see include/mpm.h):
  dense  -- x is [B, N, D] (or [B*N, D] with N given), x_off None;
  packed -- x is [R, D] and x_off an int32 device tensor [B+1]; N is the
            per-image capacity (max tokens of an image).
"""
from __future__ import annotations

import ctypes
import math
from dataclasses import dataclass

import torch

from . import _lib

_DTYPES = {torch.float32: _lib.MPM_F32, torch.bfloat16: _lib.MPM_BF16}


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def c_event(ev):
    """The hipEvent_t handle of a torch.cuda.Event that has been recorded once."""
    return ctypes.c_void_p(ev.cuda_event)


def _dt(x: torch.Tensor) -> int:
    try:
        return _DTYPES[x.dtype]
    except KeyError:
        raise TypeError(f"unsupported token dtype {x.dtype}; use float32 or bfloat16") from None


def _rows(x: torch.Tensor, N: int | None, x_off: torch.Tensor | None):
    """Returns (rows2d, B, N, D) for dense or packed tokens."""
    if not x.is_cuda:
        raise ValueError("tokens must be on the GPU")
    if not x.is_contiguous():
        raise ValueError("tokens must be contiguous")
    if x_off is None:
        if x.dim() == 3:
            B, n, D = x.shape
            if N is not None and N != n:
                raise ValueError("N does not match x.shape[1]")
            return x.view(B * n, D), B, n, D
        raise ValueError("dense tokens must be [B, N, D]")
    if x.dim() != 2 or N is None:
        raise ValueError("packed tokens are [R, D] with N given")
    if x_off.dtype != torch.int32 or not x_off.is_cuda:
        raise ValueError("x_off must be an int32 device tensor [B+1]")
    return x, x_off.numel() - 1, int(N), x.shape[1]


def _sched(schedule: str) -> int:
    try:
        return SCHEDULES[schedule]
    except KeyError:
        raise ValueError(f"unknown schedule {schedule!r}; expected one of {sorted(SCHEDULES)}") from None


def new_workspace(B: int, N: int, device) -> torch.Tensor:
    """A workspace for B images of at most N tokens, its sync region zeroed (mpm_workspace_init)."""
    ws = torch.empty((workspace_bytes(B, N),), dtype=torch.uint8, device=device)
    _lib.check("mpm_workspace_init", _lib.load().mpm_workspace_init(_p(ws), ws.numel(), _stream()))
    return ws


def _workspace(B, N, device, ws=None):
    if ws is None or ws.numel() < workspace_bytes(B, N):
        ws = new_workspace(B, N, device)
    return ws


def argmax(x, x_off=None, N=None, with_best=False, ws=None, schedule="auto"):
    """nb [B, N] int32 (and best [B, N] float32 cosines when ``with_best``)."""
    x2, B, N, D = _rows(x, N, x_off)
    nb = torch.empty((B, N), dtype=torch.int32, device=x.device)
    best = torch.empty((B, N), dtype=torch.float32, device=x.device) if with_best else None
    ws = _workspace(B, N, x.device, ws)
    lib = _lib.load()
    _lib.check("mpm_argmax", lib.mpm_argmax(_p(x2), _p(x_off), B, N, D, _dt(x), _sched(schedule), _p(nb), _p(best),
                                            _p(ws), ws.numel(), _stream()))
    return (nb, best) if with_best else nb


def affinity(x, x_off=None, N=None, x_inv=None, schedule="auto", ws=None, events=None):
    """Runs mpm_affinity (the per-candidate-tile partials in the workspace); returns the
    workspace. ``events``: optional (start, stop) timing events bound to its dispatches."""
    x2, B, N, D = _rows(x, N, x_off)
    ws = _workspace(B, N, x.device, ws)
    ev0, ev1 = (None, None) if events is None else (c_event(e) for e in events)
    _lib.check("mpm_affinity", _lib.load().mpm_affinity(_p(x2), _p(x_off), _p(x_inv), B, N, D, _dt(x),
                                                        _sched(schedule), _p(ws), ws.numel(), ev0, ev1, _stream()))
    return ws


def pair_compact(nb, x_off=None):
    """(map [B, N], src [B, N, 2], y_off [B+1]) from nb [B, N]."""
    B, N = nb.shape
    dev = nb.device
    m = torch.empty((B, N), dtype=torch.int32, device=dev)
    src = torch.empty((B, N, 2), dtype=torch.int32, device=dev)
    y_off = torch.empty((B + 1,), dtype=torch.int32, device=dev)
    lib = _lib.load()
    _lib.check("mpm_pair_compact", lib.mpm_pair_compact(_p(nb.contiguous()), _p(x_off), B, N, _p(m), _p(src),
                                                        _p(y_off), _stream()))
    return m, src, y_off


def pair_average(x, src, y_off, x_off=None, N=None, with_inv=False):
    """y [B*N, D] packed at capacity: cluster means at the offsets y_off; with
    ``with_inv`` also y_inv [B*N] float32, the inverse norms of the merged rows."""
    x2, B, N, D = _rows(x, N, x_off)
    y = torch.empty((B * N, D), dtype=x.dtype, device=x.device)
    y_inv = torch.empty((B * N,), dtype=torch.float32, device=x.device) if with_inv else None
    lib = _lib.load()
    _lib.check("mpm_pair_average", lib.mpm_pair_average(_p(x2), _p(x_off), _p(src), _p(y_off), B, N, D, _dt(x),
                                                        _p(y), _p(y_inv), _stream()))
    return (y, y_inv) if with_inv else y


def workspace_bytes(B: int, N: int) -> int:
    return int(_lib.load().mpm_workspace_bytes(B, N))


SCHEDULES = {"auto": _lib.MPM_SCHEDULE_AUTO, "full": _lib.MPM_SCHEDULE_FULL, "symmetric": _lib.MPM_SCHEDULE_SYMMETRIC,
             "full_64": _lib.MPM_SCHEDULE_FULL_64}


def affinity_schedule_used(B: int, N: int, D: int, dtype: torch.dtype, schedule: str = "auto") -> str:
    """The schedule ("full", "symmetric" or "full_64") the affinity kernel runs for
    this shape and requested schedule on the current device."""
    out = ctypes.c_int32()
    _lib.check("mpm_affinity_schedule_used",
               _lib.load().mpm_affinity_schedule_used(B, N, D, _DTYPES[dtype], _sched(schedule), ctypes.byref(out)))
    return {v: k for k, v in SCHEDULES.items()}[out.value]


def local_block_rows(B: int, N: int, D: int, dtype: torch.dtype, grid_w: int, window: int,
                     block_rows: int = 0) -> int:
    """Rows of the square blocks merge_local's affinity runs for this shape, window and
    requested block_rows (0: the library's pick) on the current device (256 or 128; N
    for rows the persistent kernel does not take)."""
    out = ctypes.c_int32()
    _lib.check("mpm_local_block_rows", _lib.load().mpm_local_block_rows(B, N, D, _DTYPES[dtype], int(grid_w),
                                                                        int(window), int(block_rows),
                                                                        ctypes.byref(out)))
    return out.value


def ws_view(ws: torch.Tensor, B: int, N: int, region: str) -> torch.Tensor:
    """A workspace region as an int32 view: "nb" [B, N] or "src" [B, N, 2]."""
    off = _lib.workspace_offsets(B, N)[region]
    if region == "nb":
        return ws[off:off + 4 * B * N].view(torch.int32).view(B, N)
    if region == "src":
        return ws[off:off + 8 * B * N].view(torch.int32).view(B, N, 2)
    raise KeyError(region)


@dataclass
class Merged:
    y: torch.Tensor       # [B*N, D] packed merged tokens (rows beyond y_off[B] unused)
    y_off: torch.Tensor   # [B+1] int32
    map: torch.Tensor     # [B, N] int32, -1 beyond n_b
    ws: torch.Tensor      # workspace (nb and src regions readable)
    B: int
    N: int
    y_inv: torch.Tensor | None = None  # [B*N] float32 inverse norms of the rows of y, when asked for
    y_pos: torch.Tensor | None = None  # [B*N] int32 grid positions of the rows of y (locality constraint)

    @property
    def nb(self) -> torch.Tensor:
        return ws_view(self.ws, self.B, self.N, "nb")

    @property
    def src(self) -> torch.Tensor:
        return ws_view(self.ws, self.B, self.N, "src")


def takes_norms(D: int, dtype: torch.dtype) -> bool:
    """Whether the affinity accepts given inverse norms for rows of D values of this
    dtype (bfloat16 rows a whole number of 64 bytes)."""
    return dtype == torch.bfloat16 and (2 * D) % 64 == 0


def merge(x, x_off=None, N=None, x_inv=None, want_inv=False, ws=None, schedule="auto") -> Merged:
    """One MPM insertion (Alg. 1) through mpm_merge: the fused affinity + compaction,
    then the pair average (also writing the inverse norms of the merged rows when
    ``want_inv``). ``x_inv``: given inverse norms of the rows of x."""
    x2, B, N, D = _rows(x, N, x_off)
    dev = x.device
    ws = _workspace(B, N, dev, ws)
    y = torch.empty((B * N, D), dtype=x.dtype, device=dev)
    y_off = torch.empty((B + 1,), dtype=torch.int32, device=dev)
    m = torch.empty((B, N), dtype=torch.int32, device=dev)
    y_inv = torch.empty((B * N,), dtype=torch.float32, device=dev) if want_inv else None
    lib = _lib.load()
    _lib.check("mpm_merge", lib.mpm_merge(_p(x2), _p(x_off), _p(x_inv), B, N, D, _dt(x), _sched(schedule), _p(y),
                                          _p(y_off), _p(y_inv), _p(m), _p(ws), ws.numel(), _stream()))
    return Merged(y, y_off, m, ws, B, N, y_inv)


def insertion(x, x_off=None, N=None, x_inv=None, want_inv=False, ws=None, schedule="auto") -> Merged:
    """One MPM insertion through the step entry points: mpm_affinity_compact, then
    mpm_pair_average with the workspace's src. Equal to merge()."""
    x2, B, N, D = _rows(x, N, x_off)
    dev = x.device
    ws = _workspace(B, N, dev, ws)
    y = torch.empty((B * N, D), dtype=x.dtype, device=dev)
    y_off = torch.empty((B + 1,), dtype=torch.int32, device=dev)
    m = torch.empty((B, N), dtype=torch.int32, device=dev)
    y_inv = torch.empty((B * N,), dtype=torch.float32, device=dev) if want_inv else None
    lib, st, dt, n = _lib.load(), _stream(), _dt(x), ws.numel()
    _lib.check("mpm_affinity_compact", lib.mpm_affinity_compact(_p(x2), _p(x_off), _p(x_inv), B, N, D, dt,
                                                                _sched(schedule), _p(m), _p(y_off), _p(ws), n, None,
                                                                None, st))
    src = ws_view(ws, B, N, "src")
    _lib.check("mpm_pair_average", lib.mpm_pair_average(_p(x2), _p(x_off), _p(src), _p(y_off), B, N, D, dt, _p(y),
                                                        _p(y_inv), st))
    return Merged(y, y_off, m, ws, B, N, y_inv)


def merge_local(x, grid_w: int, window: int, x_off=None, N=None, pos=None, ws=None, x_inv=None,
                want_inv=False, block_rows: int = 0) -> Merged:
    """One locality-constrained insertion (Sec. 5): candidates within ``window`` rows and
    columns on a grid of ``grid_w`` columns; ``pos`` the tokens' raster positions
    (packed like x; None: each token's index in its image). The merged rows'
    positions are returned in ``y_pos``; ``x_inv`` / ``want_inv`` as in merge();
    ``block_rows`` 128 or 256 forces the affinity's block size (0: the library's pick)."""
    x2, B, N, D = _rows(x, N, x_off)
    dev = x.device
    ws = _workspace(B, N, dev, ws)
    y = torch.empty((B * N, D), dtype=x.dtype, device=dev)
    y_off = torch.empty((B + 1,), dtype=torch.int32, device=dev)
    y_pos = torch.empty((B * N,), dtype=torch.int32, device=dev)
    m = torch.empty((B, N), dtype=torch.int32, device=dev)
    y_inv = torch.empty((B * N,), dtype=torch.float32, device=dev) if want_inv else None
    _lib.check("mpm_merge_local", _lib.load().mpm_merge_local(_p(x2), _p(x_off), _p(x_inv), _p(pos), B, N, D, _dt(x),
                                                              int(grid_w), int(window), int(block_rows), _p(y),
                                                              _p(y_off), _p(y_inv), _p(y_pos), _p(m), _p(ws),
                                                              ws.numel(), None, None, _stream()))
    return Merged(y, y_off, m, ws, B, N, y_inv, y_pos)


def pad(z, z_off, P: int, out=None):
    """Packed rows z [R, ...] (offsets z_off [B+1]) to [B, P, ...]: image b's rows
    first, zero rows after them (mpm_pad; the row is copied as bytes)."""
    B = z_off.numel() - 1
    row_bytes = math.prod(z.shape[1:]) * z.element_size()
    if out is None:
        out = torch.empty((B, P) + tuple(z.shape[1:]), dtype=z.dtype, device=z.device)
    _lib.check("mpm_pad", _lib.load().mpm_pad(_p(z), _p(z_off), B, int(P), int(row_bytes), _p(out), _stream()))
    return out


def unpad(padded, z_off, out=None, rows: int | None = None):
    """The inverse of pad: [B, P, ...] back to packed rows (mpm_unpad); ``out`` (or a new
    tensor of ``rows`` rows, default B * P) receives them at the offsets z_off."""
    B, P = padded.shape[:2]
    row_bytes = math.prod(padded.shape[2:]) * padded.element_size()
    if out is None:
        out = torch.empty((rows if rows is not None else B * P,) + tuple(padded.shape[2:]), dtype=padded.dtype,
                          device=padded.device)
    _lib.check("mpm_unpad", _lib.load().mpm_unpad(_p(padded), _p(z_off), B, int(P), int(row_bytes), _p(out),
                                                  _stream()))
    return out


def compose(map_a, map_b, out=None):
    """r*(i) = map_b[map_a[i]] per image (Eq. 3); maps [B, N] int32."""
    B, N = map_a.shape
    out = torch.empty_like(map_a) if out is None else out
    lib = _lib.load()
    _lib.check("mpm_compose", lib.mpm_compose(_p(map_a), _p(map_b.contiguous()), B, N, _p(out), _stream()))
    return out


def unmerge(z, z_off, rmap, z_spec=None, out=None):
    """Dense [B, E+N, D] grid: E special rows, then z[z_off[b] + rmap[b, i]] (Eq. 4)."""
    B, N = rmap.shape
    if z.dim() == 3:
        z = z.reshape(-1, z.shape[-1])
    D = z.shape[1]
    E = 0 if z_spec is None else z_spec.shape[1]
    if out is None:
        out = torch.empty((B, E + N, D), dtype=z.dtype, device=z.device)
    lib = _lib.load()
    _lib.check("mpm_unmerge", lib.mpm_unmerge(_p(z), _p(z_off), _p(rmap), _p(z_spec), E, B, N, D, _dt(z), _p(out),
                                              _stream()))
    return out


def compose_unmerge(z, z_off, map_a, map_b, z_spec=None, out=None, map_ab=None):
    """Eq. 3 folded into Eq. 4: gathers through r* = map_b[map_a] per image and
    writes r* to ``map_ab`` (allocated if None). Returns (out, map_ab)."""
    B, N = map_a.shape
    if z.dim() == 3:
        z = z.reshape(-1, z.shape[-1])
    D = z.shape[1]
    E = 0 if z_spec is None else z_spec.shape[1]
    if out is None:
        out = torch.empty((B, E + N, D), dtype=z.dtype, device=z.device)
    if map_ab is None:
        map_ab = torch.empty_like(map_a)
    lib = _lib.load()
    _lib.check("mpm_compose_unmerge", lib.mpm_compose_unmerge(_p(z), _p(z_off), _p(map_a), _p(map_b.contiguous()),
                                                              _p(map_ab), _p(z_spec), E, B, N, D, _dt(z), _p(out),
                                                              _stream()))
    return out, map_ab


@dataclass
class ScheduleResult:
    stages: list          # Merged per insertion
    rstar: torch.Tensor   # composed map [B, N]
    out: torch.Tensor     # reconstructed grid [B, N, D]


def run_schedule(x, insertions: int = 2, workspaces=None, schedule: str = "auto", grid_w: int | None = None,
                 window: int | None = None, block_rows: int = 0) -> ScheduleResult:
    """Insertions with identity blocks in between (Sec. 3.3), composed maps
    (Eq. 3) and one gather back to the full grid (Eq. 4). Each insertion after the
    first takes the inverse norms of its input rows from the pair average that
    wrote them (rows a whole number of 64 bytes), as Schedule does. With
    ``window``, every insertion is locality-constrained (merge_local, with
    ``block_rows``) on a grid of ``grid_w`` columns, the first on the raster positions."""
    B, N, D = x.shape
    norms = takes_norms(D, x.dtype)
    stages = []
    cur, cur_off, cur_inv, cur_pos = x, None, None, None
    rstar = None
    for s in range(insertions):
        ws = None if workspaces is None else workspaces[s]
        if window is not None:
            m = merge_local(cur, grid_w, window, x_off=cur_off, N=N, pos=cur_pos, ws=ws, x_inv=cur_inv,
                            want_inv=norms and s + 1 < insertions, block_rows=block_rows)
        else:
            m = merge(cur, cur_off, N=N, x_inv=cur_inv, want_inv=norms and s + 1 < insertions, ws=ws,
                      schedule=schedule)
        stages.append(m)
        rstar = m.map if rstar is None else compose(rstar, m.map)
        cur, cur_off, cur_inv, cur_pos = m.y, m.y_off, m.y_inv, m.y_pos
    out = unmerge(cur, cur_off, rstar)
    return ScheduleResult(stages, rstar, out)


class Schedule:
    """Preallocated MPM schedule for a fixed batch shape: every buffer is
    allocated once, so ``run`` only launches kernels (no allocation, no host
    synchronisation). Stage s consumes stage s-1's packed output (Sec. 3.3);
    the composed map and the reconstruction follow (Eq. 3, Eq. 4). Each
    insertion runs mpm_merge's two steps through their entry points (the fused
    affinity + compaction, then the pair average), so they can be timed one by
    one; the last composition runs inside the gather.

    ``run(x, marks=None, affinity_events=None)``: when ``marks`` is a list of
    ``n_marks()`` torch.cuda.Event objects, event k is recorded on the current
    stream just before kernel step k (in ``kernel_names`` order) and the last one
    after the gather, so consecutive events bracket single steps. When
    ``affinity_events`` is a list of one (start, stop) pair of timing events
    per insertion, each pair is bound to that insertion's affinity launches
    themselves: no stream command is added, and ``start.elapsed_time(stop)`` is
    their duration. The events must have been recorded once before (torch
    creates them lazily)."""

    def __init__(self, B: int, N: int, D: int, dtype: torch.dtype, insertions: int = 2, device="cuda",
                 schedule: str = "auto", grid_w: int | None = None, window: int | None = None):
        if insertions < 1:
            raise ValueError("at least one insertion")
        self.B, self.N, self.D, self.dtype, self.insertions = B, N, D, dtype, insertions
        self.schedule = _sched(schedule)
        self.grid_w, self.window = grid_w, window  # locality constraint (merge_local) when window is set
        dev = torch.device(device)
        i32 = dict(dtype=torch.int32, device=dev)
        self.ws = [new_workspace(B, N, dev) for _ in range(insertions)]
        self.nb = [ws_view(w, B, N, "nb") for w in self.ws]
        self.src = [ws_view(w, B, N, "src") for w in self.ws]
        self.map = [torch.empty((B, N), **i32) for _ in range(insertions)]
        self.y = [torch.empty((B * N, D), dtype=dtype, device=dev) for _ in range(insertions)]
        self.y_off = [torch.empty((B + 1,), **i32) for _ in range(insertions)]
        # Inverse norms of each insertion's merged rows, for the next insertion's affinity.
        norms = takes_norms(D, dtype)
        self.y_inv = [torch.empty((B * N,), dtype=torch.float32, device=dev) if norms and s + 1 < insertions
                      else None for s in range(insertions)]
        self.y_pos = [torch.empty((B * N,), **i32) if window is not None else None for _ in range(insertions)]
        # With one insertion the map is the composed map: the gather reads it directly.
        self.rstar = self.map[0] if insertions == 1 else torch.empty((B, N), **i32)
        self.rchain = torch.empty((B, N), **i32) if insertions > 2 else None  # maps composed before the last
        self.out = torch.empty((B, N, D), dtype=dtype, device=dev)
        self._lib = _lib.load()
        self._dt = _DTYPES[dtype]

    @property
    def kernel_names(self) -> list:
        names = []
        for s in range(self.insertions):
            names += [f"merge_local{s + 1}"] if self.window is not None else [f"affinity+compact{s + 1}",
                                                                                 f"average{s + 1}"]
        if self.insertions == 1:
            return names + ["unmerge"]
        # the last composition runs inside the gather (mpm_compose_unmerge)
        return names + ["compose"] * (self.insertions - 2) + ["compose+unmerge"]

    def n_marks(self) -> int:
        return len(self.kernel_names) + 1

    def run(self, x: torch.Tensor, marks=None, affinity_events=None) -> torch.Tensor:
        if x.shape != (self.B, self.N, self.D) or x.dtype != self.dtype or not x.is_contiguous():
            raise ValueError("input does not match the schedule's shape/dtype")
        lib, st, B, N, D, dt = self._lib, _stream(), self.B, self.N, self.D, self._dt
        k = 0

        def mark():
            nonlocal k
            if marks is not None:
                marks[k].record()
            k += 1

        cur, cur_off, cur_inv, cur_pos = x, None, None, None
        for s in range(self.insertions):
            ws = self.ws[s]
            mark()
            if self.window is not None:
                ev0, ev1 = (None, None) if affinity_events is None else (c_event(e) for e in affinity_events[s])
                _lib.check("mpm_merge_local", lib.mpm_merge_local(
                    _p(cur), _p(cur_off), _p(cur_inv), _p(cur_pos), B, N, D, dt, self.grid_w, self.window, 0,
                    _p(self.y[s]), _p(self.y_off[s]), _p(self.y_inv[s]), _p(self.y_pos[s]), _p(self.map[s]), _p(ws),
                    ws.numel(), ev0, ev1, st))
                cur, cur_off, cur_inv, cur_pos = self.y[s], self.y_off[s], self.y_inv[s], self.y_pos[s]
                continue
            ev0, ev1 = (None, None) if affinity_events is None else (c_event(e) for e in affinity_events[s])
            _lib.check("mpm_affinity_compact", lib.mpm_affinity_compact(
                _p(cur), _p(cur_off), _p(cur_inv), B, N, D, dt, self.schedule, _p(self.map[s]), _p(self.y_off[s]),
                _p(ws), ws.numel(), ev0, ev1, st))
            mark()
            _lib.check("mpm_pair_average", lib.mpm_pair_average(_p(cur), _p(cur_off), _p(self.src[s]),
                                                                _p(self.y_off[s]), B, N, D, dt, _p(self.y[s]),
                                                                _p(self.y_inv[s]), st))
            cur, cur_off, cur_inv = self.y[s], self.y_off[s], self.y_inv[s]
        if self.insertions == 1:
            mark()
            _lib.check("mpm_unmerge", lib.mpm_unmerge(_p(cur), _p(cur_off), _p(self.rstar), None, 0, B, N, D, dt,
                                                      _p(self.out), st))
        else:
            first = self.map[0]
            for s in range(1, self.insertions - 1):
                mark()
                _lib.check("mpm_compose", lib.mpm_compose(_p(first), _p(self.map[s]), B, N, _p(self.rchain), st))
                first = self.rchain
            mark()
            _lib.check("mpm_compose_unmerge", lib.mpm_compose_unmerge(
                _p(cur), _p(cur_off), _p(first), _p(self.map[-1]), _p(self.rstar), None, 0, B, N, D, dt,
                _p(self.out), st))
        mark()
        return self.out
