"""ctypes view of libmpm.so: the C ABI declared in include/mpm.h, nothing more.

Loading fails loudly when the library has not been built; there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
import re

from .build import ROOT, library_path

HEADER = os.path.join(ROOT, "include", "mpm.h")

MPM_OK = 0
MPM_ERR_INVALID_ARG = 1
MPM_ERR_UNSUPPORTED = 2
MPM_ERR_WORKSPACE = 3
MPM_ERR_HIP = 4
MPM_F32 = 0
MPM_BF16 = 1
MPM_SCHEDULE_AUTO = 0
MPM_SCHEDULE_FULL = 1
MPM_SCHEDULE_SYMMETRIC = 2
MPM_SCHEDULE_FULL_64 = 3

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_sz = ctypes.c_size_t

_szp = ctypes.POINTER(ctypes.c_size_t)

# name -> (restype, argtypes); mirrors include/mpm.h
SIGNATURES = {
    "mpm_version": (ctypes.c_char_p, []),
    "mpm_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "mpm_last_hip_error": (ctypes.c_int, []),
    "mpm_workspace_bytes": (_sz, [_i32, _i32]),
    "mpm_workspace_offsets": (ctypes.c_int, [_i32, _i32, _szp, _szp, _szp, _szp, _szp]),
    "mpm_workspace_init": (ctypes.c_int, [_vp, _sz, _vp]),
    "mpm_affinity": (ctypes.c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _sz, _vp, _vp, _vp]),
    "mpm_affinity_compact": (ctypes.c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _sz, _vp, _vp,
                                            _vp]),
    "mpm_affinity_schedule_used": (ctypes.c_int, [_i32, _i32, _i32, _i32, _i32, ctypes.POINTER(ctypes.c_int32)]),
    "mpm_local_block_rows": (ctypes.c_int, [_i32, _i32, _i32, _i32, _i32, _i32, _i32,
                                            ctypes.POINTER(ctypes.c_int32)]),
    "mpm_argmax": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _sz, _vp]),
    "mpm_pair_compact": (ctypes.c_int, [_vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp]),
    "mpm_pair_average": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _vp, _vp, _vp]),
    "mpm_merge": (ctypes.c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "mpm_merge_local": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp,
                                       _vp, _vp, _vp, _sz, _vp, _vp, _vp]),
    "mpm_merge_noalloc": (ctypes.c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp]),
    "mpm_pad": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, _vp, _vp]),
    "mpm_unpad": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, _vp, _vp]),
    "mpm_compose": (ctypes.c_int, [_vp, _vp, _i32, _i32, _vp, _vp]),
    "mpm_compose_unmerge": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp]),
    "mpm_unmerge": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp]),
}


class MPMError(RuntimeError):
    def __init__(self, fn: str, status: int, hip_error: int = 0):
        self.status = status
        self.hip_error = hip_error
        name = _STATUS_NAMES.get(status, f"status {status}")
        extra = f" (hipError_t {hip_error})" if status == MPM_ERR_HIP else ""
        super().__init__(f"{fn} returned {name}{extra}")


_STATUS_NAMES = {
    MPM_OK: "MPM_OK",
    MPM_ERR_INVALID_ARG: "MPM_ERR_INVALID_ARG",
    MPM_ERR_UNSUPPORTED: "MPM_ERR_UNSUPPORTED",
    MPM_ERR_WORKSPACE: "MPM_ERR_WORKSPACE",
    MPM_ERR_HIP: "MPM_ERR_HIP",
}

_lib = None


def header_functions() -> list[str]:
    """Names of the functions include/mpm.h declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"\b(mpm_[a-z_0-9]+)\s*\(", text)


def load():
    """Load libmpm.so (built by paper_2604_05718_amd.build); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is missing: build the HIP library first "
            "(python -c 'import __graft_entry__; __graft_entry__.build()')")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def workspace_offsets(B: int, N: int) -> dict:
    """Byte offsets of the workspace regions (sync, nb, src, pv, pi)."""
    vals = [ctypes.c_size_t() for _ in range(5)]
    check("mpm_workspace_offsets", load().mpm_workspace_offsets(B, N, *[ctypes.byref(v) for v in vals]))
    return dict(zip(("sync", "nb", "src", "pv", "pi"), (v.value for v in vals)))


def check(fn: str, status: int) -> None:
    if status != MPM_OK:
        raise MPMError(fn, status, load().mpm_last_hip_error() if status == MPM_ERR_HIP else 0)
