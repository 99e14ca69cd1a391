"""C ABI checks that need no GPU: the library loads, exports every function the
header declares, and rejects bad arguments synchronously before any launch."""
import ctypes

import pytest

from paper_2604_05718_amd import _lib

A = ctypes.c_void_p(0x10000)       # stand-in device pointers: never dereferenced,
A2 = ctypes.c_void_p(0x20000)      # the calls below return before any launch
MIS = ctypes.c_void_p(0x10004)     # 4-byte aligned, not 16-byte aligned


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_exports_every_header_function(lib):
    names = _lib.header_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
        assert n in _lib.SIGNATURES, n


def test_version_and_status_strings(lib):
    assert b"gfx950" in lib.mpm_version()
    assert lib.mpm_status_string(0) == b"MPM_OK"
    assert lib.mpm_status_string(3) == b"MPM_ERR_WORKSPACE"
    assert lib.mpm_status_string(99) == b"MPM_UNKNOWN_STATUS"
    assert lib.mpm_last_hip_error() == 0


def test_workspace_bytes_and_offsets(lib):
    r = lambda v: (v + 255) // 256 * 256
    sync = r(4 * 65536)  # MPM_MAX_B + 1 arrival counters, at offset 0 for every shape
    for B, N in [(64, 1024), (16, 4096), (3, 5), (1, 257)]:
        T = (N + 63) // 64  # partial slots per token, include/mpm.h
        want = sync + r(4 * B * N) + r(8 * B * N) + r(4 * B * T * N) + r(4 * B * T * N)
        assert lib.mpm_workspace_bytes(B, N) == want
        off = _lib.workspace_offsets(B, N)
        assert off["sync"] == 0 and off["nb"] == sync and off["src"] == sync + r(4 * B * N)
        assert off["pv"] == off["src"] + r(8 * B * N) and off["pi"] == off["pv"] + r(4 * B * T * N)
        assert all(v % 256 == 0 for v in off.values())
    assert lib.mpm_workspace_bytes(0, 5) == 0
    assert lib.mpm_workspace_offsets(0, 5, None, None, None, None, None) == 1


def test_workspace_init_rejects(lib):
    """Argument errors of mpm_workspace_init, returned before any launch."""
    assert lib.mpm_workspace_init(None, 1 << 20, None) == 1                       # NULL
    assert lib.mpm_workspace_init(ctypes.c_void_p(0x10010), 1 << 20, None) == 1   # not 256-byte aligned
    assert lib.mpm_workspace_init(A, 4 * 65536 - 1, None) == 3                    # smaller than the sync region


AUTO = 0


@pytest.mark.parametrize("args,code", [
    ((A, None, 0, 16, 64, 1, AUTO, A2, None), 1),         # B < 1
    ((A, None, 2, 0, 64, 1, AUTO, A2, None), 1),          # N < 1
    ((A, None, 2, 16, 0, 1, AUTO, A2, None), 1),          # D < 1
    ((A, None, 2, 16, 12, 1, AUTO, A2, None), 1),         # bf16 rows not 16-byte multiples
    ((A, None, 2, 16, 6, 0, AUTO, A2, None), 1),          # f32 rows not 16-byte multiples
    ((A, None, 2, 16, 64, 7, AUTO, A2, None), 1),         # unknown dtype
    ((A, None, 2, 16, 64, 1, 4, A2, None), 1),            # unknown schedule
    ((A, None, 2, 16, 64, 1, -1, A2, None), 1),           # unknown schedule
    ((None, None, 2, 16, 64, 1, AUTO, A2, None), 1),      # null tokens
    ((MIS, None, 2, 16, 64, 1, AUTO, A2, None), 1),       # misaligned tokens
    ((A, None, 2, 16, 64, 1, AUTO, None, None), 1),       # null nb
    ((A, None, 2, 16384 + 1, 64, 1, AUTO, A2, None), 2),  # N above MPM_MAX_N
    ((A, None, 65536, 16, 64, 1, AUTO, A2, None), 2),     # B above MPM_MAX_B
    ((A, None, 2, 16, 16384 + 8, 1, AUTO, A2, None), 2),  # D above MPM_MAX_D
])
def test_argmax_rejects(lib, args, code):
    big = 1 << 40
    assert lib.mpm_argmax(*args, A, big, None) == code
    if args[7] is not None:  # the same rejection holds for the affinity steps (which take no nb)
        x, x_off, B, N, D, dt, sch = args[:7]
        assert lib.mpm_affinity(x, x_off, None, B, N, D, dt, sch, A, big, None, None, None) == code
        assert lib.mpm_affinity_compact(x, x_off, None, B, N, D, dt, sch, A2, A2, A, big, None, None, None) == code
        assert lib.mpm_merge(x, x_off, None, B, N, D, dt, sch, A2, A2, None, A2, A, big, None) == code


def test_workspace_checks(lib):
    need = lib.mpm_workspace_bytes(4, 64)
    # Workspace one byte short.
    assert lib.mpm_merge(A, None, None, 4, 64, 64, 1, AUTO, A2, A2, None, A2, A, need - 1, None) == 3
    assert lib.mpm_affinity(A, None, None, 4, 64, 64, 1, AUTO, A, need - 1, None, None, None) == 3
    assert lib.mpm_affinity_compact(A, None, None, 4, 64, 64, 1, AUTO, A2, A2, A, need - 1, None, None, None) == 3
    assert lib.mpm_argmax(A, None, 4, 64, 64, 1, AUTO, A2, None, A, need - 1, None) == 3
    # Workspace not 256-byte aligned, or missing.
    assert lib.mpm_merge(A, None, None, 4, 64, 64, 1, AUTO, A2, A2, None, A2, ctypes.c_void_p(0x10010), need,
                         None) == 1
    assert lib.mpm_merge(A, None, None, 4, 64, 64, 1, AUTO, A2, A2, None, A2, None, need, None) == 1
    assert lib.mpm_affinity(A, None, None, 4, 64, 64, 1, AUTO, None, need, None, None, None) == 1
    # Null merged-token buffer, offsets or map.
    assert lib.mpm_merge(A, None, None, 4, 64, 64, 1, AUTO, None, A2, None, A2, A, need, None) == 1
    assert lib.mpm_merge(A, None, None, 4, 64, 64, 1, AUTO, A2, None, None, A2, A, need, None) == 1
    assert lib.mpm_merge(A, None, None, 4, 64, 64, 1, AUTO, A2, A2, None, None, A, need, None) == 1
    assert lib.mpm_affinity_compact(A, None, None, 4, 64, 64, 1, AUTO, None, A2, A, need, None, None, None) == 1
    assert lib.mpm_affinity_compact(A, None, None, 4, 64, 64, 1, AUTO, A2, None, A, need, None, None, None) == 1


def test_other_entry_points_reject(lib):
    assert lib.mpm_pair_compact(A, None, 0, 8, A, A, A, None) == 1
    assert lib.mpm_pair_compact(None, None, 2, 8, A, A, A, None) == 1
    assert lib.mpm_pair_compact(A, None, 2, 8, A, A, None, None) == 1            # y_off NULL
    assert lib.mpm_pair_average(A, None, A, A, 2, 8, 64, 1, MIS, None, None) == 1  # y misaligned
    assert lib.mpm_pair_average(A, None, A, None, 2, 8, 64, 1, A2, None, None) == 1  # y_off NULL
    assert lib.mpm_pair_average(A, None, A, A, 2, 8, 63, 1, A2, None, None) == 1   # D % 8 (bf16)
    assert lib.mpm_pair_average(A, None, A, A, 2, 8, 64, 1, A2, ctypes.c_void_p(0x20002), None) == 1  # y_inv
    assert lib.mpm_compose(A, None, 2, 8, A, None) == 1
    assert lib.mpm_compose(A, A, 2, 16385, A, None) == 2
    assert lib.mpm_unmerge(A, None, A, None, -1, 2, 8, 64, 1, A, None) == 1   # E < 0
    assert lib.mpm_unmerge(A, None, A, None, 2, 2, 8, 64, 1, A, None) == 1    # E > 0 needs z_spec
    assert lib.mpm_unmerge(A, None, A, None, 0, 2, 8, 64, 1, None, None) == 1
    # compose + gather: the same checks, plus the composed map must not alias an input map
    A3 = ctypes.c_void_p(0x30000)
    assert lib.mpm_compose_unmerge(A, None, A, A2, A3, None, -1, 2, 8, 64, 1, A, None) == 1   # E < 0
    assert lib.mpm_compose_unmerge(A, None, A, None, A3, None, 0, 2, 8, 64, 1, A, None) == 1  # map_b NULL
    assert lib.mpm_compose_unmerge(A, None, A, A2, A, None, 0, 2, 8, 64, 1, A, None) == 1     # map_ab == map_a
    assert lib.mpm_compose_unmerge(A, None, A, A2, A2, None, 0, 2, 8, 64, 1, A, None) == 1    # map_ab == map_b
    assert lib.mpm_compose_unmerge(A, None, A, A2, A3, None, 0, 2, 8, 63, 1, A, None) == 1    # D % 8 (bf16)
    assert lib.mpm_compose_unmerge(A, None, A, A2, A3, None, 0, 2, 16385, 64, 1, A, None) == 2
    assert lib.mpm_last_hip_error() == 0


def test_pad_unpad_and_local_reject(lib):
    """mpm_pad / mpm_unpad and mpm_merge_local return their argument errors before any
    device work: sizes, row bytes that are not whole 16-byte vectors, NULL or misaligned
    pointers, a grid or window the locality constraint cannot take, a short workspace,
    given norms for rows the norm-taking kernel does not cover."""
    for fn in (lib.mpm_pad, lib.mpm_unpad):
        assert fn(A, A, 0, 8, 64, A2, None) == 1             # B < 1
        assert fn(A, A, 2, 0, 64, A2, None) == 1             # P < 1
        assert fn(A, A, 2, 8, 8, A2, None) == 1              # row_bytes < 16
        assert fn(A, A, 2, 8, 40, A2, None) == 1             # row_bytes % 16
        assert fn(A, None, 2, 8, 64, A2, None) == 1          # z_off NULL
        assert fn(MIS, A, 2, 8, 64, A2, None) == 1           # rows misaligned
        assert fn(A, A, 2, 8, 64, MIS, None) == 1
        assert fn(A, A, 65536, 8, 64, A2, None) == 2         # B > MPM_MAX_B
        assert fn(A, A, 2, 16385, 64, A2, None) == 2         # P > MPM_MAX_N
    ws = ctypes.c_size_t(1 << 30)
    odd = ctypes.c_void_p(0x10002)
    ok = dict(pos=None, grid_w=8, window=1, y_pos=A2)

    def local(**kw):
        a = dict(ok, **kw)
        return lib.mpm_merge_local(A, None, a.get("x_inv"), a["pos"], 2, 64, a.get("D", 64), a.get("dt", 1),
                                   a["grid_w"], a["window"], a.get("block_rows", 0), A2, A2, a.get("y_inv"),
                                   a["y_pos"], A2, A2, a.get("ws", ws), None, None, None)
    assert local(grid_w=0) == 1
    assert local(grid_w=16385) == 1
    assert local(window=-1) == 1
    assert local(y_pos=None) == 1
    assert local(pos=odd) == 1                                # positions misaligned
    assert local(ws=16) == 3                                  # workspace too small
    assert local(D=63) == 1                                   # D % 8 (bf16)
    assert local(x_inv=odd) == 1                              # given norms misaligned
    assert local(y_inv=odd) == 1
    assert local(x_inv=A, D=40) == 2                          # given norms: 80-byte rows
    assert local(x_inv=A, dt=0) == 2                          # given norms: float32 rows
    for rows in (64, 192, 512, -1):
        assert local(block_rows=rows) == 1                    # block sizes: 0, 128 or 256
    out = ctypes.c_int32(-7)
    query = lib.mpm_local_block_rows
    assert query(2, 64, 64, 1, 8, 1, 0, None) == 1            # NULL output
    assert query(2, 64, 64, 1, 0, 1, 0, ctypes.byref(out)) == 1
    assert query(2, 64, 64, 1, 8, -1, 0, ctypes.byref(out)) == 1
    assert query(2, 64, 64, 1, 8, 1, 96, ctypes.byref(out)) == 1
    assert query(0, 64, 64, 1, 8, 1, 0, ctypes.byref(out)) == 1
    assert out.value == -7
    assert lib.mpm_last_hip_error() == 0


def test_given_norms_reject(lib):
    """Given inverse norms: a misaligned pointer, and rows the norm-taking kernels do
    not cover, are rejected by every affinity entry point."""
    ws = ctypes.c_size_t(1 << 30)
    bad = ctypes.c_void_p(0x10002)
    for D, dt, code in [(64, 1, 1), (40, 1, 2), (8, 1, 2), (64, 0, 2)]:  # misaligned; 80-, 16-byte, f32 rows
        ptr = bad if code == 1 else A
        assert lib.mpm_affinity(A, None, ptr, 2, 8, D, dt, AUTO, A2, ws, None, None, None) == code
        assert lib.mpm_affinity_compact(A, None, ptr, 2, 8, D, dt, AUTO, A2, A2, A2, ws, None, None, None) == code
        assert lib.mpm_merge(A, None, ptr, 2, 8, D, dt, AUTO, A2, A2, None, A2, A2, ws, None) == code
    assert lib.mpm_affinity(MIS, None, A, 2, 8, 64, 1, AUTO, A2, ws, None, None, None) == 1      # x misaligned
    assert lib.mpm_affinity(A, None, A, 2, 8, 64, 1, AUTO, A2, 16, None, None, None) == 3        # workspace
    assert lib.mpm_last_hip_error() == 0


def test_schedule_query_rejects(lib):
    """The schedule is an argument of every affinity call (the library holds no mode);
    the query rejects bad sizes, unknown schedules and a NULL output without writing it."""
    out = ctypes.c_int32(-7)
    assert lib.mpm_affinity_schedule_used(0, 1024, 768, 1, AUTO, ctypes.byref(out)) == _lib.MPM_ERR_INVALID_ARG
    assert lib.mpm_affinity_schedule_used(64, 1024, 768, 1, 9, ctypes.byref(out)) == _lib.MPM_ERR_INVALID_ARG
    assert lib.mpm_affinity_schedule_used(64, 1024, 768, 1, AUTO, None) == _lib.MPM_ERR_INVALID_ARG
    assert out.value == -7
    assert not hasattr(lib, "mpm_set_affinity_schedule")
    import paper_2604_05718_amd as mpm
    with pytest.raises(ValueError):
        mpm.affinity_schedule_used(64, 1024, 768, __import__("torch").bfloat16, "diagonal")


def test_noalloc_rejects_before_any_device_use(lib):
    """mpm_merge_noalloc: argument errors and shapes beyond its fixed device array are
    rejected before the array is looked up (no GPU needed)."""
    cap = 48 << 20
    assert lib.mpm_workspace_bytes(64, 4096) > cap >= lib.mpm_workspace_bytes(16, 4096)
    assert lib.mpm_workspace_bytes(64, 1024) <= cap and lib.mpm_workspace_bytes(32, 2304) <= cap
    assert lib.mpm_merge_noalloc(A, None, None, 64, 4096, 64, 1, AUTO, A2, A2, None, A2, None) == 3
    assert lib.mpm_merge_noalloc(A, None, None, 0, 16, 64, 1, AUTO, A2, A2, None, A2, None) == 1     # B < 1
    assert lib.mpm_merge_noalloc(MIS, None, None, 2, 16, 64, 1, AUTO, A2, A2, None, A2, None) == 1   # x misaligned
    assert lib.mpm_merge_noalloc(A, None, None, 2, 16, 64, 1, 9, A2, A2, None, A2, None) == 1        # schedule
    assert lib.mpm_merge_noalloc(A, None, None, 2, 16, 64, 1, AUTO, None, A2, None, A2, None) == 1   # y NULL
    assert lib.mpm_merge_noalloc(A, None, None, 2, 16, 64, 1, AUTO, A2, A2, None, None, None) == 1   # map NULL
    assert lib.mpm_merge_noalloc(A, None, A, 2, 16, 64, 0, AUTO, A2, A2, None, A2, None) == 2        # f32 norms
    assert lib.mpm_last_hip_error() == 0
