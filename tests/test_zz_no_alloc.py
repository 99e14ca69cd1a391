"""mpm_merge_noalloc (the insertion whose workspace is the library's own device
array, for callers that cannot allocate) against mpm_merge with a caller
workspace, through the C ABI, bit for bit: two calls in a row on one device, the
second with a smaller, packed input, so it runs on what the first left in the
array; and the size limit."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2604_05718_amd import _lib, api, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _noalloc(lib, x2, x_off, x_inv, B, N, D, dt, want_inv):
    y = torch.full((B * N, D), 7, dtype=x2.dtype, device=DEV)
    y_off = torch.full((B + 1,), -5, dtype=torch.int32, device=DEV)
    m = torch.full((B, N), -9, dtype=torch.int32, device=DEV)
    y_inv = torch.full((B * N,), -1.0, dtype=torch.float32, device=DEV) if want_inv else None
    _lib.check("mpm_merge_noalloc", lib.mpm_merge_noalloc(
        api._p(x2), api._p(x_off), api._p(x_inv), B, N, D, dt, 0, api._p(y), api._p(y_off), api._p(y_inv),
        api._p(m), api._stream()))
    return y, y_off, m, y_inv


def _same(a, b, rows):
    assert torch.equal(a.y_off, b[1])
    assert torch.equal(a.map, b[2])
    assert torch.equal(a.y[:rows].view(torch.int16), b[0][:rows].view(torch.int16))
    if a.y_inv is not None:
        assert torch.equal(a.y_inv[:rows].view(torch.int32), b[3][:rows].view(torch.int32))


def test_noalloc_matches_merge_twice():
    lib = _lib.load()
    # First call: 16 images of the ViT-B/16 512x512 shape, dense, writing the merged rows' norms.
    cfg = synth.config("vit_b_512")
    x = synth.make_batch(cfg, seed=3, images=list(range(16))).to(DEV)
    B, N, D = 16, cfg.N, cfg.D
    print(f"noalloc call 1: B={B} N={N} D={D} bf16 dense", flush=True)
    ref = api.merge(x, want_inv=True)
    got = _noalloc(lib, x.view(B * N, D), None, None, B, N, D, _lib.MPM_BF16, True)
    torch.cuda.synchronize()
    _same(ref, got, int(ref.y_off[-1]))
    # Second call: smaller and packed (the first call's merged rows of 5 images, with their
    # given inverse norms), on what the first call left in the array.
    B2 = 5
    rows = int(ref.y_off[B2])
    x2, off2, inv2 = ref.y[:rows].contiguous(), ref.y_off[: B2 + 1].contiguous(), ref.y_inv[:rows].contiguous()
    print(f"noalloc call 2: B={B2} N={N} D={D} bf16 packed ({rows} rows), given norms", flush=True)
    ref2 = api.merge(x2, off2, N=N, x_inv=inv2)
    got2 = _noalloc(lib, x2, off2, inv2, B2, N, D, _lib.MPM_BF16, False)
    torch.cuda.synchronize()
    _same(ref2, got2, int(ref2.y_off[-1]))
    assert np.all(np.diff(got2[1].cpu().numpy()) >= 1)


def test_noalloc_rejects_shapes_beyond_its_array():
    lib = _lib.load()
    cap = 48 << 20
    A = ctypes.c_void_p(0x10000)
    B, N = 64, 4096  # mpm_workspace_bytes(64, 4096) is well above the array
    assert lib.mpm_workspace_bytes(B, N) > cap
    assert lib.mpm_merge_noalloc(A, None, None, B, N, 64, _lib.MPM_BF16, 0, A, A, None, A, None) == _lib.MPM_ERR_WORKSPACE
