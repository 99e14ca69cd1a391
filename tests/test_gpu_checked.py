"""The library's checked mode (MPM_CHECKED=1, read once per process): every entry point
validates the data-dependent preconditions that are otherwise undefined behaviour, on
the device, before launching its operation, and returns MPM_ERR_INVALID_ARG with
nothing launched when one fails. One child process runs every case with the mode on
(the variable is read at the library's first call, which this process has made
already); its valid merge must match this process's unchecked one bit for bit. Each
invalid case breaks one precondition in a way the checks read within bounds (offsets
are validated before anything is walked through them), and the operation is then
never launched."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import paper_2604_05718_amd as mpm

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import json, sys
import numpy as np
import torch
sys.path.insert(0, sys.argv[1])
from paper_2604_05718_amd import api, _lib

lib = _lib.load()
dev = torch.device("cuda:0")
st = api._stream()
P = api._p
B, N, D = 3, 300, 64
rng = np.random.default_rng(5)
ns = [300, 177, 1]
off = np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)
x = torch.from_numpy(rng.standard_normal((off[-1], D)).astype(np.float32)).to(torch.bfloat16).to(dev)
x_off = torch.from_numpy(off).to(dev)
wsb = lib.mpm_workspace_bytes(B, N)
ws = torch.zeros(wsb, dtype=torch.uint8, device=dev)
assert lib.mpm_workspace_init(P(ws), wsb, st) == 0
results = {}

def merge(xx, xo, xinv=None):
    y = torch.zeros((B * N, D), dtype=torch.bfloat16, device=dev)
    y_off = torch.full((B + 1,), -7, dtype=torch.int32, device=dev)
    m = torch.full((B, N), -7, dtype=torch.int32, device=dev)
    rc = lib.mpm_merge(P(xx), P(xo), P(xinv), B, N, D, 1, 0, P(y), P(y_off), None, P(m), P(ws), wsb, st)
    torch.cuda.synchronize()
    return rc, y, y_off, m

rc, y, y_off, m = merge(x, x_off)
results["valid_merge"] = rc
np.savez(sys.argv[2], y=y.view(torch.int16).cpu().numpy(), y_off=y_off.cpu().numpy(), map=m.cpu().numpy())

def untouched(y_off, m):
    return bool((y_off.cpu() == -7).all() and (m.cpu() == -7).all())

for name, bad in [("count_above_N", [0, 301, 478, 479]), ("decreasing", [0, 300, 200, 479]),
                  ("negative_start", [-1, 299, 476, 477])]:
    rc, y2, yo2, m2 = merge(x, torch.tensor(bad, dtype=torch.int32, device=dev))
    results["offsets_" + name] = [rc, untouched(yo2, m2)]
# An empty image is valid: no merged rows, a map of -1.
rc, y2, yo2, m2 = merge(x, torch.tensor([0, 300, 300, 301], dtype=torch.int32, device=dev))
yo2 = yo2.cpu().tolist()
results["empty_image"] = [rc, yo2[2] == yo2[1] and yo2[3] == yo2[2] + 1 and bool((m2[1].cpu() == -1).all())]
xn = x.clone()
xn[200, 5] = float("nan")
rc, _, yo2, m2 = merge(xn, x_off)
results["nan_token"] = [rc, untouched(yo2, m2)]
xi = torch.full((off[-1],), 0.125, dtype=torch.float32, device=dev)
rc, _, _, _ = merge(x, x_off, xi)
results["valid_norms"] = rc
for name, val in [("zero", 0.0), ("negative", -1.0), ("inf", float("inf"))]:
    xb = xi.clone()
    xb[77] = val
    rc, _, yo2, m2 = merge(x, x_off, xb)
    results["norms_" + name] = [rc, untouched(yo2, m2)]

# locality-constrained insertion: positions
def local(pos):
    y = torch.zeros((B * N, D), dtype=torch.bfloat16, device=dev)
    yo = torch.full((B + 1,), -7, dtype=torch.int32, device=dev)
    yp = torch.zeros((B * N,), dtype=torch.int32, device=dev)
    m = torch.full((B, N), -7, dtype=torch.int32, device=dev)
    rc = lib.mpm_merge_local(P(x), P(x_off), None, P(pos), B, N, D, 1, 20, 2, 0, P(y), P(yo), None, P(yp), P(m), P(ws),
                             wsb, None, None, st)
    torch.cuda.synchronize()
    return rc, untouched(yo, m)
pos = np.concatenate([2 * np.arange(n, dtype=np.int32) for n in ns])
results["local_valid"] = local(torch.from_numpy(pos).to(dev))[0]
p2 = pos.copy(); p2[251] = p2[250] - 60          # three grid rows back (row 25 to 22)
results["local_row_back"] = local(torch.from_numpy(p2).to(dev))
p3 = pos.copy(); p3[3] = -5
results["local_negative"] = local(torch.from_numpy(p3).to(dev))

# compaction: neighbours
nb = torch.zeros((B, N), dtype=torch.int32, device=dev)
nb[0, :300] = torch.arange(300, device=dev).flip(0)
nb[0, 150] = 149; nb[0, 149] = 150
nb[1, :177] = torch.arange(177, device=dev).flip(0)
nb[1, 88] = 87; nb[1, 87] = 88
nb[2, 0] = -1
def compact(nbx):
    mm = torch.full((B, N), -7, dtype=torch.int32, device=dev)
    src = torch.zeros((B * N * 2,), dtype=torch.int32, device=dev)
    yo = torch.full((B + 1,), -7, dtype=torch.int32, device=dev)
    rc = lib.mpm_pair_compact(P(nbx), P(x_off), B, N, P(mm), P(src), P(yo), st)
    torch.cuda.synchronize()
    return rc, untouched(yo, mm), src, yo
rc, _, src, yo = compact(nb)
results["compact_valid"] = rc
for name, (b, i, v) in [("nb_out_of_range", (1, 5, 177)), ("nb_self", (0, 10, 10)), ("nb_single", (2, 0, 0))]:
    nbb = nb.clone(); nbb[b, i] = v
    results["compact_" + name] = list(compact(nbb)[:2])

# pair average: sources and merged-row offsets
def average(srcx, yox):
    y = torch.full((B * N, D), 3.0, dtype=torch.bfloat16, device=dev)
    rc = lib.mpm_pair_average(P(x), P(x_off), P(srcx), P(yox), B, N, D, 1, P(y), None, st)
    torch.cuda.synchronize()
    return rc, bool((y.float().cpu() == 3.0).all())
results["average_valid"] = average(src, yo)[0]
sb = src.clone(); sb[2 * (N + 3)] = 177            # image 1 has 177 tokens
results["average_src_out_of_range"] = list(average(sb, yo))
yob = yo.clone(); yob[3] = yob[2] + 2                # image 2 (one token) given two merged rows
results["average_too_many_rows"] = list(average(src, yob))

# compose and gather: maps
ma = torch.zeros((B, N), dtype=torch.int32, device=dev)
mb = torch.zeros((B, N), dtype=torch.int32, device=dev)
def compose(a):
    out = torch.full((B, N), -7, dtype=torch.int32, device=dev)
    rc = lib.mpm_compose(P(a), P(mb), B, N, P(out), st)
    torch.cuda.synchronize()
    return rc, bool((out.cpu() == -7).all())
results["compose_valid"] = compose(ma)[0]
mab = ma.clone(); mab[1, 2] = N
results["compose_out_of_range"] = list(compose(mab))
z_off = torch.tensor([0, 10, 20, 21], dtype=torch.int32, device=dev)
z = torch.ones((21, D), dtype=torch.bfloat16, device=dev)
def unmerge(mp, zo):
    out = torch.full((B, N, D), 3.0, dtype=torch.bfloat16, device=dev)
    rc = lib.mpm_unmerge(P(z), P(zo), P(mp), None, 0, B, N, D, 1, P(out), st)
    torch.cuda.synchronize()
    return rc, bool((out.float().cpu() == 3.0).all())
mu = torch.zeros((B, N), dtype=torch.int32, device=dev)
mu[0, :10] = torch.arange(10, device=dev)
results["unmerge_valid"] = unmerge(mu, z_off)[0]
mub = mu.clone(); mub[2, 0] = 1                      # image 2 has one merged row
results["unmerge_out_of_range"] = list(unmerge(mub, z_off))
results["unmerge_bad_offsets"] = list(unmerge(mu, torch.tensor([0, 10, 5, 21], dtype=torch.int32, device=dev)))

# padded layout
out = torch.zeros((B, 12, D), dtype=torch.bfloat16, device=dev)
results["pad_valid"] = lib.mpm_pad(P(z), P(z_off), B, 12, D * 2, P(out), st)
results["pad_rows_past_P"] = lib.mpm_pad(P(z), P(z_off), B, 9, D * 2, P(out), st)  # rows past P are dropped
results["pad_empty_image"] = lib.mpm_pad(P(z), P(torch.tensor([0, 10, 10, 21], dtype=torch.int32, device=dev)), B,
                                         12, D * 2, P(out), st)
results["pad_bad_offsets"] = lib.mpm_pad(P(z), P(torch.tensor([0, 10, 5, 21], dtype=torch.int32, device=dev)), B,
                                         12, D * 2, P(out), st)
torch.cuda.synchronize()
print("RESULTS " + json.dumps(results), flush=True)
"""


def test_checked_mode(tmp_path):
    saved = str(tmp_path / "valid.npz")
    env = dict(os.environ, MPM_CHECKED="1", PYTHONPATH=ROOT)
    env.pop("MPM_FAULT_INJECT", None)
    print("checked mode: child process with MPM_CHECKED=1", flush=True)
    p = subprocess.run([sys.executable, "-c", CHILD, ROOT, saved], capture_output=True, text=True, env=env,
                       timeout=300)
    assert p.returncode == 0, p.stdout[-3000:] + p.stderr[-3000:]
    line = [ln for ln in p.stdout.splitlines() if ln.startswith("RESULTS ")][-1]
    r = json.loads(line[len("RESULTS "):])
    ok, bad = 0, 1
    for key in ("valid_merge", "valid_norms", "local_valid", "compact_valid", "average_valid", "compose_valid",
                "unmerge_valid", "pad_valid", "pad_rows_past_P", "pad_empty_image"):
        assert r[key] == ok, (key, r[key])
    assert r["empty_image"] == [ok, True]
    for key in ("offsets_count_above_N", "offsets_decreasing", "offsets_negative_start",
                "nan_token", "norms_zero", "norms_negative", "norms_inf", "local_row_back", "local_negative",
                "compact_nb_out_of_range", "compact_nb_self", "compact_nb_single", "average_src_out_of_range",
                "average_too_many_rows", "compose_out_of_range", "unmerge_out_of_range", "unmerge_bad_offsets"):
        assert r[key] == [bad, True], (key, r[key])   # rejected, outputs untouched
    assert r["pad_bad_offsets"] == bad

    # The checked valid merge equals this process's unchecked one, bit for bit.
    got = np.load(saved)
    B, N, D = 3, 300, 64
    rng = np.random.default_rng(5)
    ns = [300, 177, 1]
    off = np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)
    dev = torch.device("cuda:0")
    x = torch.from_numpy(rng.standard_normal((off[-1], D)).astype(np.float32)).to(torch.bfloat16).to(dev)
    res = mpm.merge(x, torch.from_numpy(off).to(dev), N=N)
    torch.cuda.synchronize()
    y_off = res.y_off.cpu().numpy()
    assert np.array_equal(got["y_off"], y_off)
    assert np.array_equal(got["map"], res.map.cpu().numpy())
    assert np.array_equal(got["y"][: y_off[-1]], res.y[: y_off[-1]].view(torch.int16).cpu().numpy())
