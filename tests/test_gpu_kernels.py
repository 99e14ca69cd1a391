"""Kernel-level parity of the HIP path against the oracle, at small and odd
shapes that span several tiles and ragged tails (every call goes through the C
ABI via the ctypes binding)."""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2604_05718_amd as mpm
from golden_io import all_merge_cases, load
from parity import check_nearest, check_schedule_image, check_stage, rel_err, to64

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def clustered(rng, n, D, k=6, sigma=0.3):
    cent = rng.standard_normal((k, D))
    lab = rng.integers(0, k, n)
    return cent[lab] + sigma * rng.standard_normal((n, D))


def store(x64, dtype):
    return torch.from_numpy(np.asarray(x64, np.float32)).to(TORCH_DT[dtype])


SHAPES = [(1, 1, 64), (1, 2, 16), (2, 3, 8), (3, 17, 24), (2, 64, 64), (2, 127, 72), (1, 129, 136),
          (2, 257, 200), (1, 1000, 384), (1, 300, 1032)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,N,D", SHAPES)
def test_argmax_dense(dtype, B, N, D):
    print(f"argmax dense {dtype} B={B} N={N} D={D}", flush=True)
    rng = np.random.default_rng(N * 1000 + D)
    x = torch.stack([store(clustered(rng, N, D), dtype) for _ in range(B)])
    nb, best = mpm.argmax(x.to(DEV), with_best=True)
    torch.cuda.synchronize()
    nb = nb.cpu().numpy()
    best = best.cpu().numpy()
    for b in range(B):
        x64 = to64(x[b])
        nn, flips, near = check_nearest(x64, nb[b])
        if N == 1:
            assert nb[b, 0] == -1
            continue
        # Diagnostic cosine of the chosen pair, float32 accuracy.
        want = np.array([oracle.cosine(x64, i, int(nb[b, i])) for i in range(N)])
        assert np.abs(best[b] - want).max() < 2e-5


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_argmax_packed_ragged(dtype):
    rng = np.random.default_rng(5)
    N, D = 300, 96
    ns = [1, 2, 300, 37, 129, 128, 255, 64]
    rows = [store(clustered(rng, n, D), dtype) for n in ns]
    off = np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)
    x = torch.cat(rows).to(DEV)
    x_off = torch.from_numpy(off).to(DEV)
    nb = mpm.argmax(x, x_off=x_off, N=N)
    torch.cuda.synchronize()
    nb = nb.cpu().numpy()
    for b, n in enumerate(ns):
        print(f"packed {dtype} image {b} n={n}", flush=True)
        check_nearest(to64(rows[b]), nb[b, :n])
        if n == 1:
            assert nb[b, 0] == -1


def _pad(x, D):
    out = np.zeros((x.shape[0], D))
    out[:, : x.shape[1]] = x
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name", all_merge_cases())
def test_hand_cases(dtype, name):
    g = load(name)
    x = store(oracle.round_to(_pad(g["x"], 16), dtype), dtype)
    res = mpm.merge(x[None].to(DEV))
    torch.cuda.synchronize()
    assert res.nb[0].cpu().tolist() == g["nb"]
    assert res.map[0].cpu().tolist() == g["map"]
    off = res.y_off.cpu().tolist()
    assert off == [0, g["count"]]
    if "clusters" in g:
        y = to64(res.y[: g["count"]])
        for k, members in enumerate(g["clusters"]):
            want = oracle.round_to(to64(x)[members].mean(axis=0), dtype)
            np.testing.assert_array_equal(y[k], want)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_h6_schedule(dtype):
    g = load("h6_blocks.txt")
    x = store(_pad(g["x"], 16), dtype)[None].to(DEV)
    res = mpm.run_schedule(x, insertions=2)
    torch.cuda.synchronize()
    assert res.stages[0].nb[0].cpu().tolist() == g["nb"]
    assert res.stages[1].nb[0, :12].cpu().tolist() == g["nb2"]
    assert res.stages[1].map[0, :12].cpu().tolist() == g["map2"]
    assert res.rstar[0].cpu().tolist() == g["rstar"]
    assert torch.equal(res.out.cpu(), x.cpu())


def random_nb(rng, n, pair_frac=0.4):
    """Neighbour vectors with many mutual pairs and many one-way choices."""
    nb = np.empty(n, np.int32)
    perm = rng.permutation(n)
    npairs = int(pair_frac * n) // 2
    for k in range(npairs):
        a, b = perm[2 * k], perm[2 * k + 1]
        nb[a], nb[b] = b, a
    for i in perm[2 * npairs:]:
        j = rng.integers(0, n - 1) if n > 1 else -1
        nb[i] = j + (j >= i) if n > 1 else -1
    return nb


@pytest.mark.parametrize("N", [1, 2, 5, 1023, 1024, 1025, 4096, 5000])
def test_pair_compact_bitexact(N):
    rng = np.random.default_rng(N)
    B = 3
    ns = [N, max(1, N // 2), max(1, N - 1)]
    nb = np.full((B, N), -7, np.int32)
    for b, n in enumerate(ns):
        nb[b, :n] = random_nb(rng, n)
    off = torch.from_numpy(np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)).to(DEV)
    m, src, y_off = mpm.pair_compact(torch.from_numpy(nb).to(DEV), x_off=off)
    torch.cuda.synchronize()
    m, src, y_off = m.cpu().numpy(), src.cpu().numpy(), y_off.cpu().numpy()
    count = np.diff(y_off)
    assert y_off[0] == 0
    for b, n in enumerate(ns):
        pr = oracle.pairs(nb[b, :n])
        assert count[b] == pr.count
        assert np.array_equal(m[b, :n], pr.map)
        assert np.all(m[b, n:] == -1)
        assert np.array_equal(src[b, : pr.count, 0], pr.src_a)
        assert np.array_equal(src[b, : pr.count, 1], pr.src_b)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("D", [8, 64, 200, 768, 1024])
def test_pair_average(dtype, D):
    rng = np.random.default_rng(D)
    B, N = 3, 257
    ns = [257, 100, 1]
    rows = [store(rng.standard_normal((n, D)) * rng.uniform(0.01, 100), dtype) for n in ns]
    x = torch.cat(rows).to(DEV)
    x_off = torch.from_numpy(np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)).to(DEV)
    nb = np.full((B, N), -1, np.int32)
    prs = []
    for b, n in enumerate(ns):
        nb[b, :n] = random_nb(rng, n)
        prs.append(oracle.pairs(nb[b, :n]))
    m, src, y_off = mpm.pair_compact(torch.from_numpy(nb).to(DEV), x_off=x_off)
    y = mpm.pair_average(x, src, y_off, x_off=x_off, N=N)
    torch.cuda.synchronize()
    off = y_off.cpu().numpy()
    assert off.tolist() == [0] + np.cumsum([p.count for p in prs]).tolist()
    for b in range(B):
        want = oracle.average(to64(rows[b]), prs[b].src_a, prs[b].src_b, dtype)
        got = to64(y[off[b]:off[b + 1]])
        assert rel_err(got, want) <= (1e-5 if dtype == "f32" else 2e-2)
        # Expected bit-exact: float32 sums of two stored values are exact here.
        assert np.array_equal(got, want)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("D", [8, 64, 768, 2048, 2056, 16384])
def test_pair_average_inverse_norms(dtype, D):
    """mpm_pair_average with y_inv: the same merged rows as without, bit for bit,
    on rows of 16 bytes to 64 KB (1 to 4096 vectors of 16 bytes: 1 to 64 lanes per
    row, one or several batches of vectors per lane, a ragged last batch),
    and 1 / max(||y_k||, 1e-12) of every merged row against float64 norms of the
    stored rows (float32 sums of up to 16384 squares), the same on a second run;
    an all-zero row gives 1e12."""
    rng = np.random.default_rng(D + 7)
    N = 257 if D <= 2056 else 40
    ns = [N, max(1, N // 2), 1]
    B = len(ns)
    rows = [rng.standard_normal((n, D)) * rng.uniform(0.01, 100) for n in ns]
    rows[1][3] = 0.0  # a zero token (its cluster is a singleton or a pair)
    rows = [store(r, dtype) for r in rows]
    x = torch.cat(rows).to(DEV)
    x_off = torch.from_numpy(np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)).to(DEV)
    nb = np.full((B, N), -1, np.int32)
    for b, n in enumerate(ns):
        nb[b, :n] = random_nb(rng, n)
    nb[1, 3] = -1 if ns[1] == 1 else nb[1, 3]
    m, src, y_off = mpm.pair_compact(torch.from_numpy(nb).to(DEV), x_off=x_off)
    y = mpm.pair_average(x, src, y_off, x_off=x_off, N=N)
    y2, inv = mpm.pair_average(x, src, y_off, x_off=x_off, N=N, with_inv=True)
    _, inv2 = mpm.pair_average(x, src, y_off, x_off=x_off, N=N, with_inv=True)
    torch.cuda.synchronize()
    total = int(y_off[B].item())
    assert torch.equal(y[:total].view(torch.int16 if dtype == "bf16" else torch.int32),
                       y2[:total].view(torch.int16 if dtype == "bf16" else torch.int32))
    assert torch.equal(inv[:total].view(torch.int32), inv2[:total].view(torch.int32))
    norm = np.sqrt((to64(y2[:total]) ** 2).sum(axis=1))
    want = 1.0 / np.maximum(norm, 1e-12)
    got = inv[:total].cpu().numpy().astype(np.float64)
    zero = norm == 0
    assert np.all(got[zero] == np.float32(1e12))
    assert np.max(np.abs(got[~zero] / want[~zero] - 1.0)) < 2e-5


def test_compose_and_unmerge_with_special_rows():
    rng = np.random.default_rng(9)
    B, N, D, E = 3, 50, 24, 2
    n1s = [30, 50, 1]
    n2s = [20, 26, 1]
    r1 = np.full((B, N), -1, np.int32)
    r2 = np.full((B, N), -1, np.int32)
    for b in range(B):
        r1[b] = np.concatenate([np.arange(n1s[b]), rng.integers(0, n1s[b], N - n1s[b])])
        r2[b, : n1s[b]] = np.concatenate([np.arange(n2s[b]), rng.integers(0, n2s[b], n1s[b] - n2s[b])])
    r1[1, 7] = -1  # a token outside the image: reconstructed as zeros
    rstar = mpm.compose(torch.from_numpy(r1).to(DEV), torch.from_numpy(r2).to(DEV))
    z = torch.randn(sum(n2s), D, dtype=torch.bfloat16)
    z_off = torch.from_numpy(np.concatenate([[0], np.cumsum(n2s)]).astype(np.int32))
    spec = torch.randn(B, E, D, dtype=torch.bfloat16)
    out = mpm.unmerge(z.to(DEV), z_off.to(DEV), rstar, z_spec=spec.to(DEV))
    torch.cuda.synchronize()
    rs = rstar.cpu().numpy()
    for b in range(B):
        want_r = oracle.compose(r1[b], r2[b])
        assert np.array_equal(rs[b], want_r)
        zb = to64(z[z_off[b]:z_off[b + 1]])
        got = to64(out[b])
        assert np.array_equal(got[:E], to64(spec[b]))
        for i in range(N):
            want = zb[want_r[i]] if want_r[i] >= 0 else np.zeros(D)
            assert np.array_equal(got[E + i], want)


@pytest.mark.parametrize("B", [4, 9])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("packed,E", [(True, 2), (False, 0), (True, 0)])
def test_compose_unmerge_matches_compose_then_unmerge(dtype, packed, E, B):
    """mpm_compose_unmerge (Eq. 3 folded into Eq. 4) equals mpm_compose followed by
    mpm_unmerge bit for bit, and a host gather through the oracle's composition; it
    works with the composed-map output omitted (NULL). Nine images take the gather's
    XCD-major workgroup order, four the plain one."""
    from paper_2604_05718_amd import _lib, api

    rng = np.random.default_rng(11)
    N, D = 200, 40
    n1s = [150, 200, 1, 97, 200, 3, 64, 120, 2][:B]
    n2s = [110, 133, 1, 60, 100, 2, 33, 61, 1][:B]
    r1 = np.full((B, N), -1, np.int32)
    r2 = np.full((B, N), -1, np.int32)
    for b in range(B):
        r1[b] = np.concatenate([np.arange(n1s[b]), rng.integers(0, n1s[b], N - n1s[b])])
        r2[b, : n1s[b]] = np.concatenate([np.arange(n2s[b]), rng.integers(0, n2s[b], n1s[b] - n2s[b])])
    r1[3, 11] = -1  # a slot outside the image
    tdt = TORCH_DT[dtype]
    if packed:
        z = torch.randn(sum(n2s), D).to(tdt).to(DEV)
        z_off = torch.from_numpy(np.concatenate([[0], np.cumsum(n2s)]).astype(np.int32)).to(DEV)
    else:
        z = torch.randn(B * N, D).to(tdt).to(DEV)
        z_off = None
    spec = torch.randn(B, E, D).to(tdt).to(DEV) if E else None
    m1 = torch.from_numpy(r1).to(DEV)
    m2 = torch.from_numpy(r2).to(DEV)
    ref_r = mpm.compose(m1, m2)
    ref = mpm.unmerge(z, z_off, ref_r, z_spec=spec)
    out, rstar = api.compose_unmerge(z, z_off, m1, m2, z_spec=spec)
    out2 = torch.full_like(out, 7)
    lib = _lib.load()
    _lib.check("mpm_compose_unmerge", lib.mpm_compose_unmerge(
        api._p(z), api._p(z_off), api._p(m1), api._p(m2), None, api._p(spec), E, B, N, D,
        _lib.MPM_BF16 if dtype == "bf16" else _lib.MPM_F32, api._p(out2), api._stream()))
    torch.cuda.synchronize()
    assert torch.equal(rstar, ref_r)
    assert torch.equal(out, ref)
    assert torch.equal(out2, ref)
    rs = rstar.cpu().numpy()
    zc = z.float().cpu().numpy()
    oc = out.float().cpu().numpy()
    sc = spec.float().cpu().numpy() if E else None
    zo = np.concatenate([[0], np.cumsum(n2s)]) if packed else np.arange(B + 1) * N
    for b in range(B):
        assert np.array_equal(rs[b], oracle.compose(r1[b], r2[b]))
        want = np.zeros((E + N, D))
        if E:
            want[:E] = sc[b]
        live = rs[b] >= 0
        want[E:][live] = zc[zo[b] + rs[b][live]]
        assert np.array_equal(oc[b], want), b


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_duplicated_patches_closed_form(dtype):
    """Exact 2x2 duplicates: N1 = 3N/4, N2 = N/2, exact reconstruction."""
    G, D = 16, 64
    rng = np.random.default_rng(2)
    base = rng.standard_normal((G // 2, G // 2, D))
    x = store(np.repeat(np.repeat(base, 2, 0), 2, 1).reshape(G * G, D), dtype)[None].to(DEV)
    res = mpm.run_schedule(x, insertions=2)
    torch.cuda.synchronize()
    assert res.stages[0].y_off.cpu().tolist() == [0, 3 * G * G // 4]
    assert res.stages[1].y_off.cpu().tolist() == [0, G * G // 2]
    assert torch.equal(res.out.cpu(), x.cpu())


def test_schedule_small_batch_all_images():
    """Full protocol on a small bf16 batch: several query blocks, ragged stage 2."""
    rng = np.random.default_rng(12)
    B, N, D = 4, 700, 128
    x = torch.stack([store(clustered(rng, N, D, k=20, sigma=0.25), "bf16") for _ in range(B)])
    res = mpm.run_schedule(x.to(DEV), insertions=2)
    torch.cuda.synchronize()
    for b in range(B):
        check_schedule_image(x[b], "bf16", res, b)


@pytest.mark.parametrize("insertions", [3, 4])
def test_schedule_more_insertions(insertions):
    """Three and four insertions on a bf16 batch: every insertion after the first
    takes the inverse norms the previous pair average wrote (including rows merged
    from rows that were themselves merged with given norms). Every stage passes the
    oracle check, and the preallocated Schedule equals run_schedule bit for bit."""
    from paper_2604_05718_amd import api

    rng = np.random.default_rng(30 + insertions)
    B, N, D = 3, 700, 128
    x = torch.stack([store(clustered(rng, N, D, k=20, sigma=0.25), "bf16") for _ in range(B)])
    print(f"more insertions {insertions} B={B} N={N} D={D}", flush=True)
    xd = x.to(DEV)
    res = mpm.run_schedule(xd, insertions=insertions)
    sched = api.Schedule(B, N, D, torch.bfloat16, insertions=insertions)
    out = sched.run(xd)
    torch.cuda.synchronize()
    assert len(res.stages) == insertions
    for b in range(B):
        check_schedule_image(x[b], "bf16", res, b)
    assert torch.equal(out, res.out) and torch.equal(sched.rstar, res.rstar)
    for s in range(insertions):
        assert torch.equal(sched.map[s], res.stages[s].map)
        rows = int(sched.y_off[s][-1])
        assert torch.equal(sched.y[s][:rows], res.stages[s].y[:rows])


def test_deterministic_across_runs():
    rng = np.random.default_rng(4)
    x = torch.stack([store(clustered(rng, 1024, 256, k=30), "bf16") for _ in range(8)]).to(DEV)
    a = mpm.run_schedule(x, insertions=2)
    b = mpm.run_schedule(x, insertions=2)
    torch.cuda.synchronize()
    n_in = torch.full((x.shape[0],), x.shape[1])
    for sa, sb in zip(a.stages, b.stages):
        assert torch.equal(sa.map, sb.map) and torch.equal(sa.y_off, sb.y_off)
        for i, n in enumerate(n_in.tolist()):   # nb is written for the n_b live tokens only
            assert torch.equal(sa.nb[i, :n], sb.nb[i, :n])
        n = int(sa.y_off[-1])
        assert torch.equal(sa.y[:n], sb.y[:n])
        n_in = torch.diff(sa.y_off.cpu())
    assert torch.equal(a.out, b.out)


def test_step_entry_points_equal_merge_and_schedule():
    """The preallocated Schedule (mpm_affinity_compact, then mpm_pair_average) equals
    run_schedule (mpm_merge), bit for bit (ragged stage 2)."""
    from paper_2604_05718_amd import api

    rng = np.random.default_rng(21)
    B, N, D = 9, 600, 192
    x = torch.stack([store(clustered(rng, N, D, k=15, sigma=0.3), "bf16") for _ in range(B)]).to(DEV)
    ref = mpm.run_schedule(x, insertions=2)
    sched = api.Schedule(B, N, D, torch.bfloat16, insertions=2)
    for _ in range(2):  # the second run reuses the buffers
        out = sched.run(x)
    torch.cuda.synchronize()
    assert torch.equal(out, ref.out) and torch.equal(sched.rstar, ref.rstar)
    n_in = [N] * B
    for s in range(2):
        assert torch.equal(sched.map[s], ref.stages[s].map)
        assert torch.equal(sched.y_off[s], ref.stages[s].y_off)
        for b, n in enumerate(n_in):
            assert torch.equal(sched.nb[s][b, :n], ref.stages[s].nb[b, :n])
        rows = int(sched.y_off[s][-1])
        assert torch.equal(sched.y[s][:rows], ref.stages[s].y[:rows])
        n_in = torch.diff(sched.y_off[s].cpu()).tolist()
    # The argmax step entry point agrees with the merge's neighbours.
    nb = mpm.argmax(x)
    assert torch.equal(nb, ref.stages[0].nb)


def test_timed_schedule_equals_untimed():
    """Binding timing events to the affinity dispatches changes no result, and each pair measures a positive kernel duration."""
    from paper_2604_05718_amd import api

    rng = np.random.default_rng(22)
    B, N, D = 9, 600, 192
    x = torch.stack([store(clustered(rng, N, D, k=15, sigma=0.3), "bf16") for _ in range(B)]).to(DEV)
    sched = api.Schedule(B, N, D, torch.bfloat16, insertions=2)
    ref = sched.run(x).clone()
    ref_map = [m.clone() for m in sched.map]
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(2)]
    for e0, e1 in ev:
        e0.record()
        e1.record()
    out = sched.run(x, affinity_events=ev)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    for s in range(2):
        assert torch.equal(sched.map[s], ref_map[s])
        ms = ev[s][0].elapsed_time(ev[s][1])
        assert 0.0 < ms < 1000.0


@pytest.mark.parametrize("window", [None, 2])
def test_graph_replay_matches_eager(window):
    """The schedule (dense, or locality-constrained on a 20-column grid) captured once
    in a HIP graph and replayed several times, with eager kernels touching its outputs
    in between, reproduces the eager results bit for bit on every replay (no memset
    nodes are captured)."""
    from paper_2604_05718_amd import api

    rng = np.random.default_rng(23)
    B, N, D = 9, 600, 192
    x = torch.stack([store(clustered(rng, N, D, k=15, sigma=0.3), "bf16") for _ in range(B)]).to(DEV)
    sched = api.Schedule(B, N, D, torch.bfloat16, insertions=2, grid_w=None if window is None else 20, window=window)
    ref_out = sched.run(x).clone()
    ref_rstar = sched.rstar.clone()
    ref_maps = [m.clone() for m in sched.map]
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sched.run(x)
    for rep in range(4):
        sched.out.zero_()
        sched.rstar.fill_(-7)
        for m in sched.map:
            m.fill_(-9)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(sched.out, ref_out), f"replay {rep}"
        assert torch.equal(sched.rstar, ref_rstar), f"replay {rep}"
        for s in range(2):
            assert torch.equal(sched.map[s], ref_maps[s]), f"replay {rep} stage {s}"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_merge_with_many_candidate_tiles(dtype):
    """N above 1024 gives more than four candidate-tile partials per token, which
    takes the parallel partial reduction before the compaction scan; a packed
    ragged batch (every image a different length) through mpm_merge, checked
    against the oracle stage by stage."""
    rng = np.random.default_rng(41)
    N, D = 1400, 64
    ns = [1400, 1311, 1025, 7]
    rows = [store(clustered(rng, n, D, k=40, sigma=0.3), dtype) for n in ns]
    off = np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)
    x = torch.cat(rows).to(DEV)
    res = mpm.merge(x, torch.from_numpy(off).to(DEV), N=N)
    torch.cuda.synchronize()
    m = res.map.cpu().numpy()
    nb = res.nb.cpu().numpy()
    y = res.y.cpu()
    y_off = res.y_off.cpu().numpy()
    for b, n in enumerate(ns):
        check_stage(to64(rows[b]), dtype, nb[b, :n], m[b], to64(y[y_off[b]:y_off[b + 1]]))


def test_many_items_per_workgroup():
    """More images than workgroup slots (several work items per persistent
    workgroup, full and ragged tiles), checked completely."""
    rng = np.random.default_rng(33)
    B, N, D = 40, 512, 128
    x = torch.stack([store(clustered(rng, N, D, k=25, sigma=0.3), "bf16") for _ in range(B)])
    res = mpm.run_schedule(x.to(DEV), insertions=2)
    torch.cuda.synchronize()
    for b in (0, 7, 8, 23, 39):
        check_schedule_image(x[b], "bf16", res, b)


# ---- symmetric affinity schedule ----------------------------------------------

def _affinity_partials(x2, x_off, B, N, D, dtype, schedule, x_inv=None):
    """Run mpm_affinity under a schedule (with given inverse norms x_inv, if any);
    return the partials (pv, pi) as [B, T, N] host arrays."""
    from paper_2604_05718_amd import _lib
    ws = mpm.affinity(x2, x_off, N=N, x_inv=x_inv, schedule=schedule) if x_off is not None else \
        mpm.affinity(x2.view(B, N, D), x_inv=x_inv, schedule=schedule)
    torch.cuda.synchronize()
    o = _lib.workspace_offsets(B, N)
    T = (N + 63) // 64  # partial slots per token (the workspace layout of include/mpm.h)
    pv = ws[o["pv"]:o["pv"] + 4 * B * T * N].view(torch.float32).view(B, T, N).cpu().numpy()
    pi = ws[o["pi"]:o["pi"] + 4 * B * T * N].view(torch.int32).view(B, T, N).cpu().numpy()
    return pv, pi


def _sym_case(name, dtype):
    """(rows per image, N, D) of the partial-identity cases."""
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    if name == "dense_777":
        return [store(clustered(rng, 777, 128, k=30), dtype) for _ in range(3)], 777, 128
    if name == "rows_192_bytes":  # bf16 rows of 192 bytes: the 64-byte-chunk, four-stage pipeline
        return [store(clustered(rng, 777, 96, k=30), dtype) for _ in range(3)], 777, 96
    if name == "duplicated_rows":  # every token twice: exact ties in both directions
        imgs = []
        for _ in range(2):
            h = clustered(rng, 512, 64, k=20)
            imgs.append(store(np.repeat(h, 2, axis=0), dtype))
        return imgs, 1024, 64
    if name == "all_equal":  # every score equal: the lowest index must win everywhere
        return [store(np.tile(rng.standard_normal((1, 32)), (600, 1)), dtype)], 600, 32
    if name == "packed_ragged":
        ns = [1, 256, 257, 512, 513, 1000, 3, 700]
        return [store(clustered(rng, n, 64, k=25), dtype) for n in ns], 1000, 64
    if name == "deferred_diagonals":
        # 90 images on 8 XCD groups of 32 slots: groups of 12 images (120 blocks) take whole
        # rounds only with a last round of 24; groups of 11 (110 blocks) defer 14 diagonal
        # blocks (all of 3 images', 2 of a fourth) to the half-block second launch.
        return [store(clustered(rng, 1024, 64, k=25), dtype) for _ in range(90)], 1024, 64
    if name == "deferred_packed":
        # 88 ragged images (deferred half blocks past an image's end are skipped), every
        # fourth one made of duplicated rows (exact ties inside the half blocks).
        sizes = [1024, 1000, 769, 768, 513, 256, 1, 900]
        imgs = []
        for b in range(88):
            n = sizes[b % len(sizes)]
            if b % 4 == 3 and n > 1:
                h = clustered(rng, (n + 1) // 2, 64, k=20)
                imgs.append(store(np.repeat(h, 2, axis=0)[:n], dtype))
            else:
                imgs.append(store(clustered(rng, n, 64, k=25), dtype))
        return imgs, 1024, 64
    raise KeyError(name)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name", ["dense_777", "rows_192_bytes", "duplicated_rows", "all_equal", "packed_ragged",
                                  "deferred_diagonals", "deferred_packed"])
def test_symmetric_schedule_partials_bit_identical(dtype, name):
    """The symmetric schedule (blocks on and above the diagonal, each off-diagonal
    block's argmax taken in both directions) must reproduce the full schedule's
    per-tile partials bit for bit on every valid (token, tile) slot, ties
    included; its nearest neighbours must then pass the oracle parity check."""
    rows, N, D = _sym_case(name, dtype)
    ns = [r.shape[0] for r in rows]
    B = len(rows)
    print(f"symmetric partials {name} {dtype} ns={ns} D={D}", flush=True)
    packed = name in ("packed_ragged", "deferred_packed")
    if packed:
        x2 = torch.cat(rows).to(DEV)
        x_off = torch.from_numpy(np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)).to(DEV)
    else:
        x2 = torch.stack(rows).to(DEV).view(B * N, D)
        x_off = None
    out = {mode: _affinity_partials(x2, x_off, B, N, D, dtype, mode) for mode in ("full", "symmetric")}
    (fv, fi), (sv, si) = out["full"], out["symmetric"]
    for b, n in enumerate(ns):
        tiles = (n + 255) // 256
        assert np.array_equal(fv[b, :tiles, :n].view(np.uint32), sv[b, :tiles, :n].view(np.uint32)), b
        assert np.array_equal(fi[b, :tiles, :n], si[b, :tiles, :n]), b
    nb = mpm.argmax(x2 if packed else x2.view(B, N, D), x_off=x_off, N=N if packed else None, schedule="symmetric")
    torch.cuda.synchronize()
    nb = nb.cpu().numpy()
    for b, n in enumerate(ns):
        if n == 1:
            assert nb[b, 0] == -1
            continue
        if name == "all_equal":
            assert nb[b, 0] == 1 and np.all(nb[b, 1:n] == 0)
        check_nearest(to64(rows[b]), nb[b, :n])


@pytest.mark.parametrize("dtype", ["bf16"])
@pytest.mark.parametrize("name", ["dense_777", "rows_192_bytes", "duplicated_rows", "all_equal", "packed_ragged",
                                  "deferred_packed"])
def test_affinity_with_given_norms(dtype, name):
    """mpm_affinity with float64-exact inverse norms (rounded to float32): the
    full and symmetric schedules give bit-identical partials, and the nearest
    neighbours reduced from them (larger score, then smaller index) pass the oracle
    check, ties included."""
    rows, N, D = _sym_case(name, dtype)
    ns = [r.shape[0] for r in rows]
    B = len(rows)
    print(f"given norms {name} {dtype} B={B} D={D}", flush=True)
    packed = name in ("packed_ragged", "deferred_packed")
    if packed:
        x2 = torch.cat(rows).to(DEV)
        x_off = torch.from_numpy(np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)).to(DEV)
        inv = np.concatenate([1.0 / np.maximum(np.sqrt((to64(r) ** 2).sum(axis=1)), 1e-12) for r in rows])
    else:
        x2 = torch.stack(rows).to(DEV).view(B * N, D)
        x_off = None
        inv = np.concatenate([1.0 / np.maximum(np.sqrt((to64(r) ** 2).sum(axis=1)), 1e-12) for r in rows])
    x_inv = torch.from_numpy(inv.astype(np.float32)).to(DEV)
    out = {mode: _affinity_partials(x2, x_off, B, N, D, dtype, mode, x_inv=x_inv) for mode in ("full", "symmetric")}
    (fv, fi), (sv, si) = out["full"], out["symmetric"]
    for b, n in enumerate(ns):
        tiles = (n + 255) // 256
        assert np.array_equal(fv[b, :tiles, :n].view(np.uint32), sv[b, :tiles, :n].view(np.uint32)), b
        assert np.array_equal(fi[b, :tiles, :n], si[b, :tiles, :n]), b
        if n == 1:
            assert fi[b, 0, 0] == -1
            continue
        v, i = sv[b, :tiles, :n], si[b, :tiles, :n]
        best = v.max(axis=0)
        nb = np.where(v == best, i, np.iinfo(np.int32).max).min(axis=0)
        if name == "all_equal":
            assert nb[0] == 1 and np.all(nb[1:n] == 0)
        check_nearest(to64(rows[b]), nb)


@pytest.mark.parametrize("schedule", ["full", "symmetric"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_merge_many_tiles_both_schedules(dtype, schedule):
    """The packed ragged merge with more than four candidate tiles per image,
    with the affinity schedule forced each way."""
    rng = np.random.default_rng(43)
    N, D = 1400, 64
    ns = [1400, 1311, 1025, 257, 7]
    rows = [store(clustered(rng, n, D, k=40, sigma=0.3), dtype) for n in ns]
    off = np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)
    x = torch.cat(rows).to(DEV)
    print(f"merge many tiles {dtype} schedule={schedule}", flush=True)
    res = mpm.merge(x, torch.from_numpy(off).to(DEV), N=N, schedule=schedule)
    torch.cuda.synchronize()
    m = res.map.cpu().numpy()
    nb = res.nb.cpu().numpy()
    y = res.y.cpu()
    y_off = res.y_off.cpu().numpy()
    for b, n in enumerate(ns):
        check_stage(to64(rows[b]), dtype, nb[b, :n], m[b], to64(y[y_off[b]:y_off[b + 1]]))


def _small_block_case(name, dtype):
    """(rows per image, N, D) of the 64 x 64 block cases."""
    rng = np.random.default_rng(zlib.crc32(("small-" + name).encode()))
    if name == "one_image_1024":  # the ViT-Ti shape, scaled down in D
        return [store(clustered(rng, 1024, 64, k=12), dtype)], 1024, 64
    if name == "dense_300":  # ragged last block inside each image
        return [store(clustered(rng, 300, 96, k=10), dtype) for _ in range(2)], 300, 96
    if name == "duplicated_rows":  # exact ties across 64-row blocks
        h = clustered(rng, 100, 64, k=8)
        return [store(np.repeat(h, 2, axis=0), dtype)], 200, 64
    if name == "packed_ragged":
        ns = [1, 64, 65, 130, 500, 2]
        return [store(clustered(rng, n, 64, k=6), dtype) for n in ns], 500, 64
    raise KeyError(name)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name", ["one_image_1024", "dense_300", "duplicated_rows", "packed_ragged"])
def test_small_blocks_equal_full_schedule(dtype, name):
    """The 64 x 64 block schedule (small batches) must give the same nearest
    neighbours and cosines, bit for bit, as the full schedule on 256 x 256
    blocks (every score comes from the same MFMA sums; the lexicographic
    reduction over tiles does not depend on the tile width), and they must pass
    the oracle parity check."""
    rows, N, D = _small_block_case(name, dtype)
    ns = [r.shape[0] for r in rows]
    B = len(rows)
    print(f"small blocks {name} {dtype} ns={ns} D={D}", flush=True)
    packed = name == "packed_ragged"
    if packed:
        x = torch.cat(rows).to(DEV)
        x_off = torch.from_numpy(np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)).to(DEV)
    else:
        x = torch.stack(rows).to(DEV)
        x_off = None
    out = {}
    for mode in ("full", "full_64"):
        assert mpm.affinity_schedule_used(B, N, D, x.dtype, mode) == mode
        nb, best = mpm.argmax(x, x_off=x_off, N=N if packed else None, with_best=True, schedule=mode)
        torch.cuda.synchronize()
        out[mode] = (nb.cpu().numpy(), best.cpu().numpy())
    (fn, fb), (sn, sb) = out["full"], out["full_64"]
    for b, n in enumerate(ns):
        assert np.array_equal(fn[b, :n], sn[b, :n]), b
        assert np.array_equal(fb[b, :n].view(np.uint32), sb[b, :n].view(np.uint32)), b
        if n == 1:
            assert sn[b, 0] == -1
            continue
        check_nearest(to64(rows[b]), sn[b, :n])


def test_small_blocks_chosen_for_small_batches():
    """Auto mode takes the 64 x 64 blocks when a batch has at most 32 blocks of
    256 x 256 (rows a multiple of 64 bytes), and the large blocks otherwise."""
    assert mpm.affinity_schedule_used(1, 1024, 192, torch.float32) == "full_64"
    assert mpm.affinity_schedule_used(2, 1024, 768, torch.bfloat16) == "full_64"
    assert mpm.affinity_schedule_used(3, 1024, 768, torch.bfloat16) != "full_64"
    assert mpm.affinity_schedule_used(1, 4096, 1024, torch.bfloat16) != "full_64"
    assert mpm.affinity_schedule_used(1, 1024, 24, torch.bfloat16) == "full"  # 48-byte rows: no schedule choice
    # The schedule is per call: forcing one for a query changes nothing for the next.
    assert mpm.affinity_schedule_used(64, 1024, 768, torch.bfloat16, "full") == "full"
    assert mpm.affinity_schedule_used(64, 1024, 768, torch.bfloat16) == "symmetric"


# ---- the largest sizes the C ABI accepts -----------------------------------------

@pytest.mark.parametrize("case", ["max_tokens", "max_channels"])
def test_maximum_sizes(case):
    """Two insertions, composition and gather at N = MPM_MAX_N (compaction LDS of
    128 KB, 64 partial tiles per token) and at D = MPM_MAX_D (32 KB rows), checked
    stage by stage and end to end against the oracle."""
    rng = np.random.default_rng(zlib.crc32(case.encode()))
    if case == "max_tokens":
        B, N, D, k = 1, 16384, 64, 200
    else:
        B, N, D, k = 2, 300, 16384, 12
    print(f"maximum sizes {case}: B={B} N={N} D={D} bf16", flush=True)
    x = torch.stack([store(clustered(rng, N, D, k=k, sigma=0.3), "bf16") for _ in range(B)])
    res = mpm.run_schedule(x.to(DEV), insertions=2)
    torch.cuda.synchronize()
    for b in range(B):
        reps = check_schedule_image(x[b], "bf16", res, b)
        print(f"  image {b}: " + ", ".join(f"n={r.n} n'={r.count} flips={r.flipped_rows}" for r in reps), flush=True)


def test_many_images():
    """20000 images of 4 tokens (64-byte rows): every image's merge against the
    oracle, so the per-XCD grouping of the affinity kernel and the one-workgroup-
    per-image kernels run at a batch far beyond the CU count."""
    rng = np.random.default_rng(77)
    B, N, D = 20000, 4, 32
    x64 = rng.standard_normal((B, N, D))
    x = store(x64.reshape(B * N, D), "bf16").view(B, N, D)
    print(f"many images: B={B} N={N} D={D} bf16", flush=True)
    m = mpm.merge(x.to(DEV))
    torch.cuda.synchronize()
    nb = m.nb.cpu().numpy()
    maps = m.map.cpu().numpy()
    y_off = m.y_off.cpu().numpy()
    y = m.y.cpu().to(torch.float64).numpy()
    xs = to64(x)
    for b in range(B):
        check_nearest(xs[b], nb[b], threads=1)  # raises on anything but an accepted near-tie
        ref = oracle.merge(xs[b], "bf16", threads=1, nb=nb[b])
        assert np.array_equal(maps[b], ref.map), b
        assert y_off[b + 1] - y_off[b] == ref.count, b
        assert rel_err(y[y_off[b]:y_off[b + 1]], ref.y) <= 2e-2, b


def test_maximum_images():
    """B = MPM_MAX_B images of 5 tokens (64-byte rows): two insertions (the second on
    ragged packed survivors, with the norms the first wrote), composition and gather,
    every image checked stage by stage and end to end against the oracle. The
    compaction's arrival counter then counts the whole sync region's images, and
    every per-image grid is at its largest."""
    from parity import to_host
    rng = np.random.default_rng(65535)
    B, N, D = 65535, 5, 32
    x = store(rng.standard_normal((B * N, D)), "bf16").view(B, N, D)
    print(f"maximum images: B={B} N={N} D={D} bf16, two insertions", flush=True)
    res = mpm.run_schedule(x.to(DEV), insertions=2)
    torch.cuda.synchronize()
    h = to_host(res)
    flips = 0
    for b in range(B):
        reps = check_schedule_image(x[b], "bf16", h, b, threads=1)
        flips += sum(r.flipped_rows for r in reps)
    print(f"  {B} images checked, {flips} accepted near-tie flips", flush=True)


def test_workspace_sync_region_left_zero():
    """Every call leaves the workspace's arrival counters (the sync region, MPM_MAX_B + 1
    words at its start) zero, so one workspace serves any sequence of calls: dense and
    packed merges, the windowed merge, the fused affinity + compaction step, a batch at
    MPM_MAX_B, and a merge after a smaller one in the same workspace."""
    from paper_2604_05718_amd import _lib
    rng = np.random.default_rng(4)
    sync_words = 65536

    def sync_zero(ws):
        torch.cuda.synchronize()
        off = _lib.workspace_offsets(1, 1)["sync"]
        return int(ws[off:off + 4 * sync_words].view(torch.int32).abs().sum()) == 0

    x = store(rng.standard_normal((9 * 300, 64)), "bf16").view(9, 300, 64).to(DEV)
    ws = mpm.new_workspace(9, 300, DEV)
    assert sync_zero(ws)
    mpm.merge(x, ws=ws)
    assert sync_zero(ws), "dense merge"
    ns = [300, 0, 17, 1, 256, 299, 2, 64, 5]
    off = torch.tensor(np.concatenate([[0], np.cumsum(ns)]), dtype=torch.int32, device=DEV)
    xp = x.view(-1, 64)[: sum(ns)].contiguous()
    mpm.merge(xp, off, N=300, ws=ws, schedule="symmetric")
    assert sync_zero(ws), "packed merge"
    mpm.merge_local(x, 20, 2, ws=ws)
    assert sync_zero(ws), "windowed merge"
    mpm.insertion(x, ws=ws)
    assert sync_zero(ws), "affinity + compaction"
    mpm.merge(x[:3].contiguous(), ws=ws)
    mpm.merge(x, ws=ws)
    assert sync_zero(ws), "smaller batch, then the full one"
    xb = store(rng.standard_normal((65535 * 3, 32)), "bf16").view(65535, 3, 32).to(DEV)
    wsb = mpm.new_workspace(65535, 3, DEV)
    mpm.merge(xb, ws=wsb)
    assert sync_zero(wsb), "MPM_MAX_B images"


def test_concurrent_calls_on_two_streams():
    """Two host threads, each on a stream of its own with its own workspace, merge
    different batches (dense bfloat16 under the symmetric schedule; packed ragged
    float32 under the full one) 20 times each, their launches interleaved on the
    device. Every result equals the same call made alone: the library keeps no state
    between calls beyond the caller's workspace."""
    import threading
    rng = np.random.default_rng(8)
    xa = torch.stack([store(clustered(rng, 1024, 128, k=40), "bf16") for _ in range(16)]).to(DEV)
    ns = [700, 1, 333, 0, 512, 699, 2]
    xb = store(clustered(rng, sum(ns), 64, k=50), "f32").to(DEV)
    offb = torch.tensor(np.concatenate([[0], np.cumsum(ns)]), dtype=torch.int32, device=DEV)
    calls = [lambda ws: mpm.merge(xa, ws=ws, schedule="symmetric"),
             lambda ws: mpm.merge(xb, offb, N=700, ws=ws, schedule="full")]
    want = []
    for call in calls:
        m = call(None)
        torch.cuda.synchronize()
        want.append((m.y_off.clone(), m.map.clone(), m.y[: int(m.y_off[-1])].clone()))
    print("concurrent: two threads, two streams, 20 merges each", flush=True)
    got, errors = [[], []], []

    def worker(t):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                ws = mpm.new_workspace(16, 1024, DEV)
                for _ in range(20):
                    m = calls[t](ws)
                    got[t].append((m.y_off, m.map, m.y))
            s.synchronize()
        except Exception as exc:  # re-raised by the main thread
            errors.append(exc)

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for t in range(2):
        y_off, m, y = want[t]
        assert len(got[t]) == 20
        for k, (go, gm, gy) in enumerate(got[t]):
            assert torch.equal(go, y_off) and torch.equal(gm, m), (t, k)
            assert torch.equal(gy[: y.shape[0]].view(torch.int16 if y.dtype == torch.bfloat16 else torch.int32),
                               y.view(torch.int16 if y.dtype == torch.bfloat16 else torch.int32)), (t, k)


def _random_config(seed):
    """A seeded configuration across the shape space: 1-8 images of up to 1100 tokens
    (dense, or packed with ragged and empty images), rows of 16 bytes to about 2 KB in
    either dtype, any schedule, two insertions."""
    rng = np.random.default_rng(1000 + seed)
    dtype = ["f32", "bf16"][rng.integers(0, 2)]
    unit = 4 if dtype == "f32" else 8
    D = int(unit * rng.integers(1, 1040 // (unit * 2) + 1))
    B = int(rng.integers(1, 9))
    N = int(rng.choice([1, 2, 31, 64, 255, 256, 257, 513, 777, 1024, 1100]))
    packed = bool(rng.integers(0, 2))
    ns = [int(rng.integers(0, N + 1)) if packed and rng.random() < 0.8 else N for _ in range(B)]
    schedule = ["auto", "full", "symmetric", "full_64"][rng.integers(0, 4)]
    return rng, dtype, D, B, N, packed, ns, schedule


@pytest.mark.parametrize("seed", range(64))
def test_random_configurations(seed):
    """64 seeded configurations (_random_config): two insertions, composition and
    gather, every image checked stage by stage against the oracle and through the
    reconstruction."""
    rng, dtype, D, B, N, packed, ns, schedule = _random_config(seed)
    print(f"random config {seed}: {dtype} D={D} B={B} N={N} packed={packed} sizes={ns} schedule={schedule}",
          flush=True)
    imgs = [store(clustered(rng, n, D, k=max(1, n // int(rng.integers(2, 9)))), dtype) for n in ns]
    if packed:
        x = torch.cat(imgs).to(DEV)
        off = torch.tensor(np.concatenate([[0], np.cumsum(ns)]), dtype=torch.int32, device=DEV)
    else:
        x, off = torch.stack(imgs).to(DEV), None
    m1 = mpm.merge(x, off, N=N, schedule=schedule)
    m2 = mpm.merge(m1.y, m1.y_off, N=N, schedule=schedule)
    out, rstar = mpm.compose_unmerge(m2.y, m2.y_off, m1.map, m2.map)
    torch.cuda.synchronize()
    o1, o2 = m1.y_off.cpu().numpy(), m2.y_off.cpu().numpy()
    nb1, nb2 = m1.nb.cpu().numpy(), m2.nb.cpu().numpy()
    map1, map2, rs = m1.map.cpu().numpy(), m2.map.cpu().numpy(), rstar.cpu().numpy()
    y1, y2 = to64(m1.y[: o1[-1]]), to64(m2.y[: o2[-1]])
    up = to64(out)
    for b, n in enumerate(ns):
        if n == 0:
            assert o1[b + 1] == o1[b] and o2[b + 1] == o2[b] and np.all(rs[b] == -1) and not up[b].any(), b
            continue
        s1 = check_stage(to64(imgs[b]), dtype, nb1[b, :n], map1[b], y1[o1[b]:o1[b + 1]])
        check_stage(y1[o1[b]:o1[b + 1]], dtype, nb2[b, :s1.count], map2[b], y2[o2[b]:o2[b + 1]])
        r = oracle.compose(map1[b, :n], map2[b, :s1.count])
        assert np.array_equal(rs[b, :n], r) and np.all(rs[b, n:] == -1), f"image {b}: composed map"
        assert np.array_equal(up[b, :n], oracle.unmerge(y2[o2[b]:o2[b + 1]], r)), f"image {b}: gather"
        assert not up[b, n:].any(), f"image {b}: rows past n_b"


# ---- empty images in a packed batch --------------------------------------------------

_EMPTY_SIZES = [0, 5, 0, 300, 1, 0, 257, 2, 0, 600]
EMPTY_CASES = {  # (D, dtype, schedule, image sizes)
    "persistent_bf16": (64, "bf16", "auto", _EMPTY_SIZES),
    "persistent_bf16_full": (64, "bf16", "full", _EMPTY_SIZES),
    "persistent_bf16_symmetric": (64, "bf16", "symmetric", _EMPTY_SIZES),
    "persistent_f32": (32, "f32", "auto", _EMPTY_SIZES),
    "staged_bf16": (24, "bf16", "auto", _EMPTY_SIZES),                   # 48-byte rows
    "small_blocks": (64, "bf16", "full_64", [0, 700, 0]),
    "symmetric_deferred": (64, "bf16", "symmetric", [0, 1024, 700, 0, 1, 1024] * 15),  # the half-block launch
}


@pytest.mark.parametrize("case", list(EMPTY_CASES))
def test_empty_images(case):
    """Packed batches with empty images (n_b = 0) between ragged ones: two insertions
    (the second on the first's packed output), composition and gather. An empty image
    gets no merged rows, a map of -1 and zero rows from the gather; the others match
    the oracle stage by stage and through the reconstruction."""
    D, dtype, schedule, ns = EMPTY_CASES[case]
    rng = np.random.default_rng(zlib.crc32(("empty-" + case).encode()))
    N = max(ns)
    imgs = [store(clustered(rng, n, D, k=max(1, n // 8)), dtype) for n in ns]
    x = torch.cat(imgs).to(DEV)
    off = torch.tensor(np.concatenate([[0], np.cumsum(ns)]), dtype=torch.int32, device=DEV)
    print(f"empty images {case}: {len(ns)} images, sizes {sorted(set(ns))}, D={D} {dtype} schedule={schedule}",
          flush=True)
    m1 = mpm.merge(x, off, N=N, schedule=schedule)
    m2 = mpm.merge(m1.y, m1.y_off, N=N, schedule=schedule)
    out, rstar = mpm.compose_unmerge(m2.y, m2.y_off, m1.map, m2.map)
    # The step entry points on the same batch: neighbours, then the compaction from them.
    nb_step = mpm.argmax(x, off, N=N, schedule=schedule)
    map_step, src_step, yoff_step = mpm.pair_compact(nb_step, off)
    torch.cuda.synchronize()
    assert torch.equal(yoff_step, m1.y_off)
    for b, n in enumerate(ns):
        assert torch.equal(nb_step[b, :n], m1.nb[b, :n]) and torch.equal(map_step[b], m1.map[b]), f"image {b}"
        c = int(m1.y_off[b + 1] - m1.y_off[b])
        assert torch.equal(src_step[b, :c], m1.src[b, :c]), f"image {b}: sources"
    o1, o2 = m1.y_off.cpu().numpy(), m2.y_off.cpu().numpy()
    nb1, nb2 = m1.nb.cpu().numpy(), m2.nb.cpu().numpy()
    map1, map2, rs = m1.map.cpu().numpy(), m2.map.cpu().numpy(), rstar.cpu().numpy()
    y1, y2 = to64(m1.y[: o1[-1]]), to64(m2.y[: o2[-1]])
    up = to64(out)
    for b, n in enumerate(ns):
        if n == 0:
            assert o1[b + 1] == o1[b] and o2[b + 1] == o2[b], f"image {b}: merged rows of an empty image"
            assert np.all(map1[b] == -1) and np.all(map2[b] == -1) and np.all(rs[b] == -1), f"image {b}: maps"
            assert not up[b].any(), f"image {b}: gather of an empty image"
            continue
        x0 = to64(imgs[b])
        s1 = check_stage(x0, dtype, nb1[b, :n], map1[b], y1[o1[b]:o1[b + 1]])
        n1 = s1.count
        s2 = check_stage(y1[o1[b]:o1[b + 1]], dtype, nb2[b, :n1], map2[b], y2[o2[b]:o2[b + 1]])
        r = oracle.compose(map1[b, :n], map2[b, :n1])
        assert np.array_equal(rs[b, :n], r) and np.all(rs[b, n:] == -1), f"image {b}: composed map"
        assert np.array_equal(up[b, :n], oracle.unmerge(y2[o2[b]:o2[b + 1]], r)), f"image {b}: gather"
        assert not up[b, n:].any(), f"image {b}: rows past n_b"
        assert s2.count <= n1 <= n


# ---- the affinity + compaction step ----------------------------------------------------

def _step_case(name):
    """(rows per image, N, D, dtype, schedule, packed) of the affinity + compaction cases."""
    rng = np.random.default_rng(zlib.crc32(("step-" + name).encode()))
    if name == "symmetric_deferred":  # 90 images: the half-block second launch
        return [store(clustered(rng, 1024, 64, k=25), "bf16") for _ in range(90)], 1024, 64, "bf16", "symmetric", False
    if name == "symmetric_packed":  # ragged images, duplicated rows (exact ties) in every fourth
        sizes = [1024, 1000, 769, 768, 513, 256, 1, 900]
        imgs = []
        for b in range(88):
            n = sizes[b % len(sizes)]
            h = clustered(rng, (n + 1) // 2, 64, k=20) if b % 4 == 3 else clustered(rng, n, 64, k=25)
            imgs.append(store(np.repeat(h, 2, axis=0)[:n] if b % 4 == 3 else h, "bf16"))
        return imgs, 1024, 64, "bf16", "symmetric", True
    if name == "full_f32":
        return [store(clustered(rng, 700, 64, k=20), "f32") for _ in range(20)], 700, 64, "f32", "full", False
    if name == "full_64_one_image":
        return [store(clustered(rng, 1024, 64, k=12), "f32")], 1024, 64, "f32", "full_64", False
    if name == "rows_48_bytes":  # bf16 rows of 48 bytes: the staged kernel (one partial per token)
        return [store(clustered(rng, 300, 24, k=10), "bf16") for _ in range(3)], 300, 24, "bf16", "auto", False
    if name == "rows_192_bytes":  # the 64-byte-chunk ring
        return [store(clustered(rng, 777, 96, k=30), "bf16") for _ in range(12)], 777, 96, "bf16", "symmetric", False
    if name == "many_images":  # 20000 images of 4 tokens: the images-done counter runs to 20000
        return [store(rng.standard_normal((4, 32)), "bf16") for _ in range(20000)], 4, 32, "bf16", "auto", False
    raise KeyError(name)


@pytest.mark.parametrize("name", ["symmetric_deferred", "symmetric_packed", "full_f32", "full_64_one_image",
                                  "rows_48_bytes", "rows_192_bytes", "many_images"])
def test_affinity_compact_equals_argmax_then_compact(name):
    """mpm_affinity_compact (partials reduced inside the compaction kernel, or by the
    parallel reduction for many tiles; the workgroup that finishes the last image turns
    the counts into offsets) gives the same nb, map, src and offsets, bit for bit, as
    mpm_argmax followed by mpm_pair_compact (offsets by a second launch) on the same
    input and schedule; the arrival counters are zero again after the call, and a
    second call on the same workspace repeats the result."""
    from paper_2604_05718_amd import _lib, api

    rows, N, D, dtype, schedule, packed = _step_case(name)
    ns = [r.shape[0] for r in rows]
    B = len(rows)
    print(f"affinity + compaction {name}: B={B} N={N} D={D} {dtype} schedule={schedule}", flush=True)
    if packed:
        x = torch.cat(rows).to(DEV)
        x_off = torch.from_numpy(np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)).to(DEV)
    else:
        x = torch.stack(rows).to(DEV)
        x_off = None
    nb_ref = mpm.argmax(x, x_off=x_off, N=N, schedule=schedule)
    m_ref, src_ref, off_ref = mpm.pair_compact(nb_ref, x_off=x_off)
    ws = api.new_workspace(B, N, DEV)
    x2 = x if packed else x.view(B * N, D)
    got = []
    for rep in range(2):
        m = torch.full((B, N), -9, dtype=torch.int32, device=DEV)
        y_off = torch.full((B + 1,), -9, dtype=torch.int32, device=DEV)
        _lib.check("mpm_affinity_compact", _lib.load().mpm_affinity_compact(
            api._p(x2), api._p(x_off), None, B, N, D, api._dt(x), api._sched(schedule), api._p(m), api._p(y_off),
            api._p(ws), ws.numel(), None, None, api._stream()))
        torch.cuda.synchronize()
        sync = ws[: 4 * 65536].view(torch.int32)
        assert int(torch.count_nonzero(sync)) == 0, f"call {rep}: arrival counters not reset"
        got.append((m.clone(), y_off.clone(), api.ws_view(ws, B, N, "nb").clone(), api.ws_view(ws, B, N, "src").clone()))
    for m, y_off, nb, src in got:
        assert torch.equal(y_off, off_ref)
        assert torch.equal(m, m_ref)
        off = off_ref.cpu().numpy()
        nbh, nbr, srch, srcr = nb.cpu().numpy(), nb_ref.cpu().numpy(), src.cpu().numpy(), src_ref.cpu().numpy()
        for b, n in enumerate(ns):
            assert np.array_equal(nbh[b, :n], nbr[b, :n]), b
            c = off[b + 1] - off[b]
            assert np.array_equal(srch[b, :c], srcr[b, :c]), b
    # The neighbours themselves against the oracle, on a sample of images.
    nbh = got[0][2].cpu().numpy()
    for b in sorted({0, B // 2, B - 1}):
        check_nearest(to64(rows[b]), nbh[b, :ns[b]])
