"""Locality-constrained insertions (Sec. 5: the candidates of a token restricted to a
window on the token grid) through mpm_merge_local, against the oracle with the same
window: the hand-derived grid, random grids of several sizes, windows and ragged
second insertions (positions carried by the merged rows), and the ViT-B and ViT-L
token grids at full batch size, stage by stage with the near-tie rule."""
import numpy as np
import pytest
import torch

import oracle
import paper_2604_05718_amd as mpm
from golden_io import load
from paper_2604_05718_amd import synth
from parity import check_nearest, rel_err, to64, FEATURE_RTOL

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def store(x64, dtype):
    return torch.from_numpy(np.asarray(x64, np.float32)).to(TORCH_DT[dtype])


def check_local_schedule_image(x_img, dtype, res, b, grid_w, window, threads=None):
    """Stage by stage: the GPU's neighbours against the oracle's windowed ones (near-tie
    rule), then maps, merged rows and positions against the oracle seeded with them;
    end to end against the oracle's windowed schedule when nothing flipped."""
    cur = to64(x_img)
    pos = np.arange(cur.shape[0], dtype=np.int32)
    flips, maps = 0, []
    for s, st in enumerate(res.stages):
        n = cur.shape[0]
        nb = st.nb[b].cpu().numpy()[:n]
        # Neighbours: -1 exactly where the window holds no other token.
        nn = oracle.nearest(cur, threads, pos=pos, grid_w=grid_w, window=window)
        empty = nn.nb < 0
        assert np.array_equal(nb[empty], nn.nb[empty]) and np.all(nb[~empty] >= 0), f"stage {s + 1}: empty windows"
        idx = np.flatnonzero(~empty)
        if idx.size:
            # the near-tie check on rows with candidates: compare against the windowed top-1/2
            with np.errstate(invalid="ignore"):
                gap = nn.top1 - nn.top2
            for i in idx[nb[idx] != nn.nb[idx]]:
                j = int(nb[i])
                pi, pj = pos[i], pos[j]
                inside = abs(pi // grid_w - pj // grid_w) <= window and abs(pi % grid_w - pj % grid_w) <= window
                sc = oracle.cosine(cur, int(i), j)
                assert inside and gap[i] < 1e-5 and sc >= nn.top1[i] - 1e-5, f"stage {s + 1} row {i}"
                flips += 1
        ref = oracle.merge(cur, dtype, nb=nb, pos=pos, grid_w=grid_w, window=window)
        m = st.map[b].cpu().numpy()
        assert np.array_equal(m[:n], ref.map) and np.all(m[n:] == -1), f"stage {s + 1}: map"
        off = st.y_off.cpu().numpy()
        y = to64(st.y[off[b]:off[b + 1]])
        assert y.shape[0] == ref.count
        assert rel_err(y, ref.y) <= FEATURE_RTOL[dtype]
        yp = st.y_pos[off[b]:off[b + 1]].cpu().numpy()
        assert np.array_equal(yp, ref.y_pos), f"stage {s + 1}: positions"
        maps.append(m[:n])
        cur, pos = y, yp
    rstar = maps[0]
    for m in maps[1:]:
        rstar = oracle.compose(rstar, m)
    assert np.array_equal(res.rstar[b].cpu().numpy(), rstar)
    assert np.array_equal(to64(res.out[b]), oracle.unmerge(cur, rstar))
    if flips == 0:
        stages, r_ref, up_ref = oracle.schedule(to64(x_img), dtype, insertions=len(res.stages), threads=threads,
                                                grid_w=grid_w, window=window)
        assert np.array_equal(res.rstar[b].cpu().numpy(), r_ref), "end-to-end composed map"
    return flips


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_window_hand_case_on_gpu(dtype):
    g = load("w1_window.txt")
    x = np.zeros((9, 16))
    x[:, :2] = g["x"]
    xt = store(oracle.round_to(x, dtype), dtype)[None].to(DEV)
    res = mpm.merge_local(xt, g["grid_w"], g["window"])
    torch.cuda.synchronize()
    assert res.nb[0].cpu().tolist() == g["nb"]
    assert res.map[0].cpu().tolist() == g["map"]
    assert res.y_off.cpu().tolist() == [0, g["count"]]
    assert res.y_pos[: g["count"]].cpu().tolist() == g["y_pos"]


CASES = [  # (grid rows, grid cols, D, window, images)
    (5, 7, 64, 1, 3), (16, 16, 128, 2, 4), (17, 31, 96, 3, 2), (32, 32, 192, 0, 2), (20, 24, 64, 30, 2),
    (40, 40, 256, 4, 3),
    # rows that are not a whole number of 64 bytes (bf16 80, f32 160): the register-staged kernel
    (12, 9, 40, 2, 2),
    # eight images or more: the persistent kernel's per-XCD image groups
    (24, 24, 64, 3, 9)]


@pytest.mark.parametrize("block_rows", [128, 256])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("gh,gw,D,window,B", CASES)
def test_local_schedule_random_grids(dtype, gh, gw, D, window, B, block_rows):
    """Two windowed insertions on clustered tokens (the second on the ragged packed
    survivors and their carried positions), composition and gather, every image
    checked, with either block size of the persistent kernel (rows that are not a
    whole number of 64 bytes take the register-staged kernel either way); window 0
    leaves every token alone, a window covering the grid is the dense method."""
    rng = np.random.default_rng(gh * 1000 + gw * 10 + window)
    N = gh * gw
    imgs = []
    for _ in range(B):
        cent = rng.standard_normal((12, D))
        lab = rng.integers(0, 12, N)
        imgs.append(store(cent[lab] + 0.3 * rng.standard_normal((N, D)), dtype))
    x = torch.stack(imgs)
    print(f"local schedule {dtype} grid {gh}x{gw} D={D} window={window} B={B} blocks {block_rows}", flush=True)
    res = mpm.run_schedule(x.to(DEV), insertions=2, grid_w=gw, window=window, block_rows=block_rows)
    torch.cuda.synchronize()
    for b in range(B):
        check_local_schedule_image(x[b], dtype, res, b, gw, window)
    if window == 0:
        assert res.stages[0].y_off.cpu().tolist() == [N * k for k in range(B + 1)]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("forced", [False, True])
@pytest.mark.parametrize("name,window,images", [("vit_b_512", 3, [0, 21, 63]), ("vit_l_1024", 4, [0, 9, 15]),
                                                 ("stress_768", 4, [0, 5, 31]), ("vit_s_512", 2, [0, 31]),
                                                 ("vit_ti_512", 2, [0])])
def test_local_schedule_full_size(name, window, images, forced):
    """The windowed schedule on a full benchmark batch (ViT-Ti: one float32 image, a
    single insertion): with the block size the library picks (the launch configuration
    bench.py --window times), every image checked completely; with the other block size
    forced, sampled images."""
    cfg = synth.config(name)
    x = synth.make_batch(cfg, seed=0)
    rows = mpm.local_block_rows(cfg.B, cfg.N, cfg.D, x.dtype, cfg.G, window)
    block_rows = (384 - rows) if forced else 0   # the other of 128 and 256
    if forced:
        rows = block_rows
    else:
        images = range(cfg.B)
    print(f"local schedule {name} window={window}: B={cfg.B} N={cfg.N} D={cfg.D}, {rows}-row blocks"
          f"{' (forced)' if forced else ''}, images checked: {len(images)}", flush=True)
    res = mpm.run_schedule(x.to(DEV), insertions=cfg.insertions, grid_w=cfg.G, window=window, block_rows=block_rows)
    torch.cuda.synchronize()
    flips = sum(check_local_schedule_image(x[b], cfg.dtype, res, b, cfg.G, window) for b in images)
    counts = [torch.diff(st.y_off.cpu()).tolist() for st in res.stages]
    print(f"  survivors (mean): {[round(sum(c) / len(c), 1) for c in counts]}, accepted flips {flips}", flush=True)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("block_rows", [128, 256])
def test_local_schedule_max_size(block_rows):
    """The largest image the ABI accepts (N = 16384, a 128 x 128 grid: 128 or 64 square
    blocks, as many partial slots per token to reduce), window 2, two insertions."""
    rng = np.random.default_rng(16384)
    G, D = 128, 64
    cent = rng.standard_normal((40, D))
    lab = rng.integers(0, 40, G * G)
    x = store(cent[lab] + 0.3 * rng.standard_normal((G * G, D)), "bf16")[None]
    print(f"local schedule max size N={G * G} blocks {block_rows}", flush=True)
    res = mpm.run_schedule(x.to(DEV), insertions=2, grid_w=G, window=2, block_rows=block_rows)
    torch.cuda.synchronize()
    check_local_schedule_image(x[0], "bf16", res, 0, G, 2)


@pytest.mark.parametrize("seed", [1, 2])
@pytest.mark.parametrize("name,window", [("vit_b_512", 3), ("stress_768", 4), ("vit_l_1024", 4)])
def test_local_schedule_other_seeds(name, window, seed):
    """The windowed schedule on full batches drawn with seeds 1 and 2 (the picked block
    size), the first, a middle and the last image checked completely."""
    cfg = synth.config(name)
    x = synth.make_batch(cfg, seed=seed)
    print(f"local schedule {name} window={window} seed={seed}", flush=True)
    res = mpm.run_schedule(x.to(DEV), insertions=cfg.insertions, grid_w=cfg.G, window=window)
    torch.cuda.synchronize()
    for b in sorted({0, cfg.B // 2, cfg.B - 1}):
        check_local_schedule_image(x[b], cfg.dtype, res, b, cfg.G, window)


@pytest.mark.parametrize("block_rows", [128, 256])
@pytest.mark.parametrize("dtype,given_norms", [("f32", False), ("bf16", False), ("bf16", True)])
@pytest.mark.parametrize("given_pos", [False, True])
def test_local_packed_edge_images(dtype, given_norms, given_pos, block_rows):
    """One windowed insertion on packed ragged images: empty, one-token and two-token
    images, images ending inside a grid row and inside a 256-token block, nine images
    (the persistent kernel's per-XCD image groups), positions either each token's index
    or a given increasing subset of the grid (every other cell, as after merges); the
    inverse norms either summed by the kernel or given (float64-exact, rounded to
    float32), and those of the merged rows written."""
    ns = [0, 1, 2, 37, 300, 513, 64, 256, 5]
    grid_w, window, D = 19, 2, 64
    rng = np.random.default_rng(11)
    rows = [rng.standard_normal((n, D)) for n in ns]
    x64 = [oracle.round_to(r, dtype) for r in rows]
    off = np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)
    x = store(np.concatenate(x64), dtype).to(DEV)
    poss = [2 * np.arange(n, dtype=np.int32) + 1 if given_pos else np.arange(n, dtype=np.int32) for n in ns]
    pos = torch.from_numpy(np.concatenate(poss)).to(DEV) if given_pos else None
    xo = torch.from_numpy(off).to(DEV)
    x_inv = None
    if given_norms:
        inv = np.concatenate([1.0 / np.maximum(np.sqrt((r ** 2).sum(axis=1)), 1e-12) for r in x64])
        x_inv = torch.from_numpy(inv.astype(np.float32)).to(DEV)
    print(f"local packed {dtype} given_norms={given_norms} given_pos={given_pos} blocks {block_rows}: images {ns}",
          flush=True)
    res = mpm.merge_local(x, grid_w, window, x_off=xo, N=max(ns), pos=pos, x_inv=x_inv, want_inv=True,
                          block_rows=block_rows)
    torch.cuda.synchronize()
    y_off = res.y_off.cpu().numpy()
    for b, n in enumerate(ns):
        cur, p = x64[b], poss[b]
        nb = res.nb[b].cpu().numpy()[:n]
        if n == 0:
            assert y_off[b + 1] == y_off[b] and np.all(res.map[b].cpu().numpy() == -1), f"image {b}: empty"
            continue
        if n:
            nn = oracle.nearest(cur, pos=p, grid_w=grid_w, window=window)
            empty = nn.nb < 0
            assert np.array_equal(nb[empty], nn.nb[empty]) and np.all(nb[~empty] >= 0), f"image {b}: empty windows"
            with np.errstate(invalid="ignore"):  # rows without candidates: -inf - -inf
                gap = nn.top1 - nn.top2
            for i in np.flatnonzero((nb != nn.nb) & ~empty):
                sc = oracle.cosine(cur, int(i), int(nb[i]))
                assert gap[i] < 1e-5 and sc >= nn.top1[i] - 1e-5, f"image {b} row {i}"
        ref = oracle.merge(cur, dtype, nb=nb, pos=p, grid_w=grid_w, window=window)
        m = res.map[b].cpu().numpy()
        assert np.array_equal(m[:n], ref.map) and np.all(m[n:] == -1), f"image {b}: map"
        assert y_off[b + 1] - y_off[b] == ref.count
        y = to64(res.y[y_off[b]:y_off[b + 1]])
        assert rel_err(y, ref.y) <= FEATURE_RTOL[dtype]
        assert np.array_equal(res.y_pos[y_off[b]:y_off[b + 1]].cpu().numpy(), ref.y_pos), f"image {b}: positions"
        # the merged rows' inverse norms, from their stored values (float32 sums)
        yi = res.y_inv[y_off[b]:y_off[b + 1]].cpu().numpy().astype(np.float64)
        want = 1.0 / np.maximum(np.sqrt((y ** 2).sum(axis=1)), 1e-12)
        assert np.max(np.abs(yi / want - 1.0)) <= 1e-5, f"image {b}: merged inverse norms"


def test_local_block_choice():
    """The block size the library picks for the windowed benchmark workloads on this
    device (an estimate on a full raster grid; 256 CUs): 256-row blocks where a 128-row
    block's band would reach two blocks past its own (ViT-L/16 at 1024 px, window 4),
    128-row blocks elsewhere; a forced size is reported as forced."""
    picks = {}
    for name, window in [("vit_l_1024", 4), ("vit_l_1024", 2), ("vit_b_512", 3), ("stress_768", 4)]:
        cfg = synth.config(name)
        picks[(name, window)] = mpm.local_block_rows(cfg.B, cfg.N, cfg.D, TORCH_DT[cfg.dtype], cfg.G, window)
    print(f"block rows: {picks}", flush=True)
    if torch.cuda.get_device_properties(DEV).multi_processor_count != 256:
        pytest.skip("the picks below are for a 256-CU device")
    assert picks == {("vit_l_1024", 4): 256, ("vit_l_1024", 2): 128, ("vit_b_512", 3): 128, ("stress_768", 4): 128}
    assert mpm.local_block_rows(16, 4096, 1024, torch.bfloat16, 64, 4, block_rows=128) == 128
    assert mpm.local_block_rows(16, 4096, 40, torch.bfloat16, 64, 4) == 4096   # 80-byte rows: the staged kernel
