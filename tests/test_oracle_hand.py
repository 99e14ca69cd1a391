"""Oracle pinned to hand-derived cases (tests/golden/).

Every expected value was derived by hand from the paper's definitions (Eq. 1-4,
Sec. 3.2, Alg. 1), not produced by the oracle.
"""
import os

import numpy as np
import pytest

import oracle
from golden_io import GOLDEN, all_merge_cases, load


@pytest.mark.parametrize("name", all_merge_cases())
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_hand_case_stage1(name, dtype):
    g = load(name)
    x = oracle.round_to(g["x"], dtype)  # store the inputs in the dtype first
    res = oracle.merge(x, dtype)
    assert res.nearest.nb.tolist() == g["nb"]
    assert res.map.tolist() == g["map"]
    assert res.count == g["count"]
    if "clusters" in g:
        got = [[int(a)] if a == b else [int(a), int(b)] for a, b in zip(res.pairs.src_a, res.pairs.src_b)]
        assert got == g["clusters"]
        # Eq. 2: mean of the members, then one rounding to the storage dtype.
        for k, members in enumerate(g["clusters"]):
            want = oracle.round_to(x[members].mean(axis=0), dtype)
            np.testing.assert_array_equal(res.y[k], want)


def test_h4_mean_of_first_pair():
    g = load("h4_all_ties.txt")
    res = oracle.merge(g["x"], "f32")
    want = np.zeros(8)
    want[0] = want[1] = 0.5
    np.testing.assert_array_equal(res.y[0], want)
    for k in range(1, 4):
        np.testing.assert_array_equal(res.y[k], g["x"][k + 1])


def test_h5_unmerge_of_merge_is_identity():
    g = load("h5_dominoes.txt")
    for dtype in ("f32", "bf16"):
        x = oracle.round_to(g["x"], dtype)
        res = oracle.merge(x, dtype)
        np.testing.assert_array_equal(oracle.unmerge(res.y, res.map), x)


def test_h6_two_insertions_compose_and_reconstruct():
    g = load("h6_blocks.txt")
    blocks = g["blocks"]
    stages, rstar, x_up = oracle.schedule(g["x"], "f32", insertions=2)
    s1, s2 = stages
    assert s1.nearest.nb.tolist() == g["nb"]
    assert s1.map.tolist() == g["map"] and s1.count == g["count"]
    np.testing.assert_array_equal(s1.y, np.stack([blocks[c] for c in g["stage1_rows"]]))
    assert s2.nearest.nb.tolist() == g["nb2"]
    assert s2.map.tolist() == g["map2"] and s2.count == g["count2"]
    np.testing.assert_array_equal(s2.y, np.stack([blocks[c] for c in g["stage2_rows"]]))
    assert rstar.tolist() == g["rstar"]
    np.testing.assert_array_equal(x_up, g["x"])


def test_compose_small():
    g = load("compose_small.txt")
    assert oracle.compose(g["r1"], g["r2"]).tolist() == g["rstar"]


def test_h7_raw_dot_would_pair_differently():
    """Guards the normalisation: the raw dot product prefers (1,2), the cosine (0,2)."""
    g = load("h7_norms.txt")
    x = g["x"]
    raw = x @ x.T
    np.fill_diagonal(raw, -np.inf)
    assert np.argmax(raw, axis=1).tolist() == [1, 2, 1]
    assert oracle.merge(x, "f32").nearest.nb.tolist() == g["nb"]


def test_single_token_and_pair():
    x1 = np.array([[1.0, 2.0, 3.0, 4.0]])
    r = oracle.merge(x1, "f32")
    assert r.nearest.nb.tolist() == [-1] and r.map.tolist() == [0] and r.count == 1
    np.testing.assert_array_equal(r.y, x1)
    # Any two tokens are each other's only candidate: they always pair.
    rng = np.random.default_rng(7)
    for _ in range(20):
        x2 = rng.standard_normal((2, 6))
        r = oracle.merge(x2, "f32")
        assert r.nearest.nb.tolist() == [1, 0] and r.map.tolist() == [0, 0] and r.count == 1


def test_zero_token_goes_to_lowest_index():
    """A zero row has cosine 0 with everything (norm clamped at 1e-12)."""
    x = np.array([[1.0, 0.0], [0.0, 0.0], [0.5, 0.5], [-1.0, 0.2]])
    nn = oracle.nearest(x)
    assert nn.nb[1] == 0
    assert oracle.cosine(x, 1, 2) == 0.0


def _unit(deg):
    t = np.deg2rad(np.asarray(deg, dtype=np.float64))
    return np.stack([np.cos(t), np.sin(t)], axis=1)


def _top2_cases():
    vals = {}
    with open(os.path.join(GOLDEN, "top2_gap.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                k, _, v = line.partition(":")
                vals[k.strip()] = [float(t) for t in v.split()]
    return vals


def test_top1_top2_hand_derived():
    """The oracle's top-1 and top-2 cosines per row (the near-tie gap of the parity
    protocol) against values derived by hand from angles: distinct maxima, a maximum
    attained by every other row, a maximum attained twice or more, and a single
    candidate (no second value). A wrong update on an equal maximum, a second value
    left at -inf, or the maximum counted twice would fail one of them."""
    c = _top2_cases()
    for key in ("a", "c"):
        nn = oracle.nearest(_unit(c[f"{key}_angles_deg"]))
        np.testing.assert_allclose(nn.top1, np.cos(np.deg2rad(c[f"{key}_top1_deg"])), rtol=0, atol=1e-12)
        np.testing.assert_allclose(nn.top2, np.cos(np.deg2rad(c[f"{key}_top2_deg"])), rtol=0, atol=1e-12)
    n, d = (int(v) for v in c["b_onehot"])
    nn = oracle.nearest(np.eye(n, d))
    assert np.all(nn.top1 == 0.0) and np.all(nn.top2 == 0.0) and np.all(nn.gap == 0.0)
    nn = oracle.nearest(_unit(c["d_angles_deg"]))
    np.testing.assert_allclose(nn.top1, np.cos(np.deg2rad(c["d_top1_deg"])), rtol=0, atol=1e-12)
    assert np.all(np.isneginf(nn.top2))
    nn = oracle.nearest(_unit([30.0]))  # one token: no candidate at all
    assert nn.nb[0] == -1 and np.isneginf(nn.top1[0]) and np.isneginf(nn.top2[0])


def test_window_hand_case():
    """The locality-constrained neighbour (Sec. 5) on a hand-derived 3x3 grid: every
    neighbour, pair, id, cluster and merged position, and the dense choice the window
    rules out."""
    g = load("w1_window.txt")
    x = g["x"]
    for dtype in ("f32", "bf16"):
        xs = oracle.round_to(x, dtype)
        res = oracle.merge(xs, dtype, grid_w=g["grid_w"], window=g["window"])
        assert res.nearest.nb.tolist() == g["nb"]
        assert res.map.tolist() == g["map"]
        assert res.count == g["count"]
        assert res.y_pos.tolist() == g["y_pos"]
        for k, members in enumerate(g["clusters"]):
            np.testing.assert_array_equal(res.y[k], oracle.round_to(xs[members].mean(axis=0), dtype))
    dense = oracle.nearest(x)
    assert dense.nb[0] == g["dense_nb0"] and dense.nb[8] == g["dense_nb8"]
