"""Oracle pinned to properties the paper and the mathematics fix.

* Invariants of the pairing (Sec. 3.2, Alg. 1): each token in at most one
  cluster, every pair mutual with the lower index as representative,
  N' = N - |P|, ceil(N/2) <= N' <= N - 1, ids onto [0, N') in scan order.
* Eq. 2 preserves the token sum (before rounding).
* Eq. 3 equals two sequential gathers and is associative; Eq. 4 is a copy.
* The affinity is a cosine: invariant to positive row scaling, agrees with a
  library normalised matmul; the argmax is the lowest index attaining the max.
* Exhaustive: every symmetric affinity with off-diagonal entries in {0,1,2} for
  N <= 4 (all tie patterns).
* Closed form: images made of exact duplicated 2x2 patches give N1 = 3N/4,
  N2 = N/2 and exact reconstruction.
* Storage rounding agrees with torch's float32 -> bfloat16 conversion and with
  hand-checked ties.
"""
import itertools

import numpy as np
import pytest
import torch
from hypothesis import assume, given, settings, strategies as st
from hypothesis.extra.numpy import arrays

import oracle
from oracle.ref_numpy import mpm_numpy


def check_pairing_invariants(nb, pr, n):
    m, a, b = pr.map, pr.src_a, pr.src_b
    npairs = int((a != b).sum())
    # I1: every token in exactly one cluster.
    members = np.concatenate([a, b[a != b]])
    assert sorted(members.tolist()) == list(range(n))
    # I2: every pair mutual, representative is the lower index.
    for i, j in zip(a, b):
        if i != j:
            assert i < j and nb[i] == j and nb[j] == i
    # Singletons are exactly the tokens without a reciprocal choice.
    for i in a[a == b]:
        assert nb[i] < 0 or nb[nb[i]] != i
    # I3, I4
    assert pr.count == n - npairs
    if n >= 2:
        assert (n + 1) // 2 <= pr.count <= n - 1
    else:
        assert pr.count == 1
    # I5: ids onto [0, N'), increasing over representatives in index order, partners inherit.
    assert m[0] == 0
    assert sorted(set(m.tolist())) == list(range(pr.count))
    assert np.all(np.diff(a) > 0)
    for k, (i, j) in enumerate(zip(a, b)):
        assert m[i] == k and m[j] == k


def check_argmax_definition(S, nb):
    n = S.shape[0]
    for i in range(n):
        vals = [S[i, j] for j in range(n) if j != i]
        if not vals:
            assert nb[i] == -1
            continue
        top = max(vals)
        assert S[i, nb[i]] == top and nb[i] != i
        assert all(S[i, j] < top for j in range(nb[i]) if j != i)  # lowest index wins


tokens = st.integers(1, 40).flatmap(
    lambda n: st.integers(1, 12).flatmap(
        lambda d: arrays(np.float64, (n, d), elements=st.floats(-4, 4, allow_nan=False, width=32))))


@settings(max_examples=300, deadline=None)
@given(tokens)
def test_invariants_random(x):
    n = x.shape[0]
    nn = oracle.nearest(x)
    pr = oracle.pairs(nn.nb)
    check_pairing_invariants(nn.nb, pr, n)
    # top1 is attained by nb and is the maximum cosine of the row.
    for i in range(n if n > 1 else 0):
        assert oracle.cosine(x, i, int(nn.nb[i])) == nn.top1[i]
        assert nn.top1[i] >= nn.top2[i]
    # I7: Eq. 2 preserves the sum of tokens (exact float64 means, no rounding).
    sums = np.zeros((pr.count, x.shape[1]))
    for k, (i, j) in enumerate(zip(pr.src_a, pr.src_b)):
        sums[k] = x[i] if i == j else x[i] + x[j]
    np.testing.assert_allclose(sums.sum(0), x.sum(0), rtol=1e-12, atol=1e-12)


@settings(max_examples=200, deadline=None)
@given(tokens, st.integers(0, 2**31 - 1))
def test_cosine_is_scale_invariant(x, seed):
    """Multiplying rows by positive powers of two does not move any nearest neighbour
    (the scaling is exact, so even ties are kept), as long as no norm is clamped."""
    norms = np.linalg.norm(x, axis=1)
    assume(np.all((norms == 0) | (norms > 1e-3)))
    rng = np.random.default_rng(seed)
    scale = 2.0 ** rng.integers(-6, 7, size=(x.shape[0], 1))
    a = oracle.nearest(x).nb
    b = oracle.nearest(x * scale).nb
    assert a.tolist() == b.tolist()


def test_cosine_matches_library_normalised_matmul():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((50, 33)) * rng.uniform(0.1, 10, size=(50, 1))
    xt = x / np.linalg.norm(x, axis=1, keepdims=True)
    S = xt @ xt.T
    for i, j in [(0, 1), (3, 17), (49, 2), (10, 11)]:
        assert abs(oracle.cosine(x, i, j) - S[i, j]) < 1e-14
    nn = oracle.nearest(x)
    np.fill_diagonal(S, -np.inf)
    # No near ties in Gaussian data at this size: the library argmax agrees.
    assert (np.sort(S, 1)[:, -1] - np.sort(S, 1)[:, -2]).min() > 1e-9
    assert nn.nb.tolist() == np.argmax(S, 1).tolist()
    np.testing.assert_allclose(nn.top1, S.max(1), rtol=0, atol=1e-14)


@settings(max_examples=10_000, deadline=None)
@given(tokens)
def test_agrees_with_vectorised_numpy_reading(x):
    """The C oracle and the vectorised numpy reading agree on 10^4 random tiny inputs."""
    n = x.shape[0]
    nb, m, count, y_exact, S = mpm_numpy(x)
    nn = oracle.nearest(x)
    # Rows whose top two cosines are within rounding of each other may differ
    # between the loop and the matmul; the rest must agree exactly.
    if n > 1:
        srt = np.sort(S, axis=1)
        if (srt[:, -1] - srt[:, -2]).min() < 1e-12:
            return
    assert nn.nb.tolist() == nb.tolist()
    res = oracle.merge(x, "f32")
    assert res.map.tolist() == m.tolist() and res.count == count
    np.testing.assert_array_equal(res.y, oracle.round_to(y_exact, "f32"))


def _exhaustive_affinities(n):
    iu = [(i, j) for i in range(n) for j in range(i + 1, n)]
    for vals in itertools.product((0.0, 1.0, 2.0), repeat=len(iu)):
        S = np.zeros((n, n))
        for (i, j), v in zip(iu, vals):
            S[i, j] = S[j, i] = v
        yield S


@pytest.mark.parametrize("n", [1, 2, 3, 4])
def test_exhaustive_small_affinities(n):
    count = 0
    for S in _exhaustive_affinities(n):
        nb = oracle.nearest_from_affinity(S)
        check_argmax_definition(S, nb)
        pr = oracle.pairs(nb)
        check_pairing_invariants(nb, pr, n)
        count += 1
    assert count == 3 ** (n * (n - 1) // 2)


def test_exhaustive_n5_sampled_with_ties():
    rng = np.random.default_rng(3)
    for _ in range(2000):
        v = rng.integers(0, 3, size=10).astype(float)
        S = np.zeros((5, 5))
        S[np.triu_indices(5, 1)] = v
        S = S + S.T
        nb = oracle.nearest_from_affinity(S)
        check_argmax_definition(S, nb)
        check_pairing_invariants(nb, oracle.pairs(nb), 5)


@settings(max_examples=100, deadline=None)
@given(st.integers(1, 30), st.integers(1, 30), st.integers(0, 2**31 - 1))
def test_compose_is_sequential_gather_and_associative(n1, extra, seed):
    rng = np.random.default_rng(seed)
    # Random onto maps n0 -> n1 -> n2 -> n3, shaped like merge maps.
    def onto(n_from, n_to):
        m = np.concatenate([np.arange(n_to), rng.integers(0, n_to, n_from - n_to)])
        return rng.permutation(m).astype(np.int32)
    n0 = n1 + extra
    n2 = max(1, n1 // 2)
    n3 = max(1, n2 // 2)
    r1, r2, r3 = onto(n0, n1), onto(n1, n2), onto(n2, n3)
    z = rng.standard_normal((n2, 5))
    rstar = oracle.compose(r1, r2)
    # I6: gather through r* equals two sequential gathers.
    np.testing.assert_array_equal(oracle.unmerge(z, rstar), oracle.unmerge(oracle.unmerge(z, r2), r1))
    assert oracle.compose(oracle.compose(r1, r2), r3).tolist() == oracle.compose(r1, oracle.compose(r2, r3)).tolist()


def test_duplicated_patch_closed_form():
    """Exact duplicated 2x2 patches: within each patch all cosines equal 1 and the
    lowest-index rule pairs only the top row at stage 1 (N1 = 3N/4), and one pair
    per patch at stage 2 (N2 = N/2); gathering back reproduces the input."""
    G, D = 8, 16
    rng = np.random.default_rng(11)
    base = rng.standard_normal((G // 2, G // 2, D))
    x = np.repeat(np.repeat(base, 2, 0), 2, 1).reshape(G * G, D)
    for dtype in ("f32", "bf16"):
        xs = oracle.round_to(x, dtype)
        stages, rstar, x_up = oracle.schedule(xs, dtype, insertions=2)
        assert stages[0].count == 3 * G * G // 4
        assert stages[1].count == G * G // 2
        np.testing.assert_array_equal(x_up, xs)


@settings(max_examples=50, deadline=None)
@given(st.integers(2, 30), st.integers(0, 2**31 - 1))
def test_pair_set_permutation_equivariant(n, seed):
    """I9: relabelling tokens relabels the pair set (no ties in Gaussian data)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, 8))
    perm = rng.permutation(n)
    p1 = oracle.pairs(oracle.nearest(x).nb)
    p2 = oracle.pairs(oracle.nearest(x[perm]).nb)
    set1 = {frozenset((int(a), int(b))) for a, b in zip(p1.src_a, p1.src_b) if a != b}
    set2 = {frozenset((int(perm[a]), int(perm[b]))) for a, b in zip(p2.src_a, p2.src_b) if a != b}
    assert set1 == set2


def test_round_to_bf16_matches_torch_on_float32_values():
    rng = np.random.default_rng(5)
    v32 = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-38).astype(np.float32),   # subnormal range
        (rng.standard_normal(2000) * 1e38).astype(np.float32),
        np.array([3.3895314e38, 3.40282e38, -3.40282e38, 0.0, -0.0], np.float32),
    ])
    want = torch.from_numpy(v32).to(torch.bfloat16).to(torch.float64).numpy()
    got = oracle.round_to(v32.astype(np.float64), "bf16")
    np.testing.assert_array_equal(got, want)


def test_round_to_hand_ties():
    # bfloat16 spacing at 1 is 2^-7.
    cases = {
        1 + 2**-8: 1.0,                        # halfway, even neighbour is 1.0
        1 + 3 * 2**-8: 1 + 2**-6,              # halfway, even neighbour is above
        1 + 2**-8 + 2**-30: 1 + 2**-7,         # just above halfway (not a float32 value)
        -(1 + 3 * 2**-8): -(1 + 2**-6),
        2.0**-133 * 1.5: 2.0**-132,            # smallest subnormal spacing
    }
    got = oracle.round_to(np.array(list(cases)), "bf16")
    np.testing.assert_array_equal(got, np.array(list(cases.values())))
    # float32: C conversion rounds to nearest even.
    assert oracle.round_to(np.array([1 + 2**-24]), "f32")[0] == 1.0
    assert oracle.round_to(np.array([1 + 3 * 2**-24]), "f32")[0] == 1 + 2**-22


# ---- the locality constraint (Sec. 5) ---------------------------------------------------

def _grid_tokens(rng, gh, gw, D, k=4):
    cent = rng.standard_normal((k, D))
    lab = rng.integers(0, k, gh * gw)
    return cent[lab] + 0.3 * rng.standard_normal((gh * gw, D))


@pytest.mark.parametrize("seed", range(12))
def test_window_covering_the_grid_is_the_dense_definition(seed):
    """A window at least as wide as the grid admits every other token: exactly the
    dense oracle (neighbours and both top values)."""
    rng = np.random.default_rng(seed)
    gh, gw = int(rng.integers(1, 7)), int(rng.integers(1, 7))
    x = _grid_tokens(rng, gh, gw, 5)
    dense = oracle.nearest(x)
    win = oracle.nearest(x, grid_w=gw, window=max(gh, gw) - 1 + int(rng.integers(0, 3)))
    assert np.array_equal(win.nb, dense.nb)
    assert np.array_equal(win.top1, dense.top1) and np.array_equal(win.top2, dense.top2)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_window_zero_leaves_every_token_alone(dtype):
    """Radius 0 admits no other token: every token is a singleton, the merge is the
    identity (N' = N, r(i) = i, rows copied), positions unchanged."""
    rng = np.random.default_rng(7)
    x = oracle.round_to(_grid_tokens(rng, 5, 6, 8), dtype)
    res = oracle.merge(x, dtype, grid_w=6, window=0)
    assert np.all(res.nearest.nb == -1) and np.all(np.isneginf(res.nearest.top1))
    assert res.count == 30 and res.map.tolist() == list(range(30))
    assert np.array_equal(res.y, x) and res.y_pos.tolist() == list(range(30))


@settings(max_examples=200, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), gh=st.integers(1, 6), gw=st.integers(1, 6), window=st.integers(0, 3),
       D=st.integers(1, 6))
def test_window_choice_is_the_best_inside_the_window(seed, gh, gw, window, D):
    """Every windowed neighbour lies inside the window and attains the largest cosine
    there (lowest index among equals); a row whose dense neighbour lies inside the
    window keeps it; the window never raises a row's best score."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((gh * gw, D)).round(1)  # rounding makes exact ties common
    n = gh * gw
    win = oracle.nearest(x, grid_w=gw, window=window)
    dense = oracle.nearest(x)
    for i in range(n):
        cand = [j for j in range(n) if j != i and abs(j // gw - i // gw) <= window and abs(j % gw - i % gw) <= window]
        if not cand:
            assert win.nb[i] == -1
            continue
        s = np.array([oracle.cosine(x, i, j) for j in cand])
        assert win.nb[i] == cand[int(np.flatnonzero(s == s.max())[0])]
        assert win.top1[i] == s.max() <= dense.top1[i]
        if dense.nb[i] in cand:
            assert win.nb[i] == dense.nb[i]


@pytest.mark.parametrize("seed", range(6))
def test_window_schedule_positions(seed):
    """Over two insertions the merged tokens keep their representatives' cells: each
    stage's positions are a strictly increasing (raster-order) subset of the
    previous stage's, and every cluster's members lie within the window of its
    representative; the pairing invariants hold (except N' <= N - 1: a window may
    leave a token without candidates)."""
    rng = np.random.default_rng(100 + seed)
    gh, gw, window = 6, 7, int(rng.integers(1, 3))
    x = _grid_tokens(rng, gh, gw, 6)
    stages, rstar, up = oracle.schedule(x, "f32", insertions=2, grid_w=gw, window=window)
    pos = np.arange(gh * gw)
    for stg in stages:
        assert np.all(np.diff(stg.y_pos) > 0) and set(stg.y_pos.tolist()) <= set(pos.tolist())
        for a, b in zip(stg.pairs.src_a, stg.pairs.src_b):
            pa, pb = pos[a], pos[b]
            assert abs(pa // gw - pb // gw) <= window and abs(pa % gw - pb % gw) <= window
        n = pos.shape[0]
        assert (n + 1) // 2 <= stg.count <= n
        pos = stg.y_pos
    assert np.array_equal(up, oracle.unmerge(stages[-1].y, rstar))
