"""A second, vectorised float64 reading of Alg. 1 in numpy.

TEST INFRASTRUCTURE ONLY: used to cross-check the C oracle on small random
inputs. It follows the algorithm's steps with whole-array operations
(normalise, matmul, masked argmax, gather/compare, cumulative sum,
index-add), where the C oracle uses explicit loops. The two share no code.
"""
from __future__ import annotations

import numpy as np


def mpm_numpy(x: np.ndarray):
    """Returns (nb, map, count, y_exact) for one image; y_exact is the float64
    cluster mean before any storage rounding."""
    x = np.asarray(x, dtype=np.float64)
    n = x.shape[0]
    norms = np.maximum(np.linalg.norm(x, axis=1, keepdims=True), 1e-12)
    xt = x / norms                                   # Alg. 1 step 1
    S = xt @ xt.T                                    # step 2
    np.fill_diagonal(S, -np.inf)
    nb = np.argmax(S, axis=1) if n > 1 else np.full(1, -1)   # step 3 (first maximum)
    idx = np.arange(n)
    mutual = (nb >= 0) & (nb[np.clip(nb, 0, n - 1)] == idx) & (nb != idx)   # step 4
    rep = ~mutual | (idx < nb)                       # step 5
    ids = np.cumsum(rep) - 1                         # step 6: left-to-right scan
    r = np.where(rep, ids, ids[np.clip(nb, 0, n - 1)])
    count = int(rep.sum())
    sums = np.zeros((count, x.shape[1]))
    np.add.at(sums, r, x)                            # step 7
    sizes = np.bincount(r, minlength=count).astype(np.float64)
    return nb.astype(np.int32), r.astype(np.int32), count, sums / sizes[:, None], S
