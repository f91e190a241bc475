"""Oracle (test infrastructure only): the sort vector and the routing permute.

Fig. 2 caption: the assignment is returned as a T-dimensional vector used to
sort tokens by their assigned expert index, after which all_to_all sends row
t of the sorted features to worker floor(t E / T); Sec. 3: the expert output
is afterwards returned to the token's original position. On one device the
routing is the gather into expert-contiguous rows and the inverse scatter.
The order of tokens inside one expert's rows is not fixed by the paper; it is
read as ascending token index (a stable sort).
"""
from __future__ import annotations

import numpy as np


def stable_perm(a: np.ndarray, E: int) -> np.ndarray:
    """perm[k] = the token placed at sorted row k: tokens grouped by expert in
    ascending expert order, ascending token index within an expert. With a
    balanced a, rows [e*C, (e+1)*C) hold exactly expert e's tokens, matching
    the floor(kE/T) routing rule."""
    a = np.asarray(a)
    if a.size and (a.min() < 0 or a.max() >= E):
        raise ValueError("assignment out of range")
    return np.argsort(a, kind="stable").astype(np.int32)


def gather(H: np.ndarray, perm: np.ndarray) -> np.ndarray:
    """X[k] = H[perm[k]]: rows routed into expert-contiguous order."""
    return np.asarray(H)[np.asarray(perm, dtype=np.int64)]


def scatter(X: np.ndarray, perm: np.ndarray) -> np.ndarray:
    """Y[perm[k]] = X[k]: rows returned to their original positions."""
    X = np.asarray(X)
    Y = np.empty_like(X)
    Y[np.asarray(perm, dtype=np.int64)] = X
    return Y
