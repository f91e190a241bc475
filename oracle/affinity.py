"""Oracle (test infrastructure only): token-expert affinities.

Sec. 3.1 and Eq. 2: the score of token t for expert e is the dot product
h_t . w_e of the token representation and the expert embedding; the
assignment maximises the sum of these raw scores (no sigmoid, no softmax).
"""
from __future__ import annotations

import numpy as np


def affinity(H: np.ndarray, W: np.ndarray) -> np.ndarray:
    """S[t, e] = sum_k H[t, k] * W[e, k], computed in fp64.

    H [T x d] and W [E x d] are the exact values the GPU receives (fp32 arrays
    whose entries are bf16- or fp32-representable), so widening to fp64 is
    exact and the only rounding is the fp64 accumulation."""
    H64 = np.asarray(H, dtype=np.float64)
    W64 = np.asarray(W, dtype=np.float64)
    if H64.ndim != 2 or W64.ndim != 2 or H64.shape[1] != W64.shape[1]:
        raise ValueError("H must be [T x d] and W [E x d]")
    return H64 @ W64.T


def affinity_loops(H: np.ndarray, W: np.ndarray) -> np.ndarray:
    """The same definition as three explicit loops (small inputs only): the
    k-ordered fp64 sum, independent of any BLAS."""
    T, d = H.shape
    E = W.shape[0]
    S = np.zeros((T, E), dtype=np.float64)
    for t in range(T):
        for e in range(E):
            acc = 0.0
            for k in range(d):
                acc += float(H[t, k]) * float(W[e, k])
            S[t, e] = acc
    return S
