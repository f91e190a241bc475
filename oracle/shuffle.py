"""Oracle (test infrastructure only): routing with the random shuffle of
tokens to workers and the sharded, per-worker solve.

Sec. 3.2.1 (Sharding): the assignment over all workers' tokens is split into
independent problems, one per worker, each balancing its own T tokens over
the E experts. Sec. 3.2.1 (Shuffling): before that, tokens are sent to
workers at random, so that a worker's batch is a random sample rather than
consecutive text. With B workers of T tokens and a random permutation
`shuffle` of the B T tokens, worker b receives tokens shuffle[bT .. bT+T-1];
its token j is original token shuffle[bT + j].

The steps, in the paper's order:
  1. shuffle:  H_w[i] = H[shuffle[i]]                      (gather)
  2. per worker b: S_b = affinity of its rows (Sec. 3.1), a_b = the
     balanced optimum of Eq. 2, perm_b = its sort vector (Fig. 2 caption),
     X_b = its rows in expert order
  3. return: the expert outputs go back to the worker token order (scatter
     by perm_b), then to the original token order (scatter by shuffle).
Everything is fp64 and exact; the solver is the oracle's exact one.
"""
from __future__ import annotations

import numpy as np

from .affinity import affinity
from .assign import solve_ssp
from .gate import gate_combine
from .permute import gather, scatter, stable_perm


def route_shuffled(H, W, shuffle, B: int):
    """Steps 1-2. Returns (S [B*T, E] in worker order, a [B, T], perm [B, T],
    X [B*T, d] in each worker's expert order)."""
    H = np.asarray(H)
    shuffle = np.asarray(shuffle, dtype=np.int64)
    N = H.shape[0]
    if shuffle.shape != (N,) or N % B:
        raise ValueError("shuffle must index all B*T rows")
    T = N // B
    Hw = gather(H, shuffle)
    S = affinity(Hw, W)
    E = S.shape[1]
    a = np.empty((B, T), dtype=np.int32)
    perm = np.empty((B, T), dtype=np.int32)
    X = np.empty_like(Hw)
    for b in range(B):
        rows = slice(b * T, (b + 1) * T)
        a_b, _, _ = solve_ssp(S[rows])
        a[b] = a_b
        perm[b] = stable_perm(a_b, E)
        X[rows] = gather(Hw[rows], perm[b])
    return S, a, perm, X


def unroute_shuffled(Y, perm, shuffle):
    """Step 3: Y [B*T, d] in each worker's expert order back to the original
    token order."""
    Y = np.asarray(Y)
    perm = np.asarray(perm)
    B, T = perm.shape
    Yw = np.empty_like(Y)
    for b in range(B):
        rows = slice(b * T, (b + 1) * T)
        Yw[rows] = scatter(Y[rows], perm[b])
    return scatter(Yw, np.asarray(shuffle, dtype=np.int64))


def gate_combine_shuffled(F, H, S, a, perm, shuffle):
    """Eq. 1 for every worker, returned in the original token order: worker
    b's token j (original token shuffle[bT + j]) gets
    sigmoid(S[bT + j, a[b, j]]) f + h, with f its row of F (worker b's
    expert order) and h its row of H."""
    F = np.asarray(F)
    perm = np.asarray(perm)
    B, T = perm.shape
    shuffle = np.asarray(shuffle, dtype=np.int64)
    Hw = gather(np.asarray(H), shuffle)
    S = np.asarray(S)
    Yw = np.empty(Hw.shape, dtype=np.float64)
    for b in range(B):
        rows = slice(b * T, (b + 1) * T)
        Yw[rows] = gate_combine(F[rows], Hw[rows], S[rows], a[b], perm[b])
    return scatter(Yw, shuffle)
