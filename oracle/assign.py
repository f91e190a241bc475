"""Oracle (test infrastructure only): the balanced token-to-expert assignment.

Sec. 3.2.1, Eq. 2: given scores S[t, e] = h_t . w_e for T tokens and E
experts, choose a_t in [0, E) to maximise sum_t S[t, a_t] subject to every
expert receiving exactly T/E tokens. The paper writes the index ranges as
"0..E" and "t = 0..T"; they are read as half-open ([0, E), [0, T)), and T/E
must be an integer.

Three independent exact solvers (brute force, Hungarian on the replicated
matrix, compact successive shortest paths) plus the certificates the tests
use to pin them: the LP-duality bound, the greedy (test-time) upper bound of
Sec. 3.2.2, and the second-best gap that decides uniqueness.
"""
from __future__ import annotations

import ctypes
import itertools
import math

import numpy as np

from . import build as _build

_lib = None


def _native():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(_build.ensure_built())
        lib.oracle_hungarian.argtypes = [
            ctypes.c_int64,
            ctypes.c_void_p,
            ctypes.c_void_p,
            ctypes.c_void_p,
            ctypes.c_void_p,
        ]
        lib.oracle_hungarian.restype = ctypes.c_int
        lib.oracle_ssp_solve.argtypes = [
            ctypes.c_int64,
            ctypes.c_int64,
            ctypes.c_void_p,
            ctypes.c_void_p,
            ctypes.c_void_p,
        ]
        lib.oracle_ssp_solve.restype = ctypes.c_int
        _lib = lib
    return _lib


def _check_shape(S: np.ndarray) -> tuple[int, int, int]:
    if S.ndim != 2:
        raise ValueError("S must be [T x E]")
    T, E = S.shape
    if T <= 0 or E <= 0 or T % E:
        raise ValueError("T must be a positive multiple of E (Eq. 2 needs T/E tokens per expert)")
    return T, E, T // E


def objective(S: np.ndarray, a: np.ndarray) -> float:
    """sum_t S[t, a_t] in fp64 (Eq. 2's objective)."""
    S = np.asarray(S, dtype=np.float64)
    return float(S[np.arange(S.shape[0]), np.asarray(a, dtype=np.int64)].sum())


def balanced_counts_ok(a: np.ndarray, E: int) -> bool:
    """Eq. 2's constraint: every expert receives exactly T/E tokens, and every
    token is assigned to a valid expert exactly once."""
    a = np.asarray(a)
    T = a.shape[0]
    if T % E or a.min(initial=0) < 0 or a.max(initial=0) >= E:
        return False
    return bool(np.all(np.bincount(a, minlength=E) == T // E))


def solve_bruteforce(S: np.ndarray):
    """Enumerate every balanced assignment (T!/((T/E)!)^E of them; tiny T only).

    Returns (best objective, list of every optimal assignment as int arrays).
    Objectives are compared exactly in fp64; for integer-valued S the sums
    are exact, so the list is exactly the set of optima."""
    S = np.asarray(S, dtype=np.float64)
    T, E, C = _check_shape(S)
    if math.factorial(T) // math.factorial(C) ** E > 2_000_000:
        raise ValueError("too many balanced assignments to enumerate")
    best = -math.inf
    winners: list[tuple[int, ...]] = []
    room = [C] * E
    cur = [0] * T

    def rec(t: int, acc: float):
        nonlocal best, winners
        if t == T:
            if acc > best:
                best, winners = acc, [tuple(cur)]
            elif acc == best:
                winners.append(tuple(cur))
            return
        for e in range(E):
            if room[e]:
                room[e] -= 1
                cur[t] = e
                rec(t + 1, acc + S[t, e])
                room[e] += 1

    rec(0, 0.0)
    return best, [np.array(w, dtype=np.int32) for w in winners]


def count_balanced(T: int, E: int) -> int:
    """Number of balanced assignments, T! / ((T/E)!)^E."""
    C = T // E
    return math.factorial(T) // math.factorial(C) ** E


def replicated_cost(S: np.ndarray) -> np.ndarray:
    """Cost matrix of the square assignment problem equivalent to Eq. 2:
    expert e is replicated into T/E identical columns e*C .. e*C + C - 1,
    and cost[t, e*C + j] = -S[t, e]."""
    S = np.asarray(S, dtype=np.float64)
    T, E, C = _check_shape(S)
    return np.repeat(-S, C, axis=1)


def solve_hungarian(S: np.ndarray):
    """Exact optimum of Eq. 2 by the O(T^3) Hungarian method on the replicated
    T x T matrix (moderate T only). Returns (assignment int32 [T], objective)."""
    S = np.asarray(S, dtype=np.float64)
    T, E, C = _check_shape(S)
    cost = np.ascontiguousarray(replicated_cost(S))
    cols = np.empty(T, dtype=np.int64)
    rc = _native().oracle_hungarian(T, cost.ctypes.data, cols.ctypes.data, None, None)
    if rc != 0:
        raise RuntimeError(f"oracle_hungarian failed ({rc})")
    a = (cols // C).astype(np.int32)
    return a, objective(S, a)


def solve_ssp(S: np.ndarray):
    """Exact optimum of Eq. 2 by successive shortest paths on the E expert
    nodes (any size). Returns (assignment int32 [T], objective, prices fp64 [E])
    where the prices satisfy dual_bound(S, prices) == objective up to fp64
    rounding (exactly for integer-valued S)."""
    S = np.ascontiguousarray(np.asarray(S, dtype=np.float64))
    T, E, C = _check_shape(S)
    a = np.empty(T, dtype=np.int32)
    p = np.empty(E, dtype=np.float64)
    rc = _native().oracle_ssp_solve(T, E, S.ctypes.data, a.ctypes.data, p.ctypes.data)
    if rc != 0:
        raise RuntimeError(f"oracle_ssp_solve failed ({rc})")
    return a, objective(S, a), p


def dual_bound(S: np.ndarray, p: np.ndarray) -> float:
    """D(p) = sum_t max_e (S[t, e] - p[e]) + (T/E) * sum_e p[e].

    For any prices p and any balanced assignment a, D(p) >= OPT >= obj(a)
    (the Lagrangian dual of the transportation LP behind Eq. 2). A balanced a
    with D(p) - obj(a) <= delta is therefore within delta of the optimum.
    Integer-valued inputs (integer dtypes) are summed exactly in int64."""
    S = np.asarray(S)
    T, E, C = _check_shape(S)
    p = np.asarray(p)
    if np.issubdtype(S.dtype, np.integer) and np.issubdtype(p.dtype, np.integer):
        S64, p64 = S.astype(np.int64), p.astype(np.int64)
        return int((S64 - p64[None, :]).max(axis=1).sum() + C * p64.sum())
    S64, p64 = S.astype(np.float64), p.astype(np.float64)
    return float(math.fsum((S64 - p64[None, :]).max(axis=1)) + C * math.fsum(p64))


def greedy_argmax(S: np.ndarray) -> np.ndarray:
    """Test-time assignment (Sec. 3.2.2): every token takes its highest-scoring
    expert (lowest index on ties). Unbalanced in general; its objective
    sum_t max_e S[t, e] is an upper bound of Eq. 2's optimum, reached exactly
    when the greedy assignment happens to be balanced."""
    return np.asarray(S).argmax(axis=1).astype(np.int32)


def greedy_completion(S: np.ndarray, a: np.ndarray, p: np.ndarray) -> np.ndarray:
    """The balance-keeping completion of a solve stopped by its round bound.

    Not a step of the paper: the bounded-latency mode's reading of how to end
    a solve early and still give every expert exactly C = T/E tokens (the
    paper's balance constraint, Eq. 2). Every token still unassigned (a_t <
    0), in ascending token order, takes the expert with room (fewer than C
    tokens at that moment) that maximises S[t, e] - p[e], ties to the lowest
    expert. The difference decides an index, so it is taken in the precision
    the solver uses: float32 for float scores and prices, exact int64 for
    integer ones. S and p are in the same units (the solver's integer mode
    keeps prices in units of 1/K of a score: pass S * K there). Returns the
    completed assignment (a copy)."""
    S = np.asarray(S)
    T, E, C = _check_shape(S)
    out = np.asarray(a, dtype=np.int64).copy()
    p = np.asarray(p)
    if np.issubdtype(S.dtype, np.integer):
        V = S.astype(np.int64) - p.astype(np.int64)[None, :]
    else:
        V = S.astype(np.float32) - p.astype(np.float32)[None, :]
    count = np.bincount(out[out >= 0], minlength=E)
    for t in range(T):
        if out[t] >= 0:
            continue
        best, best_e = None, -1
        for e in range(E):
            if count[e] < C and (best is None or V[t, e] > best):
                best, best_e = V[t, e], e
        if best_e < 0:
            raise ValueError("no expert has room for an unassigned token")
        out[t] = best_e
        count[best_e] += 1
    return out.astype(np.int32)


def stable_perm_partial(a: np.ndarray, E: int) -> np.ndarray:
    """The sort vector of a possibly incomplete assignment (a_t < 0 for
    unassigned tokens): rows [e C, (e + 1) C) hold expert e's tokens in
    ascending order, then -1 for every row the expert has no token for."""
    a = np.asarray(a, dtype=np.int64)
    T = a.shape[0]
    C = T // E
    out = np.full(T, -1, dtype=np.int32)
    for e in range(E):
        toks = np.flatnonzero(a == e)
        if toks.shape[0] > C:
            raise ValueError(f"expert {e} holds more than {C} tokens")
        out[e * C:e * C + toks.shape[0]] = toks
    return out


def optimum_gap(S: np.ndarray, a: np.ndarray) -> float:
    """Second-best gap of an optimal balanced assignment a.

    Any other balanced assignment differs from a by moving tokens around
    cycles of experts (each expert gives up as many tokens as it receives).
    Moving the cheapest token of u to v costs
        w(u, v) = min over t with a_t = u of (S[t, u] - S[t, v]).
    With a optimal every cycle has weight >= 0; the optimum is unique iff the
    lightest cycle is > 0, and that lightest cycle weight (Floyd-Warshall over
    the E experts, min over the diagonal) is the gap to the second-best
    balanced assignment. Returns +inf when no cycle exists (E == 1)."""
    S = np.asarray(S, dtype=np.float64)
    T, E, C = _check_shape(S)
    a = np.asarray(a, dtype=np.int64)
    if E == 1:
        return math.inf
    w = np.full((E, E), math.inf)
    for u in range(E):
        rows = S[a == u]
        if rows.shape[0]:
            w[u] = (rows[:, [u]] - rows).min(axis=0)
    np.fill_diagonal(w, math.inf)
    d = w.copy()
    for k in range(E):
        d = np.minimum(d, d[:, [k]] + d[[k], :])
    return float(np.diagonal(d).min())


def all_pairs_exchange(S: np.ndarray, a: np.ndarray) -> np.ndarray:
    """Every single pairwise swap's objective change (for small tests)."""
    S = np.asarray(S, dtype=np.float64)
    T = S.shape[0]
    out = []
    for i, j in itertools.combinations(range(T), 2):
        if a[i] != a[j]:
            out.append(S[i, a[j]] + S[j, a[i]] - S[i, a[i]] - S[j, a[j]])
    return np.array(out)
