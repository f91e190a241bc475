"""Pins of the oracle's shuffled, sharded routing (Sec. 3.2.1, Shuffling and
Sharding) against a hand-worked instance, the permutation equivariance of
the balanced optimum, the exact round trip, and a closed form of Eq. 1 for
a row-wise expert; a planted inverse shuffle must fail them."""
import numpy as np
import pytest

import oracle
import workloads as wl
from conftest import read_golden


def _golden():
    g = read_golden("shuffle_b2_t2_e2.txt")
    B, T, E, d = (int(g[k][0]) for k in ("B", "T", "E", "d"))
    H = np.array(g["H"]).reshape(B * T, d)
    W = np.array(g["W"]).reshape(E, d)
    sh = np.array(g["shuffle"], dtype=np.int32)
    return g, B, T, E, H, W, sh


def _sources(perm, shuffle):
    """Original row of each routed row, read off the oracle's routing by
    following one row at a time (worker row b*T + perm[b, j])."""
    B, T = perm.shape
    return np.array([shuffle[b * T + perm[b, j]] for b in range(B) for j in range(T)])


def test_golden_shuffled_routing():
    g, B, T, E, H, W, sh = _golden()
    S, a, perm, X = oracle.route_shuffled(H, W, sh, B)
    np.testing.assert_array_equal(S.ravel(), g["S_worker"])
    np.testing.assert_array_equal(a.ravel(), g["assign"])
    np.testing.assert_array_equal(perm.ravel(), g["perm"])
    src = np.array(g["sources"], dtype=np.int64)
    np.testing.assert_array_equal(_sources(perm, sh), src)
    np.testing.assert_array_equal(X, H[src])
    tok = np.empty(B * T, dtype=np.int64)
    tok[sh] = a.ravel()
    np.testing.assert_array_equal(tok, g["token_expert"])


def test_planted_inverse_shuffle_fails_the_fixture():
    g, B, T, E, H, W, sh = _golden()
    wrong = np.argsort(sh).astype(np.int32)     # worker i <- token inv[i]: the inverse map
    _, a, perm, X = oracle.route_shuffled(H, W, wrong, B)
    assert not np.array_equal(X, H[np.array(g["sources"], dtype=np.int64)])


def test_single_worker_is_shuffle_equivariant():
    """One worker: shuffling the tokens permutes a unique optimum the same
    way, a_shuffled[i] = a[shuffle[i]], and the routed rows are the same."""
    T, E, d = 96, 4, 16
    rng = np.random.Generator(np.random.PCG64(5))
    H = rng.standard_normal((T, d))
    W = rng.standard_normal((E, d))
    ident = np.arange(T, dtype=np.int32)
    S0, a0, perm0, X0 = oracle.route_shuffled(H, W, ident, 1)
    assert oracle.optimum_gap(S0, a0[0]) > 0           # unique optimum
    sh = wl.shuffle_permutation(T, 11)
    S1, a1, perm1, X1 = oracle.route_shuffled(H, W, sh, 1)
    np.testing.assert_array_equal(a1[0], a0[0][sh])
    # Same tokens per expert; inside an expert the order follows worker order.
    for e in range(E):
        rows = slice(e * (T // E), (e + 1) * (T // E))
        assert sorted(map(tuple, X1[rows])) == sorted(map(tuple, X0[rows]))


@pytest.mark.parametrize("B", [1, 3])
def test_round_trip_restores_token_order(B):
    T, E, d = 24, 4, 8
    rng = np.random.Generator(np.random.PCG64(B))
    H = rng.standard_normal((B * T, d))
    W = rng.standard_normal((E, d))
    sh = wl.shuffle_permutation(B * T, 3 + B)
    S, a, perm, X = oracle.route_shuffled(H, W, sh, B)
    for b in range(B):
        assert oracle.balanced_counts_ok(a[b], E)
    np.testing.assert_array_equal(oracle.unroute_shuffled(X, perm, sh), H)


def test_gate_closed_form_for_a_rowwise_expert():
    """With expert e computing f_e(h) = (1 + e) h, Eq. 1 gives each token
    y_t = (sigmoid(h_t . w_{a_t}) (1 + a_t) + 1) h_t, where a_t is the
    expert its worker gave it."""
    B, T, E, d = 3, 16, 4, 8
    rng = np.random.Generator(np.random.PCG64(9))
    H = rng.standard_normal((B * T, d))
    W = rng.standard_normal((E, d))
    sh = wl.shuffle_permutation(B * T, 21)
    S, a, perm, X = oracle.route_shuffled(H, W, sh, B)
    C = T // E
    expert_of_row = np.tile(np.repeat(np.arange(E), C), B)
    F = X * (1.0 + expert_of_row)[:, None]
    Y = oracle.gate_combine_shuffled(F, H, S, a, perm, sh)
    tok_expert = np.empty(B * T, dtype=np.int64)
    tok_expert[sh] = a.ravel()
    s = np.einsum("td,td->t", H, W[tok_expert])
    expect = ((1.0 / (1.0 + np.exp(-s))) * (1.0 + tok_expert) + 1.0)[:, None] * H
    np.testing.assert_allclose(Y, expect, rtol=1e-12, atol=1e-12)
