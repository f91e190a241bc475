"""Pins for the CPU oracle: each check compares it with something other than
itself -- hand-worked fixtures, brute-force enumeration, a library routine,
LP duality, invariants of Eq. 2 -- so that a dropped term, a wrong sign or a
transposed operand in the oracle fails at least one of them."""
import itertools
import math

import numpy as np
import pytest
import scipy.optimize

import oracle
from oracle import assign as oassign
from oracle.affinity import affinity_loops
import workloads as wl
from conftest import read_golden

TINY = [(8, 2), (9, 3), (8, 4), (6, 6), (6, 1), (10, 5), (12, 4)]


# --------------------------------------------------------------- fixtures ----

def test_golden_handsolved_instance():
    g = read_golden("handsolved_t4_e2.txt")
    T, E = int(g["T"][0]), int(g["E"][0])
    S = np.array(g["S"]).reshape(T, E)
    want = np.array(g["assign"], dtype=np.int32)
    best, winners = oracle.solve_bruteforce(S)
    assert best == g["optimum"][0] and len(winners) == 1
    np.testing.assert_array_equal(winners[0], want)
    a, obj, p = oracle.solve_ssp(S)
    np.testing.assert_array_equal(a, want)
    assert obj == g["optimum"][0]
    ah, objh = oracle.solve_hungarian(S)
    np.testing.assert_array_equal(ah, want)
    np.testing.assert_array_equal(oracle.stable_perm(want, E), np.array(g["perm"], dtype=np.int32))
    np.testing.assert_array_equal(oracle.greedy_argmax(S), np.array(g["greedy"], dtype=np.int32))
    assert oracle.objective(S, oracle.greedy_argmax(S)) == g["greedy_objective"][0]
    assert oracle.dual_bound(S, np.array(g["prices"])) == g["dual"][0]
    assert oracle.optimum_gap(S, want) == g["optimum"][0] - g["second_best"][0]
    # the SSP's own prices certify the same optimum
    assert oracle.dual_bound(S, p) == g["optimum"][0]


def test_golden_fig8_flat_balance():
    g = read_golden("fig8_balance.txt")
    E = int(g["E"][0])
    T = 2048 * E // 16   # any multiple of E
    S = wl.random_scores(T, E, 11)
    a, _, _ = oracle.solve_ssp(S)
    share = 100.0 * np.bincount(a, minlength=E) / T
    assert np.all(np.round(share, 2) == g["percent_per_expert"][0])


def test_golden_affinity_hand_values():
    g = read_golden("affinity_t2_e3_d3.txt")
    T, E, d = int(g["T"][0]), int(g["E"][0]), int(g["d"][0])
    H = np.array(g["H"], dtype=np.float32).reshape(T, d)
    W = np.array(g["W"], dtype=np.float32).reshape(E, d)
    want = np.array(g["S"]).reshape(T, E)
    np.testing.assert_array_equal(oracle.affinity(H, W), want)
    np.testing.assert_array_equal(affinity_loops(H, W), want)


# --------------------------------------------------------------- affinity ----

def test_affinity_matches_explicit_loops():
    rng = np.random.default_rng(5)
    H = rng.standard_normal((7, 13)).astype(np.float32)
    W = rng.standard_normal((5, 13)).astype(np.float32)
    np.testing.assert_allclose(oracle.affinity(H, W), affinity_loops(H, W), rtol=1e-13, atol=1e-13)


def test_affinity_integer_inputs_exact_and_oriented():
    H, W = wl.small_integer_inputs(33, 6, 40, seed=3)
    S = oracle.affinity(H, W)
    # exact integer dot products, computed here with Python ints
    Hi, Wi = H.astype(int), W.astype(int)
    for t in range(33):
        for e in range(6):
            assert S[t, e] == sum(int(x) * int(y) for x, y in zip(Hi[t], Wi[e]))
    assert S.shape == (33, 6)  # rows are tokens, columns experts


def test_affinity_rejects_mismatched_shapes():
    with pytest.raises(ValueError):
        oracle.affinity(np.zeros((3, 4)), np.zeros((2, 5)))


# ----------------------------------------------------------------- solvers ---

@pytest.mark.parametrize("T,E", TINY)
@pytest.mark.parametrize("kind", ["int", "normal"])
def test_solvers_agree_with_bruteforce(T, E, kind):
    S = wl.random_scores(T, E, seed=100 * T + E, kind=kind).astype(np.float64)
    best, winners = oracle.solve_bruteforce(S)
    a, obj, p = oracle.solve_ssp(S)
    ah, objh = oracle.solve_hungarian(S)
    assert oracle.balanced_counts_ok(a, E) and oracle.balanced_counts_ok(ah, E)
    tol = 0 if kind == "int" else 1e-12 * (1 + abs(best))
    assert abs(obj - best) <= tol and abs(objh - best) <= tol
    if len(winners) == 1:
        np.testing.assert_array_equal(a, winners[0])
        np.testing.assert_array_equal(ah, winners[0])
    assert abs(oracle.dual_bound(S, p) - obj) <= tol


def test_bruteforce_enumerates_every_balanced_assignment():
    # all-zero scores: every balanced assignment is optimal
    for T, E in [(8, 2), (9, 3), (8, 4), (6, 6)]:
        _, winners = oracle.solve_bruteforce(np.zeros((T, E)))
        assert len(winners) == oassign.count_balanced(T, E)
        assert len({tuple(w) for w in winners}) == len(winners)
        assert all(oracle.balanced_counts_ok(w, E) for w in winners)
    assert oassign.count_balanced(8, 2) == 70 and oassign.count_balanced(12, 4) == 369600


@pytest.mark.parametrize("T,E", [(64, 8), (256, 16), (512, 8), (240, 12)])
def test_ssp_matches_scipy_linear_sum_assignment(T, E):
    S = wl.random_scores(T, E, seed=T + E).astype(np.float64)
    r, c = scipy.optimize.linear_sum_assignment(np.repeat(S, T // E, axis=1), maximize=True)
    ref = float(np.repeat(S, T // E, axis=1)[r, c].sum())
    a, obj, p = oracle.solve_ssp(S)
    ah, objh = oracle.solve_hungarian(S)
    assert abs(obj - ref) <= 1e-9 * abs(ref)
    assert abs(objh - ref) <= 1e-9 * abs(ref)
    assert oracle.balanced_counts_ok(a, E)


def test_square_case_is_plain_lsap():
    # T == E: one token per expert, the classic square assignment problem
    S = wl.random_scores(40, 40, seed=9).astype(np.float64)
    r, c = scipy.optimize.linear_sum_assignment(S, maximize=True)
    a, obj, _ = oracle.solve_ssp(S)
    np.testing.assert_array_equal(a, c.astype(np.int32))
    assert abs(obj - S[r, c].sum()) < 1e-9


def test_single_expert_takes_everything():
    S = wl.random_scores(17, 1, seed=4).astype(np.float64)
    a, obj, p = oracle.solve_ssp(S)
    assert np.all(a == 0) and abs(obj - S.sum()) < 1e-12
    assert oracle.optimum_gap(S, a) == math.inf


def test_greedy_balanced_special_case():
    # Token t strongly prefers expert t % E: the greedy (test-time) choice is
    # already balanced, so it is the balanced optimum and the upper bound
    # sum_t max_e S[t, e] is reached.
    T, E = 96, 8
    S = wl.random_scores(T, E, seed=21).astype(np.float64)
    S[np.arange(T), np.arange(T) % E] += 10.0
    g = oracle.greedy_argmax(S)
    assert oracle.balanced_counts_ok(g, E)
    a, obj, _ = oracle.solve_ssp(S)
    np.testing.assert_array_equal(a, g)
    assert obj == pytest.approx(S.max(axis=1).sum(), rel=1e-14)


def test_greedy_is_upper_bound():
    S = wl.random_scores(256, 16, seed=2).astype(np.float64)
    _, obj, _ = oracle.solve_ssp(S)
    assert S.max(axis=1).sum() >= obj


def test_weak_duality_holds_for_any_prices():
    rng = np.random.default_rng(0)
    T, E = 12, 4
    S = wl.random_scores(T, E, seed=3, kind="int").astype(np.float64)
    best, _ = oracle.solve_bruteforce(S)
    for _ in range(50):
        p = rng.normal(0, 500, E)
        assert oracle.dual_bound(S, p) >= best - 1e-9
        a = rng.permutation(np.repeat(np.arange(E), T // E))
        assert oracle.dual_bound(S, p) >= oracle.objective(S, a)


def test_dual_bound_integer_path_is_exact():
    S = wl.random_scores(64, 8, seed=5, kind="int16")
    a, obj, p = oracle.solve_ssp(S)
    assert np.all(p == np.round(p))
    assert oracle.dual_bound(S, p.astype(np.int64)) == int(obj)


def test_dual_bound_shift_invariance():
    S = wl.random_scores(32, 4, seed=8).astype(np.float64)
    p = np.array([0.3, -1.2, 2.0, 0.7])
    assert oracle.dual_bound(S, p) == pytest.approx(oracle.dual_bound(S, p + 5.25), rel=1e-14)


def test_optimum_gap_matches_bruteforce_second_best():
    for seed in range(6):
        T, E = 9, 3
        S = wl.random_scores(T, E, seed=seed, kind="int").astype(np.float64) // 100
        best, winners = oracle.solve_bruteforce(S)
        vals = sorted({float(sum(S[t, e] for t, e in enumerate(x)))
                       for x in itertools.product(range(E), repeat=T)
                       if all(x.count(k) == T // E for k in range(E))}, reverse=True)
        gap = oracle.optimum_gap(S, winners[0])
        if len(winners) > 1:
            assert gap == 0
        else:
            assert gap == vals[0] - vals[1]


# ------------------------------------------------------------ metamorphic ---

def test_column_and_row_shifts():
    T, E = 120, 6
    S = wl.random_scores(T, E, seed=31, kind="int").astype(np.float64)
    a, obj, _ = oracle.solve_ssp(S)
    assert oracle.optimum_gap(S, a) > 0
    c = np.arange(E) * 7.0 - 11.0
    r = np.arange(T) * 3.0 + 1.0
    a2, obj2, _ = oracle.solve_ssp(S + c[None, :] + r[:, None])
    np.testing.assert_array_equal(a2, a)
    assert obj2 == obj + (T // E) * c.sum() + r.sum()


def test_token_and_expert_permutations():
    T, E = 120, 6
    S = wl.random_scores(T, E, seed=32, kind="int").astype(np.float64)
    a, obj, _ = oracle.solve_ssp(S)
    assert oracle.optimum_gap(S, a) > 0
    rng = np.random.default_rng(1)
    pt, pe = rng.permutation(T), rng.permutation(E)
    a_t, obj_t, _ = oracle.solve_ssp(S[pt])
    np.testing.assert_array_equal(a_t, a[pt])
    a_e, obj_e, _ = oracle.solve_ssp(S[:, pe])
    inv = np.argsort(pe)
    np.testing.assert_array_equal(a_e, inv[a])
    assert obj_t == obj and obj_e == obj


# ------------------------------------------------------------------ permute -

def test_stable_perm_definition_and_routing_rule():
    T, E = 60, 5
    rng = np.random.default_rng(3)
    a = rng.permutation(np.repeat(np.arange(E), T // E)).astype(np.int32)
    perm = oracle.stable_perm(a, E)
    want = [t for e in range(E) for t in range(T) if a[t] == e]
    np.testing.assert_array_equal(perm, want)
    # Fig. 2: sorted row k goes to expert floor(k E / T)
    np.testing.assert_array_equal(a[perm], (np.arange(T) * E) // T)


# ---------------------------------------------- round-bounded completion ----

def test_greedy_completion_hand_example_capacity_binds():
    # worked by hand, C = 2: tokens 0 and 1 fill expert 0, so token 2 (which
    # prefers expert 0) and token 3 go to expert 1
    S = np.array([[1.0, 0.0], [2.0, 0.0], [3.0, 0.0], [0.0, 5.0]])
    a = oracle.greedy_completion(S, np.full(4, -1), np.zeros(2))
    np.testing.assert_array_equal(a, [0, 0, 1, 1])


def test_greedy_completion_ties_and_existing_holders():
    # ties go to the lowest expert; C = 1
    a = oracle.greedy_completion(np.ones((2, 2)), np.full(2, -1), np.zeros(2))
    np.testing.assert_array_equal(a, [0, 1])
    # token 0 already holds a slot of expert 1 (C = 2): token 1 takes the
    # other one, tokens 2 and 3 (both preferring expert 1) go to expert 0;
    # the prices enter as S - p (expert 0 made cheaper by p = -1 changes
    # nothing here, expert 1 made dearer by 10 sends token 1 to expert 0)
    S = np.array([[0.0, 1.0], [0.0, 2.0], [0.0, 3.0], [0.0, 4.0]])
    start = np.array([1, -1, -1, -1])
    np.testing.assert_array_equal(oracle.greedy_completion(S, start, np.zeros(2)), [1, 1, 0, 0])
    np.testing.assert_array_equal(
        oracle.greedy_completion(S, start, np.array([-1.0, 10.0])), [1, 0, 0, 1])


def test_greedy_completion_unconstrained_is_argmax_of_values():
    # tokens 0..15 are unassigned and token t strongly prefers expert t % 4;
    # every expert already holds 12 of its C = 16 slots, so each has exactly
    # the room its 4 admirers need: the rule reduces to numpy's argmax of
    # S - p, row by row
    T, E = 64, 4
    rng = np.random.default_rng(11)
    S = rng.standard_normal((T, E)).astype(np.float32)
    S[np.arange(16), np.arange(16) % E] += 10.0
    p = (0.1 * rng.standard_normal(E)).astype(np.float32)
    a = np.full(T, -1)
    a[16:] = np.arange(T - 16) % E
    out = oracle.greedy_completion(S, a, p)
    np.testing.assert_array_equal(out[:16], np.argmax(S[:16] - p[None, :], axis=1))
    np.testing.assert_array_equal(out[16:], a[16:])
    assert oracle.balanced_counts_ok(out, E)
    assert oracle.balanced_counts_ok(oracle.greedy_completion(S, np.full(T, -1), p), E)


def test_greedy_completion_decides_in_float32():
    # 1 and 1 + 2^-30 are equal in float32: the tie goes to expert 0 (an fp64
    # comparison would pick expert 1)
    S = np.array([[1.0, 1.0 + 2.0 ** -30], [0.0, 0.0]])
    np.testing.assert_array_equal(oracle.greedy_completion(S, np.full(2, -1), np.zeros(2)),
                                  [0, 1])
    # integer scores and prices are exact
    Si = np.array([[3, 5], [7, 2]], dtype=np.int16)
    pi = np.array([0, 3], dtype=np.int64)
    np.testing.assert_array_equal(oracle.greedy_completion(Si, np.full(2, -1), pi), [0, 1])


def test_stable_perm_partial_pads_empty_rows():
    np.testing.assert_array_equal(oracle.stable_perm_partial([1, -1, 0, 1], 2), [2, -1, 0, 3])
    a = np.repeat(np.arange(3), 4)[np.random.default_rng(5).permutation(12)]
    np.testing.assert_array_equal(oracle.stable_perm_partial(a, 3), oracle.stable_perm(a, 3))


def test_gather_scatter_roundtrip_bitwise():
    T, E, d = 48, 4, 9
    rng = np.random.default_rng(4)
    H = rng.standard_normal((T, d)).astype(np.float32)
    a = rng.permutation(np.repeat(np.arange(E), T // E))
    perm = oracle.stable_perm(a, E)
    X = oracle.gather(H, perm)
    for k in range(T):
        assert np.array_equal(X[k], H[perm[k]])
    Y = oracle.scatter(X, perm)
    assert np.array_equal(Y.view(np.uint32), H.view(np.uint32))


# --------------------------------------------------------- planted mistakes -
# Each test plants a plausible mistake in a copy of an oracle routine and
# checks that the pins above would reject it.

def test_planted_dropped_price_term_breaks_weak_duality():
    def bad_dual(S, p):
        return float(np.max(S - p[None, :], axis=1).sum())   # drops (T/E) sum p
    T, E = 12, 4
    S = wl.random_scores(T, E, seed=3, kind="int").astype(np.float64)
    best, _ = oracle.solve_bruteforce(S)
    p = np.full(E, 400.0)
    assert bad_dual(S, p) < best          # the bug is caught
    assert oracle.dual_bound(S, p) >= best


def test_planted_sign_flip_fails_bruteforce_pin():
    T, E = 8, 2
    S = wl.random_scores(T, E, seed=77, kind="int").astype(np.float64)
    best, _ = oracle.solve_bruteforce(S)
    a_bad, _, _ = oracle.solve_ssp(-S)     # a solver that minimises
    assert oracle.objective(S, a_bad) < best


def test_planted_transposed_operand_fails_affinity_fixture():
    g = read_golden("affinity_t2_e3_d3.txt")
    H = np.array(g["H"]).reshape(2, 3)
    W = np.array(g["W"]).reshape(3, 3)
    want = np.array(g["S"]).reshape(2, 3)
    bad = H @ W          # forgot the transpose
    assert not np.array_equal(bad, want)


def test_planted_unbalanced_solver_fails_count_pin():
    S = wl.random_scores(64, 8, seed=1)
    assert not oracle.balanced_counts_ok(oracle.greedy_argmax(S), 8)


def test_planted_unstable_sort_fails_perm_pin():
    a = np.array([1, 0, 1, 0, 1, 0], dtype=np.int32)
    bad = np.argsort(-a, kind="stable")[::-1]   # groups by expert, but token order reversed
    assert not np.array_equal(bad, oracle.stable_perm(a, 2))
