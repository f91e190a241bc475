"""Pins of the oracle's gated residual (Eq. 1) and its gradient, against what
the equation and calculus fix: closed forms, a hand-worked routed example,
and central finite differences of L = sum_t dY_t . y_t."""
import numpy as np
import pytest

import oracle


def test_sigmoid_closed_forms():
    np.testing.assert_allclose(oracle.gate.sigmoid([0.0, np.log(3.0), -np.log(3.0)]),
                               [0.5, 0.75, 0.25], rtol=0, atol=1e-15)


def test_combine_hand_worked_routed_example():
    # Two experts, three tokens; routed order perm = [2, 0, 1]: expert 0 holds
    # token 2 (row 0) and token 0 (row 1)... rows of F_perm belong to tokens
    # perm[k]. Scores chosen so the gates are 1/2, 3/4 and 1/4.
    H = np.array([[1.0, 2.0], [0.0, -1.0], [4.0, 0.5]])
    F_perm = np.array([[10.0, 20.0], [30.0, 40.0], [50.0, 60.0]])
    perm = np.array([2, 0, 1])
    a = np.array([0, 1, 0])
    S = np.array([[0.0, 9.0], [9.0, np.log(3.0)], [-np.log(3.0), 9.0]])
    y = oracle.gate_combine(F_perm, H, S, a, perm)
    # token 0: row 1, gate 1/2; token 1: row 2, gate 3/4; token 2: row 0, gate 1/4
    expect = np.array([[1.0 + 15.0, 2.0 + 20.0],
                       [0.0 + 37.5, -1.0 + 45.0],
                       [4.0 + 2.5, 0.5 + 5.0]])
    np.testing.assert_allclose(y, expect, rtol=0, atol=1e-12)


def test_combine_special_cases():
    rng = np.random.Generator(np.random.PCG64(1))
    T, E, d = 7, 3, 5
    H = rng.standard_normal((T, d))
    F = rng.standard_normal((T, d))
    a = rng.integers(0, E, T)
    perm = oracle.stable_perm(a, E)
    np.testing.assert_allclose(oracle.gate_combine(np.zeros((T, d)), H, rng.standard_normal((T, E)), a, perm), H)
    y0 = oracle.gate_combine(F, H, np.zeros((T, E)), a, perm)
    np.testing.assert_allclose(y0, 0.5 * oracle.scatter(F, perm) + H, rtol=1e-15)


def test_expert_offsets():
    a = np.array([2, 0, 2, 2, 1, 0])
    np.testing.assert_array_equal(oracle.expert_offsets(a, 4), [0, 2, 3, 6, 6])


@pytest.mark.parametrize("seed", [0, 1])
def test_backward_matches_finite_differences(seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    T, E, d = 6, 3, 4
    H = rng.standard_normal((T, d))
    W = rng.standard_normal((E, d)) / np.sqrt(d)
    F = rng.standard_normal((T, d))
    dY = rng.standard_normal((T, d))
    a = np.array([0, 2, 1, 2, 0, 1])
    perm = oracle.stable_perm(a, E)

    def loss(H_, W_, F_):
        S_ = H_ @ W_.T
        return float(np.sum(dY * oracle.gate_combine(F_, H_, S_, a, perm)))

    S = H @ W.T
    dH, dF, dW, dS = oracle.gate_backward(dY, F, H, W, S, a, perm)
    h = 1e-6
    for (X, G) in ((H, dH), (W, dW), (F, dF)):
        num = np.zeros_like(X)
        for idx in np.ndindex(X.shape):
            Xp = X.copy(); Xp[idx] += h
            Xm = X.copy(); Xm[idx] -= h
            args = [H, W, F]
            k = 0 if X is H else (1 if X is W else 2)
            ap = list(args); ap[k] = Xp
            am = list(args); am[k] = Xm
            num[idx] = (loss(*ap) - loss(*am)) / (2 * h)
        np.testing.assert_allclose(G, num, rtol=1e-6, atol=1e-7)
    # dS is the derivative with respect to the gate score itself
    num_s = np.zeros(T)
    for t in range(T):
        Sp = S.copy(); Sp[t, a[t]] += h
        Sm = S.copy(); Sm[t, a[t]] -= h
        yp = oracle.gate_combine(F, H, Sp, a, perm)
        ym = oracle.gate_combine(F, H, Sm, a, perm)
        num_s[t] = np.sum(dY * (yp - ym)) / (2 * h)
    np.testing.assert_allclose(dS, num_s, rtol=1e-6, atol=1e-8)


def test_finite_differences_reject_planted_mistakes():
    # The finite-difference pin separates the true gate derivative from the
    # plausible slips: sigmoid in place of its derivative, a missing score
    # path in dL/dh, and the gate applied to h instead of f.
    rng = np.random.Generator(np.random.PCG64(5))
    T, E, d = 5, 2, 3
    H = rng.standard_normal((T, d))
    W = rng.standard_normal((E, d))
    F = rng.standard_normal((T, d))
    dY = rng.standard_normal((T, d))
    a = np.array([0, 1, 1, 0, 1])
    perm = oracle.stable_perm(a, E)
    S = H @ W.T
    dH, _, _, dS = oracle.gate_backward(dY, F, H, W, S, a, perm)
    g = oracle.gate.sigmoid(S[np.arange(T), a])
    f = oracle.scatter(F, perm)
    wrong_dS = g * np.sum(dY * f, axis=1)
    wrong_dH = dY.copy()
    assert not np.allclose(wrong_dS, dS, rtol=1e-3)
    assert not np.allclose(wrong_dH, dH, rtol=1e-3)
    y_wrong = g[:, None] * H + H
    assert not np.allclose(y_wrong, oracle.gate_combine(F, H, S, a, perm))
