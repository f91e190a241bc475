"""Oracle (test infrastructure only): the gated residual of Eq. 1 and the
gradient of its gate.

Sec. 3.1, Eq. 1: a BASE layer returns, for token t with features h_t and
assigned expert a_t,
    y_t = sigmoid(h_t . w_{a_t}) f_{a_t}(h_t) + h_t .
The expert output f_{a_t}(h_t) is computed in expert-contiguous (routed)
order, so it arrives here as F_perm with row k belonging to token perm[k]
(Fig. 2 caption; Sec. 3: the output returns to the token's position). The
score s_t = h_t . w_{a_t} is the affinity S[t, a_t].

Test-time routing (Sec. 3.2.2) sends every token to its best expert; the
routed order then has expert e's tokens in rows [offsets[e], offsets[e+1]).

Everything is fp64; inputs are the exact values the device receives.
"""
from __future__ import annotations

import numpy as np


def sigmoid(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return 1.0 / (1.0 + np.exp(-x))


def expert_offsets(a: np.ndarray, E: int) -> np.ndarray:
    """offsets[e] = number of tokens assigned to experts below e (E + 1
    entries): expert e's rows of the routed order are [offsets[e], offsets[e+1])."""
    counts = np.bincount(np.asarray(a, dtype=np.int64), minlength=E)
    return np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)


def _token_order(F_perm: np.ndarray, perm: np.ndarray) -> np.ndarray:
    f = np.empty(F_perm.shape, dtype=np.float64)
    f[np.asarray(perm, dtype=np.int64)] = np.asarray(F_perm, dtype=np.float64)
    return f


def gate_combine(F_perm, H, S, a, perm) -> np.ndarray:
    """Eq. 1: y_t = sigmoid(S[t, a_t]) * f_t + h_t, with f_t taken from the
    routed row of token t. Returns y in token order."""
    H = np.asarray(H, dtype=np.float64)
    T = H.shape[0]
    a = np.asarray(a, dtype=np.int64)
    g = sigmoid(np.asarray(S, dtype=np.float64)[np.arange(T), a])
    return g[:, None] * _token_order(F_perm, perm) + H


def gate_backward(dY, F_perm, H, W, S, a, perm):
    """Gradients of L = sum_t dY_t . y_t for y of Eq. 1 with the expert output
    held fixed (its own backward is the expert's business):
        dL/ds_t  = sigmoid'(s_t) (dY_t . f_t),  sigmoid' = sigmoid (1 - sigmoid)
        dL/dh_t  = dY_t + dL/ds_t w_{a_t}      (residual + gate score)
        dL/dw_e  = sum over t with a_t = e of dL/ds_t h_t
        dL/df_t  = sigmoid(s_t) dY_t           (returned in routed order)
    Returns (dH, dF_perm, dW, dS)."""
    dY = np.asarray(dY, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    T = H.shape[0]
    a = np.asarray(a, dtype=np.int64)
    perm = np.asarray(perm, dtype=np.int64)
    s = np.asarray(S, dtype=np.float64)[np.arange(T), a]
    g = sigmoid(s)
    f = _token_order(F_perm, perm)
    dS = g * (1.0 - g) * np.sum(dY * f, axis=1)
    dH = dY + dS[:, None] * W[a]
    dW = np.zeros_like(W)
    np.add.at(dW, a, dS[:, None] * H)
    dF_perm = (g[:, None] * dY)[perm]
    return dH, dF_perm, dW, dS
