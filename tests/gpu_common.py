"""Helpers of the GPU parity tests: moving the seeded inputs onto the device
and the tolerances the comparisons use. Nothing here computes any step of
the method."""
from __future__ import annotations

import math

import numpy as np
import torch

import workloads as wl

EPS_FINAL = 1e-4          # default final epsilon of the float-mode solve (score units)
AFF_TOL = {"bf16": 2e-3, "f32": 1e-5}   # relative to sum_k |H[t,k] W[e,k]|


def dev(x: np.ndarray) -> torch.Tensor:
    """A host array on the GPU, bit for bit (uint16 arrays become bfloat16)."""
    if x.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(x: torch.Tensor) -> np.ndarray:
    if x.dtype == torch.bfloat16:
        return x.view(torch.int16).cpu().numpy().view(np.uint16)
    return x.cpu().numpy()


def inputs_on_device(inp: wl.Inputs):
    return dev(inp.H_store), dev(inp.W_store)


def affinity_bound(H: np.ndarray, W: np.ndarray, rel: float) -> np.ndarray:
    """rel * sum_k |H[t,k] W[e,k]|: the error scale of an fp32-accumulated dot
    product, well defined where the dot product itself is near zero."""
    return rel * (np.abs(H.astype(np.float64)) @ np.abs(W.astype(np.float64)).T) + 1e-30


def rounding_slack(T: int, S: np.ndarray, p: np.ndarray) -> float:
    """fp32 rounding allowance of the float-mode duality certificate: a few
    ulps per token at the magnitude scores and prices reach."""
    mag = float(np.abs(S).max()) + float(np.abs(p).max())
    return T * 16.0 * float(np.finfo(np.float32).eps) * mag


def eps_expected(S: np.ndarray, eps: float) -> float:
    """The epsilon bound a float-mode solve must report for scores S and a
    requested eps_final: eps itself, raised to the fp32 resolution floor
    2^-20 * (max|S| + 3 * (max S - min S)) when that is larger (about eight
    ulps of the largest price a solve can reach). Computed here from S in
    double, independently of the device."""
    S32 = np.asarray(S, dtype=np.float32)
    smax, smin = float(S32.max()), float(S32.min())
    mag = max(abs(smax), abs(smin)) + 3.0 * (smax - smin) + 1e-30
    return max(float(eps), math.ldexp(mag, -20))


def fp32_accumulation_bound(H: np.ndarray, W: np.ndarray) -> np.ndarray:
    """(d + 1) * 2^-24 * sum_k |H[t,k] W[e,k]|: the worst-case error of a dot
    product of length d accumulated in fp32 in any order (gamma_d), with one
    more rounding for fp32 products (bf16 products are exact in fp32)."""
    d = H.shape[1]
    return (d + 1) * 2.0 ** -24 * (np.abs(H.astype(np.float64)) @ np.abs(W.astype(np.float64)).T) + 1e-30
