"""Seeded synthetic inputs for the balanced token-to-expert assignment path.

This module is shared by the tests, the benchmark and the smoke check. It
draws token features H [T x d] and expert embeddings W [E x d] with the
shapes and value distributions of the BASE-layer workloads, rounds them to
the storage type, and hands out the exact bit patterns both the GPU path and
the CPU oracle receive. It holds none of the method's arithmetic: no
affinity, no assignment, no permutation.

Recipe (stated once, used everywhere):
  * generator  numpy.random.Generator(PCG64(seed)), fp32 draws
  * W          N(0, 1/d)   -> token-expert scores h.w have unit variance
  * H          N(0, 1), or, for the contention workload, a mixture of 8
               clusters: H[t] = W[c(t)] + 0.3 z with c(t) uniform over 8
               experts picked by rng.choice(E, 8, replace=False)
  * bf16       fp32 -> bf16 with round-to-nearest-even on the bit pattern
  * int16      scores for the integer variant: clip(rne(S * 2^s)) with the
               largest s that keeps max|S| * 2^s <= 32767
"""
from __future__ import annotations

import dataclasses
import numpy as np

BASE_SEED = 2103_16716


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    T: int
    E: int
    d: int
    dtype: str          # "f32" or "bf16": storage type of H and W
    dist: str           # "normal" or "mixture8"
    seed: int

    @property
    def C(self) -> int:
        return self.T // self.E


# The six workload shapes. The first five are the measured shapes; the last
# one is the per-worker problem of the paper's training runs (2 sequences of
# 1024 tokens, 128 experts, model dimension 2048; Sec. 4.1 and Sec. 4.2).
WORKLOADS = {
    w.name: w
    for w in [
        Workload("t512-e8-d128-f32", 512, 8, 128, "f32", "normal", BASE_SEED + 0),
        Workload("t4096-e16-d512", 4096, 16, 512, "bf16", "normal", BASE_SEED + 1),
        Workload("t8192-e64-d1024", 8192, 64, 1024, "bf16", "normal", BASE_SEED + 2),
        Workload("t32768-e128-d2048-mix8", 32768, 128, 2048, "bf16", "mixture8", BASE_SEED + 3),
        Workload("t65536-e256-d4096", 65536, 256, 4096, "bf16", "normal", BASE_SEED + 4),
        Workload("t2048-e128-d2048-worker", 2048, 128, 2048, "bf16", "normal", BASE_SEED + 5),
    ]
}
HEADLINE = "t32768-e128-d2048-mix8"


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); return the uint16 patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    out = ((u + rounding) >> np.uint32(16)).astype(np.uint16)
    # keep NaN a NaN (no NaN is ever drawn; this only guards the helper)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to fp32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Inputs:
    """One problem instance. `H`/`W` hold the exact values (fp32 arrays whose
    entries are representable in `dtype`); `H_store`/`W_store` hold what the
    device receives (uint16 bf16 patterns, or the fp32 arrays)."""
    wl: Workload
    H: np.ndarray
    W: np.ndarray
    H_store: np.ndarray
    W_store: np.ndarray
    centres: np.ndarray | None = None


def make_inputs(wl: Workload | str) -> Inputs:
    """Draw H and W for a workload (deterministic in the workload's seed)."""
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    rng = np.random.Generator(np.random.PCG64(wl.seed))
    W = rng.standard_normal((wl.E, wl.d), dtype=np.float32)
    W *= np.float32(1.0 / np.sqrt(wl.d))
    centres = None
    if wl.dist == "normal":
        H = rng.standard_normal((wl.T, wl.d), dtype=np.float32)
    elif wl.dist == "mixture8":
        centres = rng.choice(wl.E, 8, replace=False)
        c = centres[rng.integers(0, 8, wl.T)]
        H = rng.standard_normal((wl.T, wl.d), dtype=np.float32)
        H *= np.float32(0.3)
        H += W[c]
    else:
        raise ValueError(wl.dist)
    if wl.dtype == "bf16":
        Hs, Ws = f32_to_bf16_bits(H), f32_to_bf16_bits(W)
        H, W = bf16_bits_to_f32(Hs), bf16_bits_to_f32(Ws)
    elif wl.dtype == "f32":
        H, W = np.ascontiguousarray(H), np.ascontiguousarray(W)
        Hs, Ws = H, W
    else:
        raise ValueError(wl.dtype)
    return Inputs(wl, H, W, Hs, Ws, centres)


def small_integer_inputs(T: int, E: int, d: int, seed: int, lo: int = -3, hi: int = 3):
    """H, W with integer entries in [lo, hi]: every product and partial sum is
    an integer far below 2^24, so fp32, bf16 and fp64 all hold them exactly."""
    rng = np.random.Generator(np.random.PCG64(seed))
    H = rng.integers(lo, hi + 1, (T, d)).astype(np.float32)
    W = rng.integers(lo, hi + 1, (E, d)).astype(np.float32)
    return H, W


def random_scores(T: int, E: int, seed: int, kind: str = "normal") -> np.ndarray:
    """A score matrix drawn directly (for solver-only tests).
    kind: "normal" fp32 N(0,1); "int" integers in [-1000, 1000] as fp32;
    "int16" int16 values over the full range."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if kind == "normal":
        return rng.standard_normal((T, E), dtype=np.float32)
    if kind == "int":
        return rng.integers(-1000, 1001, (T, E)).astype(np.float32)
    if kind == "int16":
        return rng.integers(-32768, 32768, (T, E)).astype(np.int16)
    raise ValueError(kind)


def quantize_scores_int16(S: np.ndarray) -> tuple[np.ndarray, int]:
    """Integer variant of a score matrix: scale by the largest power of two
    that keeps max|S| within int16, round to nearest even, clip.
    Returns (int16 scores, shift s)."""
    S = np.asarray(S, dtype=np.float64)
    m = float(np.max(np.abs(S)))
    s = int(np.floor(np.log2(32767.0 / m))) if m > 0 else 0
    q = np.clip(np.rint(S * (2.0 ** s)), -32768, 32767).astype(np.int16)
    return q, s


def shuffle_permutation(n: int, seed: int) -> np.ndarray:
    """The random routing of tokens to workers before the solve (Sec. 3.2.1,
    Shuffling), drawn here and passed to both sides as an input: worker
    token i is original token shuffle[i]. int32 [n], a permutation of [0, n)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.permutation(n).astype(np.int32)
