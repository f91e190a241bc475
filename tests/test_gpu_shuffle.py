"""The random shuffle of tokens to workers and the batched, sharded route
(Sec. 3.2.1, Shuffling and Sharding), through the C ABI, against the oracle.

The device never materialises the shuffled rows: the affinity GEMM, the
batched permute and the batched gated combine all read H through the shuffle
index. Affinity: the tolerance of the unshuffled GEMM, and bit-identical to
base_affinity of the gathered rows (same arithmetic on the same values).
Permutes: bit-exact. Combine: the gate tests' bound. Solves: the bound of
every float-mode solve, per worker."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2103_16716_amd as pb
import workloads as wl
from gpu_common import AFF_TOL, EPS_FINAL, affinity_bound, dev, eps_expected, host
from test_gpu_parity import check_assignment

pytestmark = pytest.mark.gpu

F32_EPS = float(np.finfo(np.float32).eps)
BF16_REL = 2.0 ** -8


def as_f64(x: np.ndarray) -> np.ndarray:
    return wl.bf16_bits_to_f32(x).astype(np.float64) if x.dtype == np.uint16 else x.astype(np.float64)


def rand_rows(rng, n, d, dtype):
    x = rng.standard_normal((n, d), dtype=np.float32)
    return wl.f32_to_bf16_bits(x) if dtype == "bf16" else x


@pytest.mark.parametrize("dtype,d", [("bf16", 264), ("bf16", 192), ("f32", 264)])
def test_affinity_gather(dtype, d):
    """Rows of H taken through an index with repeats, N ragged against the
    64- and 128-row tiles, E and d ragged too (d = 192: the pipelined bf16
    kernel)."""
    h_rows, N, E = 1000, 777, 200
    rng = np.random.Generator(np.random.PCG64(31))
    H = rand_rows(rng, h_rows, d, dtype)
    W = rand_rows(rng, E, d, dtype) if dtype == "bf16" else \
        (rng.standard_normal((E, d), dtype=np.float32) / np.sqrt(d)).astype(np.float32)
    rows = rng.integers(0, h_rows, size=N).astype(np.int32)
    S = pb.affinity(dev(H), dev(W), rows=dev(rows))
    S_mat = pb.affinity(dev(H[rows]), dev(W))
    torch.cuda.synchronize()
    assert torch.equal(S, S_mat)
    ref = oracle.affinity(as_f64(H)[rows], as_f64(W))
    bound = affinity_bound(as_f64(H)[rows], as_f64(W), AFF_TOL[dtype])
    assert np.all(np.abs(host(S) - ref) <= bound)


@pytest.mark.parametrize("d", [32, 128])
def test_affinity_gather_out_of_range_rows_are_zero(d):
    rng = np.random.Generator(np.random.PCG64(32))
    H = rand_rows(rng, 64, d, "bf16")
    W = rand_rows(rng, 16, d, "bf16")
    rows = np.array([3, -1, 64, 63, 1 << 30, 0], dtype=np.int32)
    S = host(pb.affinity(dev(H), dev(W), rows=dev(rows)))
    assert np.all(S[[1, 2, 4]] == 0.0)
    ok = [0, 3, 5]
    ref = oracle.affinity(as_f64(H)[rows[ok]], as_f64(W))
    assert np.all(np.abs(S[ok] - ref) <= affinity_bound(as_f64(H)[rows[ok]], as_f64(W), AFF_TOL["bf16"]))


def _row_perms(rng, B, T):
    return np.stack([rng.permutation(T) for _ in range(B)]).astype(np.int32)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shuffled", [False, True])
def test_permute_batched_bit_exact(dtype, shuffled):
    B, T, d = 5, 96, 40                      # 80-byte bf16 rows: 5 chunks, ragged blocks
    rng = np.random.Generator(np.random.PCG64(41 + shuffled))
    x = rand_rows(rng, B * T, d, dtype)
    perm = _row_perms(rng, B, T)
    sh = wl.shuffle_permutation(B * T, 43) if shuffled else None
    src = (np.arange(B)[:, None] * T + perm).ravel()
    if shuffled:
        src = sh[src]
    out = host(pb.permute_batched(dev(x), dev(perm), shuffle=dev(sh) if shuffled else None))
    np.testing.assert_array_equal(out, oracle.gather(x, src))
    back = host(pb.permute_batched(dev(out), dev(perm), shuffle=dev(sh) if shuffled else None,
                                   inverse=True))
    np.testing.assert_array_equal(back, oracle.scatter(out, src))
    np.testing.assert_array_equal(back, x)


def test_permute_batched_many_tiny_problems():
    B, T, d = 1000, 8, 16
    rng = np.random.Generator(np.random.PCG64(45))
    x = rand_rows(rng, B * T, d, "bf16")
    perm = _row_perms(rng, B, T)
    sh = wl.shuffle_permutation(B * T, 46)
    src = sh[(np.arange(B)[:, None] * T + perm).ravel()]
    out = host(pb.permute_batched(dev(x), dev(perm), shuffle=dev(sh)))
    np.testing.assert_array_equal(out, x[src])


def test_permute_batched_single_problem_is_base_permute():
    rng = np.random.Generator(np.random.PCG64(44))
    T, d = 300, 64
    x = dev(rand_rows(rng, T, d, "bf16"))
    perm = dev(rng.permutation(T).astype(np.int32))
    for inv in (False, True):
        a = pb.permute(x, perm, inverse=inv)
        b = pb.permute_batched(x, perm.view(1, T), inverse=inv)
        assert torch.equal(a, b)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_shuffled_route_and_gate_against_oracle(dtype):
    """The whole shuffled route of B workers on small problems: scores of
    the shuffled rows, one balanced solve per worker, the routed rows, the
    return to token order and Eq. 1, each against the oracle's steps."""
    B, T, E, d = 4, 64, 4, 64
    rng = np.random.Generator(np.random.PCG64(51))
    H = rand_rows(rng, B * T, d, dtype)
    W = rand_rows(rng, E, d, dtype)
    sh = wl.shuffle_permutation(B * T, 52)
    Hd, shd = dev(H), dev(sh)
    S = pb.affinity(Hd, dev(W), rows=shd)
    res = pb.assign_batched(S.view(B, T, E))
    X = pb.permute_batched(Hd, res.perm, shuffle=shd)
    F = rand_rows(rng, B * T, d, dtype)
    Y = pb.gate_combine_batched(dev(F), Hd, S, res.assign, res.perm, shuffle=shd)
    torch.cuda.synchronize()
    Sh = host(S).astype(np.float64)
    a, perm = host(res.assign), host(res.perm)
    S_ref, _, _, _ = oracle.route_shuffled(as_f64(H), as_f64(W), sh, B)
    assert np.all(np.abs(Sh - S_ref) <= affinity_bound(as_f64(H)[sh], as_f64(W), AFF_TOL[dtype]))
    batch_eps = max(eps_expected(Sh[b * T:(b + 1) * T], EPS_FINAL) for b in range(B))
    for b in range(B):
        rows = slice(b * T, (b + 1) * T)
        a_opt, obj_opt, _ = oracle.solve_ssp(Sh[rows])
        one = pb.AssignResult(res.assign[b], res.perm[b], res.prices[b], res.stats)
        check_assignment(Sh[rows], one, EPS_FINAL, opt=(a_opt, obj_opt), batch_eps=batch_eps)
    # Routed rows: worker b's tokens in its expert order, read from the unshuffled H.
    Hw = oracle.gather(H, sh)
    X_ref = np.concatenate([oracle.gather(Hw[b * T:(b + 1) * T], perm[b]) for b in range(B)])
    np.testing.assert_array_equal(host(X), X_ref)
    np.testing.assert_array_equal(oracle.unroute_shuffled(host(X), perm, sh), H)
    ref = oracle.gate_combine_shuffled(as_f64(F), as_f64(H), Sh, a, perm, sh)
    mag = np.abs(oracle.gate_combine_shuffled(np.abs(as_f64(F)), np.abs(as_f64(H)), Sh, a, perm, sh))
    err = np.abs(as_f64(host(Y)) - ref)
    bound = 8 * F32_EPS * mag + (BF16_REL * np.abs(ref) if dtype == "bf16" else 0.0) + 1e-30
    assert np.all(err <= bound), float((err / bound).max())


def test_gate_combine_batched_unshuffled_matches_single_calls():
    B, T, E, d = 3, 128, 8, 32
    rng = np.random.Generator(np.random.PCG64(61))
    S = dev(rng.standard_normal((B * T, E), dtype=np.float32))
    res = pb.assign_batched(S.view(B, T, E))
    F = dev(rand_rows(rng, B * T, d, "bf16"))
    H = dev(rand_rows(rng, B * T, d, "bf16"))
    Y = pb.gate_combine_batched(F, H, S, res.assign, res.perm)
    for b in range(B):
        r = slice(b * T, (b + 1) * T)
        one = pb.gate_combine(F[r], H[r], S[r], res.assign[b], res.perm[b])
        assert torch.equal(Y[r], one)


def test_shuffled_route_at_the_worker_shape():
    """16 workers of the paper's per-worker problem (T = 2048, E = 128,
    d = 2048) shuffled together, in the launch configuration of the batched
    benchmark: every worker's solve meets the oracle's bound, the routed rows
    are exact, and the return restores H bit for bit."""
    base = wl.WORKLOADS["t2048-e128-d2048-worker"]
    B, T, E, d = 16, base.T, base.E, base.d
    hs = [wl.make_inputs(dataclasses.replace(base, seed=base.seed + 1000 * b)) for b in range(B)]
    H = np.concatenate([i.H_store for i in hs])
    W = hs[0].W_store
    sh = wl.shuffle_permutation(B * T, 2103)
    Hd, shd = dev(H), dev(sh)
    S = pb.affinity(Hd, dev(W), rows=shd)
    res = pb.assign_batched(S.view(B, T, E))
    X = pb.permute_batched(Hd, res.perm, shuffle=shd)
    back = pb.permute_batched(X, res.perm, shuffle=shd, inverse=True)
    torch.cuda.synchronize()
    assert res.stats.converged == 1
    assert torch.equal(back, Hd)
    Sh = host(S).astype(np.float64)
    perm = host(res.perm)
    src = sh[(np.arange(B)[:, None] * T + perm).ravel()]
    np.testing.assert_array_equal(host(X), H[src])
    sample = np.random.Generator(np.random.PCG64(5)).choice(B * T, 512, replace=False)
    ref = oracle.affinity(as_f64(H)[sh[sample]], as_f64(W))
    assert np.all(np.abs(Sh[sample] - ref) <=
                  affinity_bound(as_f64(H)[sh[sample]], as_f64(W), AFF_TOL["bf16"]))
    batch_eps = max(eps_expected(Sh[b * T:(b + 1) * T], EPS_FINAL) for b in range(B))
    for b in (0, 7, B - 1):
        rows = slice(b * T, (b + 1) * T)
        a_opt, obj_opt, _ = oracle.solve_ssp(Sh[rows])
        one = pb.AssignResult(res.assign[b], res.perm[b], res.prices[b], res.stats)
        check_assignment(Sh[rows], one, EPS_FINAL, opt=(a_opt, obj_opt), batch_eps=batch_eps)
