"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Affinity: elementwise within 2e-3 (bf16 inputs) / 1e-5 (fp32 inputs) of
sum_k |H W|; bit-exact on integer-valued inputs. Assignment: every expert
holds exactly T/E tokens, perm is the stable sort vector of the assignment
bit for bit, the objective is at least the oracle optimum minus T * eps, the
returned prices certify the same bound by LP duality, and the assignment is
identical to the oracle's wherever the optimum is unique by more than T * eps
(always in integer mode). Permute: bit-exact gather and scatter."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2103_16716_amd as pb
import workloads as wl
from gpu_common import (AFF_TOL, EPS_FINAL, affinity_bound, dev, eps_expected,
                        fp32_accumulation_bound, host, inputs_on_device, rounding_slack)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "the GPU tests need an MI355X"
    pb.lib()


def gpu_affinity(H: np.ndarray, W: np.ndarray) -> np.ndarray:
    S = pb.affinity(dev(H), dev(W))
    torch.cuda.synchronize()
    return host(S)


def check_assignment(S: np.ndarray, res, eps: float, opt=None, unique_gap=None, batch_eps=None):
    """The properties every float-mode solve must have, against the oracle."""
    T, E = S.shape
    a = host(res.assign)
    perm = host(res.perm)
    p = host(res.prices).astype(np.float64)
    assert res.stats.converged == 1
    assert oracle.balanced_counts_ok(a, E)
    np.testing.assert_array_equal(perm, oracle.stable_perm(a, E))
    obj = oracle.objective(S, a)
    # The bound is the requested epsilon, raised only to the fp32 floor that
    # the host computes from S itself: the device may not pick its own. With
    # one expert nothing is solved (the only balanced assignment is exact)
    # and the reported bound is 0. A batch reports the largest bound of its
    # problems (batch_eps); each problem is held to its own.
    eps_used = eps_expected(S, eps) if E > 1 else 0.0
    reported = eps_used if batch_eps is None else batch_eps
    assert res.stats.eps_final == pytest.approx(reported, rel=1e-12, abs=0)
    gap = oracle.dual_bound(S, p) - obj
    assert gap >= -1e-9 * max(1.0, abs(obj))            # weak duality
    assert gap <= T * eps_used + rounding_slack(T, S, p)
    if opt is not None:
        a_opt, obj_opt = opt
        assert obj >= obj_opt - T * eps_used
        if unique_gap is not None and unique_gap > T * eps_used + rounding_slack(T, S, p):
            np.testing.assert_array_equal(a, a_opt)
    return a, obj


# ---------------------------------------------------------------- affinity --

@pytest.mark.parametrize("d", [264, 256])
def test_affinity_bf16_integer_inputs_bit_exact(d):
    # T and E ragged against both tilings (64 x 128 and 128 x 128 tokens x
    # experts); d = 264 takes the register-staged kernel, d = 256 (a multiple
    # of 64) the pipelined one
    H, W = wl.small_integer_inputs(300, 200, d, seed=7)
    S = gpu_affinity(wl.f32_to_bf16_bits(H), wl.f32_to_bf16_bits(W))
    np.testing.assert_array_equal(S.astype(np.float64), oracle.affinity(H, W))


def test_affinity_f32_integer_inputs_bit_exact():
    H, W = wl.small_integer_inputs(130, 70, 40, seed=8)
    S = gpu_affinity(H, W)
    np.testing.assert_array_equal(S.astype(np.float64), oracle.affinity(H, W))


@pytest.mark.parametrize("T,E,d", [(1000, 200, 520), (64, 128, 64), (1, 1, 8), (77, 3, 2048),
                                   (1000, 200, 576), (129, 257, 64), (1, 1, 64)])
def test_affinity_bf16_random_ragged(T, E, d):
    rng = np.random.Generator(np.random.PCG64(T * 7 + E))
    Hb = wl.f32_to_bf16_bits(rng.standard_normal((T, d), dtype=np.float32))
    Wb = wl.f32_to_bf16_bits(rng.standard_normal((E, d), dtype=np.float32) / np.sqrt(d))
    H, W = wl.bf16_bits_to_f32(Hb), wl.bf16_bits_to_f32(Wb)
    S = gpu_affinity(Hb, Wb)
    err = np.abs(S - oracle.affinity(H, W))
    assert np.all(err <= affinity_bound(H, W, AFF_TOL["bf16"]))
    assert np.all(err <= fp32_accumulation_bound(H, W))


@pytest.mark.parametrize("T,E,d", [(512, 8, 128), (100, 70, 40), (65, 65, 1032)])
def test_affinity_f32_random_ragged(T, E, d):
    rng = np.random.Generator(np.random.PCG64(T + 3 * E))
    H = rng.standard_normal((T, d), dtype=np.float32)
    W = rng.standard_normal((E, d), dtype=np.float32) / np.float32(np.sqrt(d))
    S = gpu_affinity(H, W)
    err = np.abs(S - oracle.affinity(H, W))
    assert np.all(err <= affinity_bound(H, W, AFF_TOL["f32"]))
    assert np.all(err <= fp32_accumulation_bound(H, W))


@pytest.mark.parametrize("name", ["t512-e8-d128-f32", "t4096-e16-d512", "t8192-e64-d1024",
                                  "t2048-e128-d2048-worker"])
def test_affinity_workloads(name):
    inp = wl.make_inputs(name)
    S = gpu_affinity(inp.H_store, inp.W_store)
    err = np.abs(S - oracle.affinity(inp.H, inp.W))
    assert np.all(err <= affinity_bound(inp.H, inp.W, AFF_TOL[inp.wl.dtype]))
    assert np.all(err <= fp32_accumulation_bound(inp.H, inp.W))


# ---------------------------------------------------------------- assign ---

TINY = [(8, 2), (9, 3), (8, 4), (6, 6), (10, 5), (12, 4), (2, 2), (4, 1)]


@pytest.mark.parametrize("T,E", TINY)
def test_assign_tiny_against_bruteforce(T, E):
    for kind in ("int", "normal"):
        S = wl.random_scores(T, E, seed=1000 + 10 * T + E, kind=kind)
        best, winners = oracle.solve_bruteforce(S)
        res = pb.assign(dev(S))
        a, obj = check_assignment(S.astype(np.float64), res, EPS_FINAL)
        assert obj >= best - T * res.stats.eps_final
        if kind == "int" and len(winners) == 1:
            np.testing.assert_array_equal(a, winners[0])


@pytest.mark.parametrize("T,E", TINY)
def test_assign_tiny_integer_mode_exact(T, E):
    S = wl.random_scores(T, E, seed=2000 + 10 * T + E, kind="int16")
    best, winners = oracle.solve_bruteforce(S.astype(np.float64))
    res = pb.assign(dev(S))
    a = host(res.assign)
    assert oracle.balanced_counts_ok(a, E)
    assert oracle.objective(S, a) == best
    if len(winners) == 1:
        np.testing.assert_array_equal(a, winners[0])
    np.testing.assert_array_equal(host(res.perm), oracle.stable_perm(a, E))


@pytest.mark.parametrize("T,E", [(600, 12), (1000, 40), (64, 64), (17, 1), (2048, 128),
                                 (256, 2)])
def test_assign_ragged_shapes_against_ssp(T, E):
    S = wl.random_scores(T, E, seed=T + E)
    S64 = S.astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    res = pb.assign(dev(S))
    check_assignment(S64, res, EPS_FINAL, opt=(a_opt, obj_opt),
                     unique_gap=oracle.optimum_gap(S64, a_opt))


@pytest.mark.parametrize("T,E", [(3000, 600), (8192, 1024), (4096, 2048), (2048, 2)])
@pytest.mark.parametrize("full", [False, True])
def test_assign_without_the_engine(T, E, full):
    """Shapes the single-workgroup engine does not serve (E > 512 or
    C = T/E > 512): the wide rounds, the round loop and the one-workgroup
    tail solve every phase, with and without the duality check."""
    S = wl.random_scores(T, E, seed=T + E)
    S64 = S.astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    res = pb.assign(dev(S), flags=pb.BASE_ASSIGN_FULL_SCHEDULE if full else 0)
    check_assignment(S64, res, EPS_FINAL, opt=(a_opt, obj_opt),
                     unique_gap=oracle.optimum_gap(S64, a_opt) if E <= 64 else None)
    if full:
        assert res.stats.certified == 0


def test_assign_without_the_engine_integer_and_fallback():
    """The tail path in integer mode (an exact optimum) and under a round
    bound with the greedy completion (balanced, the loss certified)."""
    T, E = 1800, 600
    rng = np.random.Generator(np.random.PCG64(31))
    Si = rng.integers(-500, 500, size=(T, E), dtype=np.int16)
    S64 = Si.astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    r = pb.assign(dev(Si))
    assert r.stats.converged == 1
    assert oracle.balanced_counts_ok(host(r.assign), E)
    assert oracle.objective(S64, host(r.assign)) == obj_opt
    S = wl.random_scores(T, E, seed=32)
    Sf = S.astype(np.float64)
    _, obj_f, _ = oracle.solve_ssp(Sf)
    res = pb.assign(dev(S), max_rounds=3, flags=pb.BASE_ASSIGN_GREEDY_FALLBACK)
    a = host(res.assign)
    assert res.stats.fell_back == 1 and res.stats.converged == 1
    assert oracle.balanced_counts_ok(a, E)
    np.testing.assert_array_equal(host(res.perm), oracle.stable_perm(a, E))
    p = host(res.prices).astype(np.float64)
    gap = oracle.dual_bound(Sf, p) - oracle.objective(Sf, a)
    assert abs(res.stats.dual_gap - gap) <= rounding_slack(T, Sf, p)
    assert obj_f - oracle.objective(Sf, a) <= res.stats.dual_gap + 1e-6 * T


def test_assign_batched_more_problems_than_compute_units():
    """300 problems: more than the 256 compute units, so the batch runs
    without the round loop (its blocks could not all be resident); each
    problem still equals its own solve."""
    B, T, E = 300, 256, 8
    rng = np.random.Generator(np.random.PCG64(301))
    S = rng.standard_normal((B, T, E), dtype=np.float32)
    res = pb.assign_batched(dev(S))
    assert res.stats.converged == 1
    for b in (0, 137, B - 1):
        one = pb.assign(dev(S[b].copy()))
        assert torch.equal(res.assign[b], one.assign)
        assert torch.equal(res.prices[b], one.prices)
        S64 = S[b].astype(np.float64)
        a_opt, obj_opt, _ = oracle.solve_ssp(S64)
        check_assignment(S64, one, EPS_FINAL, opt=(a_opt, obj_opt))


def test_assign_batched_without_the_engine():
    B, T, E = 3, 3000, 600
    S = np.stack([wl.random_scores(T, E, seed=77 + b) for b in range(B)])
    res = pb.assign_batched(dev(S))
    for b in range(B):
        one = pb.assign(dev(S[b].copy()))
        assert torch.equal(res.assign[b], one.assign)
        assert torch.equal(res.prices[b], one.prices)


@pytest.mark.parametrize("name", ["t512-e8-d128-f32", "t4096-e16-d512", "t8192-e64-d1024",
                                  "t2048-e128-d2048-worker"])
def test_assign_workloads_against_ssp(name):
    inp = wl.make_inputs(name)
    Sg = pb.affinity(*inputs_on_device(inp))
    res = pb.assign(Sg)
    S = host(Sg).astype(np.float64)   # the oracle solves the scores the GPU solved
    a_opt, obj_opt, _ = oracle.solve_ssp(S)
    assert res.stats.eps_final == EPS_FINAL     # the stated epsilon, not raised
    check_assignment(S, res, EPS_FINAL, opt=(a_opt, obj_opt),
                     unique_gap=oracle.optimum_gap(S, a_opt))


def test_assign_integer_variant_identical_to_oracle():
    # The int16-quantised scores of the T=4096, E=16 workload: the optimum is
    # unique, and the integer-mode solve is exact, so the assignments match.
    inp = wl.make_inputs("t4096-e16-d512")
    Sq, _ = wl.quantize_scores_int16(oracle.affinity(inp.H, inp.W))
    a_opt, obj_opt, _ = oracle.solve_ssp(Sq.astype(np.float64))
    assert oracle.optimum_gap(Sq.astype(np.float64), a_opt) > 0
    res = pb.assign(dev(Sq))
    a = host(res.assign)
    np.testing.assert_array_equal(a, a_opt)
    np.testing.assert_array_equal(host(res.perm), oracle.stable_perm(a_opt, 16))
    # integer prices certify exact optimality: D(p / K) == OPT
    K = 8192
    p = host(res.prices)
    assert oracle.dual_bound(Sq.astype(np.int64) * K, p) - int(obj_opt) * K < 4096 + 1


@pytest.mark.parametrize("T,E", [(600, 12), (240, 8), (512, 64)])
def test_assign_integer_mode_random_matches_ssp(T, E):
    S = wl.random_scores(T, E, seed=3 * T + E, kind="int16")
    S64 = S.astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    res = pb.assign(dev(S))
    a = host(res.assign)
    assert oracle.balanced_counts_ok(a, E)
    assert oracle.objective(S64, a) == obj_opt
    if oracle.optimum_gap(S64, a_opt) > 0:
        np.testing.assert_array_equal(a, a_opt)


@pytest.mark.parametrize("name", ["t4096-e16-d512", "t32768-e128-d2048-mix8"])
def test_assign_deterministic(name):
    """Five solves of the same scores: identical assignment, sort vector,
    prices and counters (the bid keys order every tie)."""
    inp = wl.make_inputs(name)
    Sg = pb.affinity(*inputs_on_device(inp))
    runs = [pb.assign(Sg) for _ in range(5)]
    for r in runs[1:]:
        assert torch.equal(r.assign, runs[0].assign)
        assert torch.equal(r.perm, runs[0].perm)
        assert torch.equal(r.prices, runs[0].prices)
        assert (r.stats.rounds, r.stats.bids, r.stats.phases) == (
            runs[0].stats.rounds, runs[0].stats.bids, runs[0].stats.phases)


def test_assign_greedy_balanced_case_is_argmax():
    T, E = 960, 12
    S = wl.random_scores(T, E, seed=21)
    S[np.arange(T), np.arange(T) % E] += 10.0
    res = pb.assign(dev(S))
    np.testing.assert_array_equal(host(res.assign), oracle.greedy_argmax(S))


def test_assign_not_converged_and_greedy_fallback():
    S = wl.random_scores(512, 8, seed=5)
    with pytest.raises(pb.BaseError) as ei:
        pb.assign(dev(S), max_rounds=1)
    assert ei.value.status == pb.BASE_ERR_NOT_CONVERGED
    res = pb.assign(dev(S), max_rounds=1, flags=pb.BASE_ASSIGN_GREEDY_FALLBACK)
    assert res.stats.fell_back == 1 and res.stats.converged == 1
    a = host(res.assign)
    assert oracle.balanced_counts_ok(a, 8)
    np.testing.assert_array_equal(host(res.perm), oracle.stable_perm(a, 8))


def test_assign_nonfinite_scores_rejected():
    S = wl.random_scores(64, 8, seed=6)
    S[10, 3] = np.nan
    with pytest.raises(pb.BaseError) as ei:
        pb.assign(dev(S), flags=pb.BASE_ASSIGN_CHECK_FINITE)
    assert ei.value.status == pb.BASE_ERR_NONFINITE
    S[10, 3] = np.inf
    with pytest.raises(pb.BaseError) as ei:
        pb.assign(dev(S), flags=pb.BASE_ASSIGN_CHECK_FINITE)
    assert ei.value.status == pb.BASE_ERR_NONFINITE


def test_assign_user_epsilon_schedule():
    S = wl.random_scores(1024, 16, seed=12)
    S64 = S.astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    res = pb.assign(dev(S), eps_final=1e-3, eps_initial=0.5, eps_factor=4.0)
    assert res.stats.eps_final == pytest.approx(1e-3)
    check_assignment(S64, res, 1e-3, opt=(a_opt, obj_opt))


@pytest.mark.parametrize("name,seed,div,factor", [("t32768-e128-d2048-mix8", 79, 2.0, 24.0),
                                                  ("t65536-e256-d4096", None, 32.0, 8.0)])
def test_assign_phases_that_stay_large(name, seed, div, factor):
    """Epsilon schedules under which many tokens stay active after the fixed
    wide rounds of a phase, so the grid-barrier round loop takes over before
    the single-workgroup engine: the result still meets the epsilon bound
    against the exact optimum."""
    w = wl.WORKLOADS[name]
    if seed is not None:
        w = dataclasses.replace(w, seed=seed)
    inp = wl.make_inputs(w)
    H, W = inputs_on_device(inp)
    S = pb.affinity(H, W)
    torch.cuda.synchronize()
    Sh = host(S)
    rng = float(Sh.max() - Sh.min())
    res = pb.assign(S, eps_initial=rng / div, eps_factor=factor)
    S64 = Sh.astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    check_assignment(S64, res, EPS_FINAL, opt=(a_opt, obj_opt))


@pytest.mark.parametrize("div", [8.0, 64.0, 512.0])
def test_assign_single_phase_large_epsilon(div):
    """One epsilon phase at a coarse epsilon (eps_initial = eps_final): bids
    carry large margins, so within one round an expert's lowest holder is
    often replaced, and the replacing key replaced again. Every token must be
    held exactly once at the end (a lost holder-table store shows up as an
    unbalanced assignment), within T * eps of the optimum."""
    inp = wl.make_inputs("t8192-e64-d1024")
    H, W = inputs_on_device(inp)
    S = pb.affinity(H, W)
    torch.cuda.synchronize()
    Sh = host(S)
    eps = float(Sh.max() - Sh.min()) / div
    res = pb.assign(S, eps_initial=eps, eps_final=eps)
    assert res.stats.phases == 1
    S64 = Sh.astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    check_assignment(S64, res, eps, opt=(a_opt, obj_opt))


def _worker_batch(B, seed0):
    """B independent problems of the paper's per-worker shape (T=2048, E=128,
    d=2048), each drawn with its own seed, as fp32 scores [B, T, E]."""
    base = wl.WORKLOADS["t2048-e128-d2048-worker"]
    Ss = []
    for b in range(B):
        inp = wl.make_inputs(dataclasses.replace(base, seed=seed0 + b))
        H, W = inputs_on_device(inp)
        Ss.append(pb.affinity(H, W))
    return torch.stack(Ss).contiguous()


@pytest.mark.parametrize("route", [None, "1", "0"])
def test_assign_batched_identical_to_single_solves(monkeypatch, route):
    """Sec. 3.2.1 (Sharding): B independent worker problems in one call give,
    problem by problem, exactly what base_assign gives for each alone, and
    each meets the oracle's bound; on the default route and with the
    single-workgroup rounds forced on and off."""
    if route is not None:
        monkeypatch.setenv("BASE_SMALL_PATH", route)
    B = 6
    S = _worker_batch(B, 900)
    res = pb.assign_batched(S)
    assert res.stats.converged == 1
    T, E = S.shape[1], S.shape[2]
    bids = 0
    for b in range(B):
        one = pb.assign(S[b].contiguous())
        bids += one.stats.bids
        assert torch.equal(res.assign[b], one.assign)
        assert torch.equal(res.perm[b], one.perm)
        assert torch.equal(res.prices[b], one.prices)
    assert res.stats.bids == bids
    batch_eps = max(eps_expected(host(S[b]), EPS_FINAL) for b in range(B))
    for b in (0, B - 1):
        S64 = host(S[b]).astype(np.float64)
        a_opt, obj_opt, _ = oracle.solve_ssp(S64)
        one = pb.AssignResult(res.assign[b], res.perm[b], res.prices[b], res.stats)
        check_assignment(S64, one, EPS_FINAL, opt=(a_opt, obj_opt), batch_eps=batch_eps)


def test_assign_batched_integer_mode_and_single_expert():
    B, T, E = 3, 512, 8
    rng = np.random.Generator(np.random.PCG64(77))
    Si = rng.integers(-300, 300, size=(B, T, E), dtype=np.int16)
    res = pb.assign_batched(dev(Si))
    for b in range(B):
        one = pb.assign(dev(Si[b].copy()))
        assert torch.equal(res.assign[b], one.assign)
        assert torch.equal(res.prices[b], one.prices)
        S64 = Si[b].astype(np.float64)
        a_opt, obj_opt, _ = oracle.solve_ssp(S64)
        a = host(res.assign[b])
        assert oracle.balanced_counts_ok(a, E)
        assert oracle.objective(S64, a) == obj_opt      # integer mode: exact optimum
        if oracle.optimum_gap(S64, a_opt) > 0:
            np.testing.assert_array_equal(a, a_opt)
    S1 = torch.randn((4, 96, 1), device="cuda")
    r1 = pb.assign_batched(S1)
    assert torch.all(r1.assign == 0)
    assert torch.equal(r1.perm, torch.arange(96, dtype=torch.int32, device="cuda").repeat(4, 1))


def test_dual_gap_statistic_matches_oracle():
    inp = wl.make_inputs("t8192-e64-d1024")
    S = pb.affinity(*inputs_on_device(inp))
    res = pb.assign(S)
    S64 = host(S).astype(np.float64)
    p = host(res.prices).astype(np.float64)
    gap = oracle.dual_bound(S64, p) - oracle.objective(S64, host(res.assign))
    T = S64.shape[0]
    assert abs(res.stats.dual_gap - gap) <= rounding_slack(T, S64, p)
    assert res.stats.dual_gap <= T * res.stats.eps_final + rounding_slack(T, S64, p)


def test_fallback_dual_gap_certifies_the_loss():
    """Bounded-latency mode: a round budget far below what the solve needs,
    with the balance-keeping greedy completion; the reported gap still bounds
    the distance to the optimum from above."""
    inp = wl.make_inputs("t8192-e64-d1024")
    S = pb.affinity(*inputs_on_device(inp))
    res = pb.assign(S, max_rounds=20, flags=pb.BASE_ASSIGN_GREEDY_FALLBACK)
    assert res.stats.fell_back == 1
    S64 = host(S).astype(np.float64)
    a = host(res.assign)
    assert oracle.balanced_counts_ok(a, S64.shape[1])
    _, obj_opt, _ = oracle.solve_ssp(S64)
    loss = obj_opt - oracle.objective(S64, a)
    p = host(res.prices).astype(np.float64)
    assert loss >= -1e-6
    # the device's gap is the oracle's D(p) - objective at the returned prices
    gap = oracle.dual_bound(S64, p) - oracle.objective(S64, a)
    assert abs(res.stats.dual_gap - gap) <= rounding_slack(S64.shape[0], S64, p)
    assert res.stats.dual_gap >= loss - rounding_slack(S64.shape[0], S64, p)


def test_warm_start_prices():
    """Prices of a previous, similar batch as the starting point: the result
    meets the same bound, typically in fewer rounds."""
    inp = wl.make_inputs("t8192-e64-d1024")
    S = pb.affinity(*inputs_on_device(inp))
    first = pb.assign(S)
    rng = np.random.Generator(np.random.PCG64(3))
    noise = torch.from_numpy(rng.standard_normal(tuple(S.shape), dtype=np.float32)).cuda()
    S2 = (S + 0.01 * noise).contiguous()
    cold = pb.assign(S2)
    prices = first.prices.clone()
    warm = pb.assign(S2, out_prices=prices, warm_start=True)
    S64 = host(S2).astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    check_assignment(S64, warm, EPS_FINAL, opt=(a_opt, obj_opt))
    check_assignment(S64, cold, EPS_FINAL, opt=(a_opt, obj_opt))
    print("rounds cold", cold.stats.rounds, "warm", warm.stats.rounds)


def test_duality_check_stops_early_within_the_bound():
    """After each phase but the last the device measures the duality gap and
    stops once it meets T eps_final: the result is then certified by weak
    duality, not by eps_final-complementary slackness. Against the exact
    optimum both the early result and the full schedule meet the bound; the
    full schedule runs more phases and certifies nothing."""
    inp = wl.make_inputs("t32768-e128-d2048-mix8")
    S = pb.affinity(*inputs_on_device(inp))
    early = pb.assign(S)
    full = pb.assign(S, flags=pb.BASE_ASSIGN_FULL_SCHEDULE)
    S64 = host(S).astype(np.float64)
    T = S64.shape[0]
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    check_assignment(S64, early, EPS_FINAL, opt=(a_opt, obj_opt))
    check_assignment(S64, full, EPS_FINAL, opt=(a_opt, obj_opt))
    assert early.stats.certified == 1 and full.stats.certified == 0
    assert early.stats.phases < full.stats.phases
    assert early.stats.eps_last > early.stats.eps_final
    assert full.stats.eps_last == pytest.approx(full.stats.eps_final)
    # The device's gap agrees with the oracle's dual bound at the returned prices.
    gap = oracle.dual_bound(S64, host(early.prices).astype(np.float64)) - \
        oracle.objective(S64, host(early.assign))
    assert abs(early.stats.dual_gap - gap) <= 1e-6 * T
    assert gap <= T * early.stats.eps_final


def test_duality_check_missed_then_guided():
    """A bound tight enough that the first checks miss it: the next phases
    take the gap-guided steps and the solve still ends within the bound (or
    at the last phase)."""
    inp = wl.make_inputs("t8192-e64-d1024")
    S = pb.affinity(*inputs_on_device(inp))
    S64 = host(S).astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    for eps in (2e-5, 1e-3, 3e-2):
        res = pb.assign(S, eps_final=eps)
        check_assignment(S64, res, eps, opt=(a_opt, obj_opt))
        if eps <= 1e-3:
            assert res.stats.phases >= 2


def test_duality_check_batched_and_integer():
    """The check runs per problem of a batch (each stops on its own), and in
    integer mode a certified stop is still the exact optimum."""
    B = 4
    S = _worker_batch(B, 4200)
    res = pb.assign_batched(S)
    for b in range(B):
        one = pb.assign(S[b].contiguous())
        assert torch.equal(res.assign[b], one.assign)
        assert torch.equal(res.prices[b], one.prices)
    T, E = 2048, 16
    rng = np.random.Generator(np.random.PCG64(91))
    Si = rng.integers(-2000, 2000, size=(T, E), dtype=np.int16)
    r = pb.assign(dev(Si))
    S64 = Si.astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    assert oracle.objective(S64, host(r.assign)) == obj_opt
    print("integer phases", r.stats.phases, "certified", r.stats.certified)


def test_engine_launch_timing():
    """The measurement hook brackets each engine launch with events on the
    call's stream: one record per phase slot, each within the whole call."""
    S = wl.random_scores(8192, 64, seed=5)
    Sd = dev(S)
    ws = torch.empty(pb.assign_workspace_size(8192, 64), dtype=torch.uint8, device="cuda")
    pb.assign(Sd, workspace=ws)
    pb.timing_enable(64)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    pb.assign(Sd, workspace=ws, sync_stats=False)
    e1.record()
    torch.cuda.synchronize()
    n, ms = pb.timing_read()
    pb.timing_enable(0)
    assert n >= 1
    assert 0.0 < ms <= e0.elapsed_time(e1) * 1.01
    res = pb.assign(Sd, workspace=ws)
    assert 0 <= res.stats.engine_bids <= res.stats.bids


# ---------------------------------------------------------------- permute --

@pytest.mark.parametrize("dtype,d", [("bf16", 2048), ("bf16", 24), ("f32", 40), ("f32", 8)])
def test_permute_gather_scatter_bitwise(dtype, d):
    T, E = 1000, 20
    rng = np.random.Generator(np.random.PCG64(d))
    x = rng.standard_normal((T, d), dtype=np.float32)
    xs = wl.f32_to_bf16_bits(x) if dtype == "bf16" else x
    a = rng.permutation(np.repeat(np.arange(E), T // E)).astype(np.int32)
    perm = oracle.stable_perm(a, E)
    X = pb.permute(dev(xs), dev(perm))
    np.testing.assert_array_equal(host(X), oracle.gather(xs, perm))
    Y = pb.permute(X, dev(perm), inverse=True)
    np.testing.assert_array_equal(host(Y), oracle.scatter(oracle.gather(xs, perm), perm))
    np.testing.assert_array_equal(host(Y), xs)


def test_permute_single_row():
    x = wl.f32_to_bf16_bits(np.arange(8, dtype=np.float32)[None, :])
    X = pb.permute(dev(x), dev(np.zeros(1, np.int32)))
    np.testing.assert_array_equal(host(X), x)


# ------------------------------------------------- full sizes, bench setup --

@pytest.mark.parametrize("name", ["t32768-e128-d2048-mix8", "t65536-e256-d4096"])
def test_full_pipeline_against_oracle(name):
    """The whole path at full size, in the launch configuration bench.py times
    (one stream, caller-provided workspace): affinity elementwise, the solve
    against the exact optimum of the scores it solved, the sort vector and
    the permute bit for bit, and the un-permute round trip."""
    inp = wl.make_inputs(name)
    w = inp.wl
    H, W = inputs_on_device(inp)
    S = torch.empty((w.T, w.E), dtype=torch.float32, device="cuda")
    ws = torch.empty(pb.assign_workspace_size(w.T, w.E), dtype=torch.uint8, device="cuda")
    a = torch.empty(w.T, dtype=torch.int32, device="cuda")
    perm = torch.empty(w.T, dtype=torch.int32, device="cuda")
    prices = torch.empty(w.E, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    pb.affinity(H, W, out=S, stream=stream)
    res = pb.assign(S, workspace=ws, out_assign=a, out_perm=perm, out_prices=prices,
                    stream=stream)
    X = pb.permute(H, perm, stream=stream)
    Y = pb.permute(X, perm, inverse=True, stream=stream)
    torch.cuda.synchronize()

    Sh = host(S)
    err = np.abs(Sh - oracle.affinity(inp.H, inp.W))
    assert np.all(err <= affinity_bound(inp.H, inp.W, AFF_TOL["bf16"]))
    S64 = Sh.astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    a_h, _ = check_assignment(S64, res, EPS_FINAL, opt=(a_opt, obj_opt))
    Xh = host(X)
    np.testing.assert_array_equal(Xh, oracle.gather(inp.H_store, host(perm)))
    assert torch.equal(Y.view(torch.int16), H.view(torch.int16))
