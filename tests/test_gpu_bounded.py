"""Bounded latency: a solve stopped by its round bound.

Without the greedy completion the outputs describe the partial assignment
(assign[t] = -1 for unassigned tokens; each expert's rows of perm hold its
tokens in ascending order, then -1). With it, every unassigned token, in
ascending order, takes its best expert with room at the returned prices: the
device's compacted walk must give exactly the oracle's sequential rule
(decided in float32, as the solver decides it), starting from the same
partial state (the solve is deterministic and the flag changes nothing
before the completion)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2103_16716_amd as pb
import workloads as wl
from gpu_common import dev, host, inputs_on_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "the GPU tests need an MI355X"
    pb.lib()


def _scores(name):
    S = pb.affinity(*inputs_on_device(wl.make_inputs(name)))
    torch.cuda.synchronize()
    return S


def _check_completion(S, rounds):
    T, E = S.shape
    ws = torch.empty(pb.assign_workspace_size(T, E), dtype=torch.uint8, device=S.device)
    part = pb.assign(S, max_rounds=rounds, sync_stats=False, workspace=ws)
    st, stats = pb.assign_status(ws, T, E)
    assert st == pb.BASE_ERR_NOT_CONVERGED and stats.fell_back == 0
    a0 = host(part.assign)
    p0 = host(part.prices)
    assert (a0 < 0).any()
    np.testing.assert_array_equal(host(part.perm), oracle.stable_perm_partial(a0, E))
    full = pb.assign(S, max_rounds=rounds, flags=pb.BASE_ASSIGN_GREEDY_FALLBACK)
    assert full.stats.fell_back == 1 and full.stats.converged == 1
    np.testing.assert_array_equal(host(full.prices), p0)
    Sh = host(S)
    if np.issubdtype(Sh.dtype, np.integer):
        # integer mode: prices are in scaled units, the scores times
        # K = 2^ceil(log2(T + 1)); the rule compares both in those units
        Sh = Sh.astype(np.int64) * (1 << int(T).bit_length())
    want = oracle.greedy_completion(Sh, a0, p0)
    np.testing.assert_array_equal(host(full.assign), want)
    np.testing.assert_array_equal(host(full.perm), oracle.stable_perm(want, E))
    return int((a0 < 0).sum())


@pytest.mark.parametrize("name,rounds", [("t32768-e128-d2048-mix8", 20), ("t8192-e64-d1024", 20),
                                         ("t4096-e16-d512", 3), ("t2048-e128-d2048-worker", 6),
                                         ("t2048-e128-d2048-worker", 1), ("t512-e8-d128-f32", 1)])
def test_greedy_completion_matches_the_sequential_rule(name, rounds):
    """Few experts open (the sorted-preference walk) and many (after one
    round: the re-choosing walk)."""
    _check_completion(_scores(name), rounds)


def test_greedy_completion_many_experts_and_integer_scores():
    """E = 600 (ten experts per lane of the walking wave, no engine) and
    integer mode (int64 values)."""
    T, E = 1800, 600
    S = dev(wl.random_scores(T, E, seed=32))
    _check_completion(S, 3)
    rng = np.random.Generator(np.random.PCG64(94))
    Si = dev(rng.integers(-2000, 2000, size=(4096, 16), dtype=np.int16))
    _check_completion(Si, 2)


def test_greedy_completion_batched_equals_single():
    T, E, B = 2048, 64, 3
    S = torch.stack([dev(wl.random_scores(T, E, seed=70 + b)) for b in range(B)]).contiguous()
    rb = pb.assign_batched(S, max_rounds=4, flags=pb.BASE_ASSIGN_GREEDY_FALLBACK)
    for b in range(B):
        one = pb.assign(S[b].contiguous(), max_rounds=4, flags=pb.BASE_ASSIGN_GREEDY_FALLBACK)
        assert torch.equal(rb.assign[b], one.assign)
        assert torch.equal(rb.perm[b], one.perm)
        assert torch.equal(rb.prices[b], one.prices)
