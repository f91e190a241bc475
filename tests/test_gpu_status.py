"""How a solve ended, read after the fact (base_assign_status), and the
defined end of a solve whose device-side check fails.

The asynchronous path (no BASE_ASSIGN_SYNC_STATS) is the one a training step
uses; its outcome is read afterwards from the control blocks the workspace
keeps. A failure of the round loop's bounded grid-barrier wait is forced from
the host (BASE_TEST_BARRIER_POLLS=0: every wait gives up at once, so every
block still exits normally); the solve must then end as BASE_ERR_INTERNAL
with no later kernel running on from the half-finished round."""
import math
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2103_16716_amd as pb
import workloads as wl
from gpu_common import dev, host, rounding_slack

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "the GPU tests need an MI355X"
    pb.lib()


def _ws(T, E, B=1):
    n = pb.assign_batched_workspace_size(B, T, E)
    return torch.empty(n, dtype=torch.uint8, device="cuda")


def test_status_of_an_asynchronous_solve():
    T, E = 4096, 16
    S = dev(wl.random_scores(T, E, seed=41))
    ws = _ws(T, E)
    res = pb.assign(S, workspace=ws, sync_stats=False)
    st, stats = pb.assign_status(ws, T, E)
    assert st == pb.BASE_OK
    assert stats.converged == 1 and stats.phases >= 1 and stats.rounds >= 1
    assert math.isnan(stats.dual_gap)
    a = host(res.assign)
    assert oracle.balanced_counts_ok(a, E)
    # the same statistics as a synchronous solve of the same scores
    sync = pb.assign(S)
    assert (sync.stats.phases, sync.stats.rounds, sync.stats.bids) == (
        stats.phases, stats.rounds, stats.bids)
    assert sync.stats.eps_final == stats.eps_final


def test_status_reports_the_round_limit():
    T, E = 512, 8
    S = dev(wl.random_scores(T, E, seed=5))
    ws = _ws(T, E)
    pb.assign(S, workspace=ws, max_rounds=1, sync_stats=False)
    st, stats = pb.assign_status(ws, T, E)
    assert st == pb.BASE_ERR_NOT_CONVERGED
    assert stats.converged == 0
    # with the greedy completion the same bound ends balanced
    res = pb.assign(S, workspace=ws, max_rounds=1, flags=pb.BASE_ASSIGN_GREEDY_FALLBACK,
                    sync_stats=False)
    st, stats = pb.assign_status(ws, T, E)
    assert st == pb.BASE_OK and stats.fell_back == 1 and stats.converged == 1
    assert oracle.balanced_counts_ok(host(res.assign), E)


def test_status_of_a_batch():
    B, T, E = 3, 1024, 16
    S = torch.stack([dev(wl.random_scores(T, E, seed=60 + b)) for b in range(B)]).contiguous()
    ws = _ws(T, E, B)
    pb.assign_batched(S, workspace=ws, sync_stats=False)
    st, stats = pb.assign_status(ws, T, E, B=B)
    assert st == pb.BASE_OK and stats.converged == 1


def test_barrier_give_up_ends_the_solve_as_internal(monkeypatch):
    """Every bounded wait of the round loop's grid barrier gives up at once:
    the solve must stop (no engine, tail or check kernel going on from the
    half-finished round, no greedy completion) and report INTERNAL, both
    synchronously and through the status read. A later solve on the same
    workspace is unaffected."""
    T, E = 8192, 64
    Sh = wl.random_scores(T, E, seed=77)
    S = dev(Sh)
    ws = _ws(T, E)
    # Many plain phases: from the third phase slot on, the round loop takes
    # every phase from its first round (all T tokens active).
    kw = dict(eps_initial=0.5, eps_factor=2.0, flags=pb.BASE_ASSIGN_FULL_SCHEDULE |
              pb.BASE_ASSIGN_GREEDY_FALLBACK)
    monkeypatch.setenv("BASE_TEST_BARRIER_POLLS", "0")
    pb.assign(S, workspace=ws, sync_stats=False, **kw)
    st, stats = pb.assign_status(ws, T, E)
    assert st == pb.BASE_ERR_INTERNAL
    assert stats.converged == 0 and stats.fell_back == 0
    with pytest.raises(pb.BaseError) as ei:
        pb.assign(S, workspace=ws, **kw)
    assert ei.value.status == pb.BASE_ERR_INTERNAL
    monkeypatch.delenv("BASE_TEST_BARRIER_POLLS")
    res = pb.assign(S, workspace=ws, **kw)
    assert res.stats.converged == 1
    a = host(res.assign)
    assert oracle.balanced_counts_ok(a, E)
    st, _ = pb.assign_status(ws, T, E)
    assert st == pb.BASE_OK
    S64 = Sh.astype(np.float64)
    p = host(res.prices).astype(np.float64)
    gap = oracle.dual_bound(S64, p) - oracle.objective(S64, a)
    assert gap <= T * res.stats.eps_final + rounding_slack(T, S64, p)
