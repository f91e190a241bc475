"""base_assign_noalloc (the solve on the library's own per-device workspace
array, for callers that cannot allocate) against base_assign with a caller
workspace: bit-identical assignment, sort vector and prices, on two calls in
a row on the same device, the second with a smaller problem (the array keeps
the first call's state, which the second must not see), each also meeting
the oracle's bound. Sizes beyond the array are rejected before anything is
enqueued."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2103_16716_amd as pb
import workloads as wl
from gpu_common import dev, host, rounding_slack

pytestmark = pytest.mark.gpu


def _noalloc(L, S, out_a, out_p, out_pr, stats):
    """One call through the C ABI (no binding logic in between)."""
    T, E = S.shape
    opts = pb.AssignOpts(0.0, 0.0, 0.0, 0, pb.BASE_ASSIGN_SYNC_STATS)
    return L.base_assign_noalloc(S.data_ptr(), pb.BASE_F32, T, E, ctypes.byref(opts),
                                 out_a.data_ptr(), out_p.data_ptr(), out_pr.data_ptr(),
                                 ctypes.byref(stats), int(torch.cuda.current_stream().cuda_stream))


def _check_against_base_assign(L, Sh):
    T, E = Sh.shape
    S = dev(Sh)
    out_a = torch.full((T,), -7, dtype=torch.int32, device="cuda")
    out_p = torch.full((T,), -7, dtype=torch.int32, device="cuda")
    out_pr = torch.zeros(E, dtype=torch.float32, device="cuda")
    stats = pb.AssignStats()
    assert _noalloc(L, S, out_a, out_p, out_pr, stats) == pb.BASE_OK
    ref = pb.assign(S)
    torch.cuda.synchronize()
    assert torch.equal(out_a, ref.assign)
    assert torch.equal(out_p, ref.perm)
    assert torch.equal(out_pr, ref.prices)
    assert (stats.phases, stats.rounds, stats.bids) == (ref.stats.phases, ref.stats.rounds,
                                                        ref.stats.bids)
    S64 = Sh.astype(np.float64)
    a = host(out_a)
    assert oracle.balanced_counts_ok(a, E)
    np.testing.assert_array_equal(host(out_p), oracle.stable_perm(a, E))
    p = host(out_pr).astype(np.float64)
    _, obj_opt, _ = oracle.solve_ssp(S64)
    assert oracle.objective(S64, a) >= obj_opt - T * stats.eps_final - rounding_slack(T, S64, p)


def test_noalloc_matches_base_assign_twice():
    L = pb.lib()
    big = wl.random_scores(8192, 64, seed=901)
    small = wl.random_scores(2048, 16, seed=902)
    _check_against_base_assign(L, big)
    _check_against_base_assign(L, small)


def test_noalloc_rejects_sizes_beyond_the_array():
    L = pb.lib()
    T, E = 1 << 20, 1024          # workspace far above 32 MiB
    assert pb.assign_workspace_size(T, E) > pb.NOALLOC_MAX_WORKSPACE
    stats = pb.AssignStats()
    opts = pb.AssignOpts(0.0, 0.0, 0.0, 0, 0)
    x = torch.zeros(16, dtype=torch.int32, device="cuda")
    st = L.base_assign_noalloc(x.data_ptr(), pb.BASE_F32, T, E, ctypes.byref(opts), x.data_ptr(),
                               x.data_ptr(), None, ctypes.byref(stats), None)
    assert st == pb.BASE_ERR_RANGE
    # the headline shape fits
    assert pb.assign_workspace_size(32768, 128) <= pb.NOALLOC_MAX_WORKSPACE
    assert pb.assign_workspace_size(65536, 256) <= pb.NOALLOC_MAX_WORKSPACE
