"""The shortest-path finish of an epsilon phase (the last few unassigned
tokens placed by shortest augmenting paths over the experts) against the
oracle: the result keeps the auction's guarantee (balanced, within T * eps of
the exact optimum, certified by the returned prices), with the finish taking
over at different numbers of unassigned tokens, switched off, and with every
step sent through its fallback paths (recomputing whole rows of the exchange
matrix; received rows read by the owners)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2103_16716_amd as pb
import workloads as wl
from gpu_common import EPS_FINAL, dev, host, inputs_on_device
from test_gpu_parity import check_assignment

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "the GPU tests need an MI355X"
    pb.lib()


@pytest.fixture(autouse=True)
def _multi_kernel_path(monkeypatch):
    # The finish belongs to the multi-kernel path: the worker shape would
    # otherwise take the single-workgroup solve.
    monkeypatch.setenv("BASE_SMALL_PATH", "0")


def _scores(name):
    inp = wl.make_inputs(name)
    S = pb.affinity(*inputs_on_device(inp))
    torch.cuda.synchronize()
    return S


@pytest.mark.parametrize("name", ["t2048-e128-d2048-worker", "t8192-e64-d1024", "t4096-e16-d512"])
@pytest.mark.parametrize("cap,fallbacks", [("0", "0"), ("8", "0"), ("32", "0"), ("8", "1"),
                                           ("32", "1")])
def test_finish_settings_against_ssp(monkeypatch, name, cap, fallbacks):
    S = _scores(name)
    S64 = host(S).astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    monkeypatch.setenv("BASE_SSP_CAP", cap)
    monkeypatch.setenv("BASE_TEST_SSP_FALLBACKS", fallbacks)
    res = pb.assign(S)
    check_assignment(S64, res, EPS_FINAL, opt=(a_opt, obj_opt),
                     unique_gap=oracle.optimum_gap(S64, a_opt))
    if cap == "0":
        assert res.stats.augmentations == 0
    else:
        assert res.stats.augmentations > 0


def test_finish_deterministic_and_batched(monkeypatch):
    """Repeated solves and a batch of the same problems give identical
    results with the finish active (its ties are broken by expert and token
    index, not by the order of atomics)."""
    monkeypatch.setenv("BASE_SSP_CAP", "16")
    S = _scores("t2048-e128-d2048-worker")
    runs = [pb.assign(S) for _ in range(3)]
    assert runs[0].stats.augmentations > 0
    for r in runs[1:]:
        assert torch.equal(r.assign, runs[0].assign)
        assert torch.equal(r.prices, runs[0].prices)
    Sb = torch.stack([S, S.flip(0).contiguous(), S]).contiguous()
    rb = pb.assign_batched(Sb)
    assert torch.equal(rb.assign[0], runs[0].assign)
    assert torch.equal(rb.assign[2], runs[0].assign)
    assert torch.equal(rb.prices[0], runs[0].prices)
    one = pb.assign(Sb[1].contiguous())
    assert torch.equal(rb.assign[1], one.assign)


def test_finish_integer_mode_not_used():
    """Integer mode keeps the pure auction (its exactness argument is the
    auction's): no augmentations, exact optimum."""
    T, E = 2048, 16
    rng = np.random.Generator(np.random.PCG64(93))
    Si = rng.integers(-2000, 2000, size=(T, E), dtype=np.int16)
    r = pb.assign(dev(Si))
    assert r.stats.augmentations == 0
    S64 = Si.astype(np.float64)
    _, obj_opt, _ = oracle.solve_ssp(S64)
    assert oracle.objective(S64, host(r.assign)) == obj_opt
