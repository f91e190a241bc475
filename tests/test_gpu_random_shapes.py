"""A seeded sweep of small solver shapes against the oracle's exact optimum:
E from 1 to 700 (across the engine's 512-expert limit), C = T/E from 1 to
600 (across its 512-slot limit), float and int16 scores, clustered and
normal score distributions, the default schedule with the duality check and
the full schedule. Each case must be balanced, carry its sort vector, and
meet the bound (float) or the exact optimum (integer). Every case runs
twice: on the default route (the single-workgroup solve for T <= 2048 and
E <= 256) and with that route switched off (the multi-kernel path)."""
import numpy as np
import pytest

import oracle
import paper_2103_16716_amd as pb
import workloads as wl
from gpu_common import EPS_FINAL, dev, host
from test_gpu_parity import check_assignment

pytestmark = pytest.mark.gpu


def _cases(n=48, seed=2103):
    rng = np.random.Generator(np.random.PCG64(seed))
    out = []
    while len(out) < n:
        E = int(rng.choice([1, 2, 3, 7, 16, 33, 64, 128, 200, 257, 511, 513, 600, 700]))
        C = int(rng.choice([1, 2, 5, 16, 31, 64, 200, 513, 600]))
        if E * C > 6000 or E * C < 2:
            continue
        out.append((E * C, E, str(rng.choice(["normal", "clustered"])),
                    bool(rng.integers(2)), bool(rng.integers(2)), int(rng.integers(1 << 30))))
    return out


@pytest.mark.parametrize("small", ["1", "0"])
@pytest.mark.parametrize("T,E,kind,integer,full,seed", _cases())
def test_random_shape(monkeypatch, small, T, E, kind, integer, full, seed):
    monkeypatch.setenv("BASE_SMALL_PATH", small)
    flags = pb.BASE_ASSIGN_FULL_SCHEDULE if full else 0
    rng = np.random.Generator(np.random.PCG64(seed))
    if integer:
        S = rng.integers(-1000, 1000, size=(T, E), dtype=np.int16)
        if kind == "clustered":
            S[:, : max(1, E // 4)] += 600
    else:
        S = rng.standard_normal((T, E), dtype=np.float32)
        if kind == "clustered":
            S[:, : max(1, E // 4)] += 2.0
    S64 = S.astype(np.float64)
    a_opt, obj_opt, _ = oracle.solve_ssp(S64)
    res = pb.assign(dev(S), flags=flags)
    if integer:
        a = host(res.assign)
        assert res.stats.converged == 1
        assert oracle.balanced_counts_ok(a, E)
        np.testing.assert_array_equal(host(res.perm), oracle.stable_perm(a, E))
        assert oracle.objective(S64, a) == obj_opt
    else:
        check_assignment(S64, res, EPS_FINAL, opt=(a_opt, obj_opt))
