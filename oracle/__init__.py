"""CPU oracle for the BASE-layer balanced assignment path.

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports, calls, links
or executes anything under this directory; only the tests, the smoke check
and the benchmark's CPU-baseline leg do. It shares no code with the GPU
path: its own C sources (plain C, gcc), numpy and scipy.

What it computes, each function citing the passage it follows:
  affinity          token-expert scores h_t . w_e in fp64        (Sec. 3.1, Eq. 2)
  solve_ssp         exact optimum of the balanced assignment    (Sec. 3.2.1, Eq. 2)
  solve_hungarian   the same on the expert-replicated matrix    (Sec. 3.2.1, Eq. 2)
  solve_bruteforce  the same by enumeration, tiny inputs        (Sec. 3.2.1, Eq. 2)
  greedy_argmax     test-time assignment, best expert per token (Sec. 3.2.2)
  greedy_completion balance-keeping end of a round-bounded solve (a reading; Eq. 2's balance)
  stable_perm_partial  sort vector of an incomplete assignment, -1 for empty rows
  dual_bound        LP-duality upper bound of Eq. 2 for prices p
  optimum_gap       second-best gap / uniqueness of an optimum
  stable_perm       sort vector grouping tokens by expert        (Fig. 2 caption)
  gather / scatter  routing into expert-contiguous rows and back (Fig. 2, Sec. 3)
  expert_offsets    row ranges of a (possibly unbalanced) routed order (Sec. 3.2.2)
  gate_combine      gated residual y = sigmoid(h.w_a) f + h          (Sec. 3.1, Eq. 1)
  gate_backward     gradients of Eq. 1's gate and residual           (Sec. 3.1, Eq. 1)
  route_shuffled    shuffle to workers, per-worker solve and route   (Sec. 3.2.1)
  unroute_shuffled  expert rows back to the original token order     (Sec. 3.2.1, Sec. 3)
  gate_combine_shuffled  Eq. 1 over shuffled workers, token order    (Sec. 3.1, 3.2.1)
"""
from .affinity import affinity
from .assign import (
    balanced_counts_ok,
    dual_bound,
    greedy_argmax,
    greedy_completion,
    objective,
    optimum_gap,
    solve_bruteforce,
    solve_hungarian,
    solve_ssp,
    stable_perm_partial,
)
from .gate import expert_offsets, gate_backward, gate_combine
from .permute import gather, scatter, stable_perm
from .shuffle import gate_combine_shuffled, route_shuffled, unroute_shuffled

__all__ = [
    "affinity",
    "expert_offsets",
    "gate_backward",
    "gate_combine",
    "gate_combine_shuffled",
    "route_shuffled",
    "unroute_shuffled",
    "balanced_counts_ok",
    "dual_bound",
    "gather",
    "greedy_argmax",
    "greedy_completion",
    "objective",
    "optimum_gap",
    "scatter",
    "solve_bruteforce",
    "solve_hungarian",
    "solve_ssp",
    "stable_perm",
    "stable_perm_partial",
]
