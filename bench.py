"""Throughput of the balanced-assignment path on one MI355X.

One step = the whole path on one batch of resident synthetic input:
affinity GEMM (S = H W^T), balanced assignment (auction), and the permute of
H into expert-contiguous rows (plus the inverse permute on the workload that
includes it). Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--no-cpu-baseline] [--batch B] [--no-shuffle] [--layer]
                    [--max-rounds R] [--seed-spread N]

With --max-rounds R the timed solves stop after R bidding rounds and the
greedy completion fills the free slots (bounded latency; the line reports
the solve time next to the duality gap the result keeps). On the headline
workload the line also reports the step over N mixture seeds (default 5;
--seed-spread 0 skips it).

With --batch B > 1 it measures B independent problems of the paper's
per-worker shape (Sec. 3.2.1 Sharding; T=2048, E=128, d=2048) with the
random shuffle of tokens to workers (Sec. 3.2.1 Shuffling; a seeded
permutation of the B * T tokens, an input): one affinity GEMM over the
shuffled rows against the shared expert embeddings (base_affinity_gather),
one base_assign_batched call, and one permute of all problems' rows
(base_permute_batched), both reading H through the shuffle index.

With --layer it measures the layer's calls around the experts instead
(Sec. 3.1 Eq. 1, Sec. 3.2.2): test-time routing (base_greedy_assign), the
gated residual returned to token order (base_gate_combine) and its
backward (base_gate_backward), on the workload's scores with seeded random
expert outputs and upstream gradients.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads as wl  # noqa: E402

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix-core peak, TFLOP/s
UNPERMUTE_WORKLOADS = {"t65536-e256-d4096"}
COLD_STEPS = 5                 # steps timed after evicting the caches
ENGINE_KERNEL = "engine_kernel"   # the solve's dominant kernel (rounds with few active tokens)
PROFILES = os.path.join(ROOT, "profiles")


def engine_source_digest() -> str:
    """sha256 of the solver source: counters taken on another version of the
    kernel do not describe this one."""
    import hashlib
    path = os.path.join(ROOT, "paper_2103_16716_amd", "csrc", "auction.hip")
    return hashlib.sha256(open(path, "rb").read()).hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per engine launch from the committed counter summary of this
    workload (FETCH_SIZE and WRITE_SIZE per dispatch, each scaled by what the
    counter reads for a plain copy of known size), or None when there is no
    summary or it was taken on a different version of the solver source."""
    path = os.path.join(PROFILES, f"engine_kernel_traffic_{workload}.json")
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != engine_source_digest():
        return None
    return (rec["fetch_kib_per_dispatch"] * rec["fetch_factor"] +
            rec["write_kib_per_dispatch"] * rec["write_factor"]) * 1024.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=wl.HEADLINE, choices=sorted(wl.WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--no-shuffle", action="store_true")
    ap.add_argument("--layer", action="store_true")
    ap.add_argument("--max-rounds", type=int, default=0)
    ap.add_argument("--seed-spread", type=int, default=-1)
    return ap.parse_args()


def bench_layer(args) -> None:
    """Routing and gate calls of one layer step (see the module note)."""
    import torch

    import paper_2103_16716_amd as pb

    torch.cuda.set_device(0)
    inp = wl.make_inputs(args.workload)
    w = inp.wl
    T, E, d = w.T, w.E, w.d
    if w.dtype != "bf16":
        print("--layer measures bf16 workloads", file=sys.stderr)
        sys.exit(2)
    H = torch.from_numpy(inp.H_store.view(np.int16)).cuda().view(torch.bfloat16)
    W = torch.from_numpy(inp.W_store.view(np.int16)).cuda().view(torch.bfloat16)
    S = pb.affinity(H, W)
    r = pb.assign(S)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(20210331)
    F = torch.randn((T, d), generator=gen, device="cuda").to(torch.bfloat16)
    dY = torch.randn((T, d), generator=gen, device="cuda").to(torch.bfloat16)
    Y = torch.empty_like(H)
    offsets = pb.balanced_offsets(T, E, H.device)
    gws = torch.empty(max(int(pb.lib().base_greedy_workspace_size(T, E)), 256),
                      dtype=torch.uint8, device="cuda")
    ga = torch.empty(T, dtype=torch.int32, device="cuda")
    gp = torch.empty(T, dtype=torch.int32, device="cuda")
    go = torch.empty(E + 1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    names = ("greedy", "combine", "backward")

    def step(evs=None):
        if evs is not None:
            evs[0].record(stream)
        pb.greedy_assign(S, workspace=gws, stream=stream, out_assign=ga, out_perm=gp,
                         out_offsets=go)
        if evs is not None:
            evs[1].record(stream)
        pb.gate_combine(F, H, S, r.assign, r.perm, out=Y, stream=stream)
        if evs is not None:
            evs[2].record(stream)
        pb.gate_backward(dY, F, H, W, S, r.assign, r.perm, offsets=offsets, stream=stream)
        if evs is not None:
            evs[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    per = {n: sum(ev[i].elapsed_time(ev[i + 1]) for ev in events) / args.steps
           for i, n in enumerate(names)}
    # Algorithmic HBM bytes per call: the greedy route reads the scores and
    # writes the routing; the combine reads F and H rows and writes y rows
    # (plus index and score); the backward reads dY and F rows, writes dH and
    # dF rows, and reads each H row once more for dW.
    row = 2 * d
    nbytes = {
        "greedy": T * 4 * E + 3 * T * 4 + 4 * (E + 1),
        "combine": 3 * T * row + 12 * T,
        "backward": 5 * T * row + 12 * T + 4 * E * d + 4 * T,
    }
    roof = {n: {"bound": "hbm", "achieved": round(nbytes[n] / (per[n] * 1e-3) / 1e9, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(nbytes[n] / (per[n] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
            for n in names}
    total_ms = sum(per.values())
    out = {
        "metric": f"tokens/sec through test-time routing + gate + gate backward at "
                  f"T={T},E={E},d={d}",
        "value": T / (total_ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": total_ms,
        "wall_ms_per_step": wall_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded scores, expert outputs and upstream gradients)",
        "config": {"workload": w.name, "T": T, "E": E, "d": d, "calls": list(names)},
        "per_call_ms": {n: round(per[n], 4) for n in names},
        "per_call_roofline": roof,
    }
    print(json.dumps(out), flush=True)


def bench_batched(args) -> None:
    """B independent worker-shape problems per step (see the module note)."""
    import dataclasses

    import torch

    import paper_2103_16716_amd as pb

    torch.cuda.set_device(0)
    B = args.batch
    base = wl.WORKLOADS["t2048-e128-d2048-worker"]
    T, E, d = base.T, base.E, base.d
    hs = []
    W = None
    for b in range(B):
        inp = wl.make_inputs(dataclasses.replace(base, seed=base.seed + 1000 * b))
        hs.append(inp.H_store)
        if W is None:
            W = torch.from_numpy(inp.W_store.view(np.int16)).cuda().view(torch.bfloat16)
    H = torch.from_numpy(np.concatenate(hs).view(np.int16)).cuda().view(torch.bfloat16)
    S = torch.empty((B * T, E), dtype=torch.float32, device="cuda")
    a = torch.empty((B, T), dtype=torch.int32, device="cuda")
    perm = torch.empty((B, T), dtype=torch.int32, device="cuda")
    prices = torch.empty((B, E), dtype=torch.float32, device="cuda")
    ws = torch.empty(pb.assign_batched_workspace_size(B, T, E), dtype=torch.uint8, device="cuda")
    X = torch.empty((B * T, d), dtype=torch.bfloat16, device="cuda")
    shuffle = None if args.no_shuffle else \
        torch.from_numpy(wl.shuffle_permutation(B * T, 2103)).cuda()
    stream = torch.cuda.current_stream()

    def step(evs=None):
        if evs is not None:
            evs[0].record(stream)
        pb.affinity(H, W, out=S, rows=shuffle, stream=stream)
        if evs is not None:
            evs[1].record(stream)
        pb.assign_batched(S.view(B, T, E), sync_stats=False, workspace=ws, out_assign=a,
                          out_perm=perm, out_prices=prices, stream=stream)
        if evs is not None:
            evs[2].record(stream)
        pb.permute_batched(H, perm, shuffle=shuffle, out=X, stream=stream)
        if evs is not None:
            evs[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    pb.timing_enable(64 * args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    eng_launches, eng_ms = pb.timing_read()
    pb.timing_enable(0)
    names = ["affinity", "assign", "permute"]
    per_call_ms = {n: float(np.mean([ev[i].elapsed_time(ev[i + 1]) for ev in events]))
                   for i, n in enumerate(names)}
    gpu_ms = float(np.mean([ev[0].elapsed_time(ev[-1]) for ev in events]))
    res = pb.assign_batched(S.view(B, T, E), workspace=ws, out_assign=a, out_perm=perm,
                            out_prices=prices)
    st = res.stats
    counts_ok = bool(torch.all(torch.stack([torch.bincount(a[b].long(), minlength=E)
                                            for b in range(B)]) == T // E))
    BT = B * T
    bytes_aff = BT * d * 2 + E * d * 2 + BT * E * 4 + BT * 4
    bytes_perm = 2 * BT * d * 2 + BT * 4
    bytes_assign = st.bids * (4 * E + 16) + BT * 8
    rl = {"affinity": bytes_aff, "assign": bytes_assign, "permute": bytes_perm}
    small_route = st.engine_bids == 0 and st.bids > 0
    kernel = "small_solve_kernel" if small_route else ENGINE_KERNEL
    launches = eng_launches / args.steps if eng_launches else 0.0
    eng_avg_ms = eng_ms / eng_launches if eng_launches else None
    eng_bytes = ((st.bids if small_route else st.engine_bids) * (4 * E + 16) / launches
                 if launches else 0.0)
    eng_ach = eng_bytes / (eng_avg_ms * 1e-3) / 1e9 if eng_launches else 0.0
    out = {
        "metric": f"tokens assigned/sec, {B} independent problems of T=2048,E=128,d=2048",
        "value": BT * args.steps / wall,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded generator; no dataset or trained weights)",
        "config": {"workload": f"t2048-e128-d2048-worker x {B}", "B": B, "T": T, "E": E, "d": d,
                   "shuffle": shuffle is not None},
        "roofline": {"kernel": kernel, "bound": "hbm", "achieved": eng_ach,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": eng_ach / HBM_PEAK_GBS,
                     "traffic": None,
                     "bytes_model": "bids x (4E + 16) B over all problems: an upper bound",
                     "algorithmic_bytes_per_launch": eng_bytes, "avg_launch_ms": eng_avg_ms,
                     "launches_per_step": launches,
                     "share_of_step": eng_ms / args.steps / gpu_ms if gpu_ms > 0 else None},
        "per_call_ms": {k: round(v, 4) for k, v in per_call_ms.items()},
        "gpu_ms_per_step": gpu_ms,
        "per_call_roofline": {k: {"bound": "hbm",
                                  "achieved": round(v / (per_call_ms[k] * 1e-3) / 1e9, 2),
                                  "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                  "frac": round(v / (per_call_ms[k] * 1e-3) / 1e9 / HBM_PEAK_GBS,
                                                4)}
                              for k, v in rl.items()},
        "assign_stats": {"phases": st.phases, "rounds_max": st.rounds, "bids": st.bids,
                         "engine_bids": st.engine_bids, "converged": st.converged,
                         "dual_gap": st.dual_gap, "eps_final": st.eps_final},
        "balanced_problems": counts_ok,
    }
    if not args.no_cpu_baseline:
        # A bounded sample: the oracle on the first problems of the batch.
        sample = []
        for b in range(min(B, 16)):
            sample.append(wl.make_inputs(dataclasses.replace(base, seed=base.seed + 1000 * b)))
        out["cpu_baseline"] = cpu_baseline_many(sample)
    print(json.dumps(out), flush=True)


def cpu_baseline_many(inps) -> dict:
    """The CPU oracle over several independent problems (one pass each)."""
    import oracle
    t0 = time.perf_counter()
    tokens = 0
    for inp in inps:
        S = oracle.affinity(inp.H, inp.W)
        a, _, _ = oracle.solve_ssp(S)
        oracle.gather(inp.H_store, oracle.stable_perm(a, inp.wl.E))
        tokens += inp.wl.T
    spent = time.perf_counter() - t0
    return {"value": tokens / spent, "unit": "tokens/s", "cores": _blas_threads(),
            "kind": "oracle",
            "sample": f"{len(inps)} problems of {inps[0].wl.name} (the first of the batch), "
                      f"one pass each: fp64 affinity, SSP solve, stable sort vector, gather"}


def _blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        return int(max((i.get("num_threads", 1) for i in threadpool_info()), default=1))
    except Exception:  # threadpoolctl missing: report the host count
        return os.cpu_count() or 1


def cpu_baseline(inp: wl.Inputs, min_s: float = 10.0, budget_s: float = 30.0) -> dict:
    """The CPU oracle (as it stands) on the same workload: fp64 affinity
    (BLAS, all host threads), exact successive-shortest-path solve (one
    thread), stable sort vector and row gather. Repeated until about min_s
    seconds of CPU work (a pass that would end past budget_s is not started)."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # threadpoolctl missing: report the host count
        blas_threads = os.cpu_count() or 1
    T, E = inp.wl.T, inp.wl.E
    reps, spent = 0, 0.0
    parts = {"affinity_s": 0.0, "solve_s": 0.0, "permute_s": 0.0}
    while reps == 0 or (spent < min_s and spent + spent / reps <= budget_s):
        t0 = time.perf_counter()
        S = oracle.affinity(inp.H, inp.W)
        t1 = time.perf_counter()
        a, _, _ = oracle.solve_ssp(S)
        t2 = time.perf_counter()
        perm = oracle.stable_perm(a, E)
        oracle.gather(inp.H_store, perm)
        t3 = time.perf_counter()
        parts["affinity_s"] += t1 - t0
        parts["solve_s"] += t2 - t1
        parts["permute_s"] += t3 - t2
        spent += t3 - t0
        reps += 1
    per = {k: v / reps for k, v in parts.items()}
    return {
        "value": T * reps / spent,
        "unit": "tokens/s",
        "cores": int(blas_threads),
        "kind": "oracle",
        "sample": f"full workload {inp.wl.name}, {reps} repetition(s); fp64 affinity on "
                  f"{blas_threads} BLAS threads, SSP solve and permute on 1 thread",
        "per_pass_s": {k: round(v, 4) for k, v in per.items()},
        "host_cpu": platform.processor() or platform.machine(),
        "host_cpu_count": os.cpu_count(),
    }


def seed_spread(args, w, n: int) -> dict:
    """The whole step on n seeds of the workload's generator (the given seed
    first, then seed + 1000 i): per seed, the median of a few timed steps."""
    import dataclasses

    import torch

    import paper_2103_16716_amd as pb

    T, E = w.T, w.E
    S = torch.empty((T, E), dtype=torch.float32, device="cuda")
    a = torch.empty(T, dtype=torch.int32, device="cuda")
    perm = torch.empty(T, dtype=torch.int32, device="cuda")
    ws = torch.empty(pb.assign_workspace_size(T, E), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    rows = []
    for i in range(n):
        wi = dataclasses.replace(w, seed=w.seed + 1000 * i)
        inp = wl.make_inputs(wi)
        H = torch.from_numpy(inp.H_store.view(np.int16)).cuda().view(torch.bfloat16) \
            if inp.H_store.dtype == np.uint16 else torch.from_numpy(inp.H_store).cuda()
        W = torch.from_numpy(inp.W_store.view(np.int16)).cuda().view(torch.bfloat16) \
            if inp.W_store.dtype == np.uint16 else torch.from_numpy(inp.W_store).cuda()
        X = torch.empty_like(H)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(5)]

        def step(e=None):
            if e is not None:
                e[0].record(stream)
            pb.affinity(H, W, out=S, stream=stream)
            pb.assign(S, sync_stats=False, workspace=ws, out_assign=a, out_perm=perm,
                      stream=stream)
            if e is not None:
                e[1].record(stream)
            pb.permute(H, perm, out=X, stream=stream)
            if e is not None:
                e[2].record(stream)

        for _ in range(2):
            step()
        for e in ev:
            step(e)
        torch.cuda.synchronize()
        step_ms = float(np.median([e[0].elapsed_time(e[2]) for e in ev]))
        res = pb.assign(S, workspace=ws, out_assign=a, out_perm=perm)
        ok = bool(torch.all(torch.bincount(a.long(), minlength=E) == T // E))
        rows.append({"seed": wi.seed, "step_ms": round(step_ms, 4),
                     "tokens_per_s": round(T / (step_ms * 1e-3)), "rounds": res.stats.rounds,
                     "phases": res.stats.phases, "balanced": ok})
        del H, W, X
    tps = np.array([r["tokens_per_s"] for r in rows], dtype=np.float64)
    return {"seeds": rows, "tokens_per_s_median": float(np.median(tps)),
            "tokens_per_s_min": float(tps.min()), "tokens_per_s_max": float(tps.max()),
            "note": "GPU step time (events) per seed, median of 5 steps"}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the assignment path has no multi-GPU mode "
              "(each GPU solves its own batch independently). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.batch > 1:
        bench_batched(args)
        return
    if args.layer:
        bench_layer(args)
        return

    import torch

    import paper_2103_16716_amd as pb

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    torch.cuda.set_device(0)
    inp = wl.make_inputs(args.workload)
    w = inp.wl
    T, E, d = w.T, w.E, w.d
    bf16 = w.dtype == "bf16"
    tdt = torch.bfloat16 if bf16 else torch.float32

    def to_dev(x):
        if x.dtype == np.uint16:
            return torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)
        return torch.from_numpy(x).cuda()

    H, W = to_dev(inp.H_store), to_dev(inp.W_store)
    S = torch.empty((T, E), dtype=torch.float32, device="cuda")
    a = torch.empty(T, dtype=torch.int32, device="cuda")
    # every timed solve writes its own assignment, checked after the timing
    a_timed = torch.empty((args.steps, T), dtype=torch.int32, device="cuda")
    perm = torch.empty(T, dtype=torch.int32, device="cuda")
    prices = torch.empty(E, dtype=torch.float32, device="cuda")
    ws = torch.empty(pb.assign_workspace_size(T, E), dtype=torch.uint8, device="cuda")
    X = torch.empty((T, d), dtype=tdt, device="cuda")
    Y = torch.empty((T, d), dtype=tdt, device="cuda")
    unpermute = w.name in UNPERMUTE_WORKLOADS

    stream = torch.cuda.current_stream()
    n_ev = 5 if unpermute else 4
    bounded = dict(max_rounds=args.max_rounds, flags=pb.BASE_ASSIGN_GREEDY_FALLBACK) \
        if args.max_rounds > 0 else {}

    def step(evs=None, out_a=None):
        if evs is not None:
            evs[0].record(stream)
        pb.affinity(H, W, out=S, stream=stream)
        if evs is not None:
            evs[1].record(stream)
        pb.assign(S, sync_stats=False, workspace=ws, out_assign=a if out_a is None else out_a,
                  out_perm=perm, out_prices=prices, stream=stream, **bounded)
        if evs is not None:
            evs[2].record(stream)
        pb.permute(H, perm, out=X, stream=stream)
        if evs is not None:
            evs[3].record(stream)
        if unpermute:
            pb.permute(X, perm, inverse=True, out=Y, stream=stream)
            if evs is not None:
                evs[4].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(args.steps)]
    # The library brackets each engine launch with its own events on the same
    # stream (base_timing_enable), so the dominant kernel is timed live.
    pb.timing_enable(64 * args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k], a_timed[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    eng_launches, eng_ms = pb.timing_read()
    pb.timing_enable(0)
    timed_balanced = sum(int(bool(torch.all(torch.bincount(a_timed[k].long(), minlength=E) ==
                                            T // E))) for k in range(args.steps))

    names = ["affinity", "assign", "permute"] + (["unpermute"] if unpermute else [])
    per_call_ms = {n: float(np.mean([ev[i].elapsed_time(ev[i + 1]) for ev in events]))
                   for i, n in enumerate(names)}
    step_ms = np.array([ev[0].elapsed_time(ev[-1]) for ev in events])
    gpu_ms = float(np.mean(step_ms))
    ms_per_step = wall * 1e3 / args.steps

    # Cold caches: a 512 MiB write before each of a few more steps evicts the
    # inputs from L2 and the last-level cache (they stay resident in HBM).
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    cold = []
    for k in range(COLD_STEPS):
        scratch.fill_(k & 0xff)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_ev)]
        step(ev)
        torch.cuda.synchronize()
        cold.append(ev[0].elapsed_time(ev[-1]))
    del scratch

    # Solves with statistics and balance checks on a few more steps: the solve
    # is deterministic, so every repetition must give the same rounds, bids
    # and assignment.
    checked, balanced = 0, 0
    runs = []
    for _ in range(3):
        step()
        res = pb.assign(S, workspace=ws, out_assign=a, out_perm=perm, out_prices=prices,
                        **bounded)
        counts = torch.bincount(a.long(), minlength=E)
        balanced += int(bool(torch.all(counts == T // E)))
        checked += 1
        runs.append((res.stats.rounds, res.stats.bids, a.clone()))
    deterministic = all(r[0] == runs[0][0] and r[1] == runs[0][1] and torch.equal(r[2], runs[0][2])
                        for r in runs)
    assert deterministic, "repeated solves differ"
    st = res.stats

    # Algorithmic traffic per call (bytes), and flops for the GEMM.
    esz = 2 if bf16 else 4
    bytes_aff = T * d * esz + E * d * esz + T * E * 4
    flops_aff = 2.0 * T * E * d
    bytes_perm = 2 * T * d * esz
    bytes_assign = st.bids * (4 * E + 16) + T * 8      # score row + bid key per bid, assign/perm out
    rl = {
        "affinity": ("hbm", bytes_aff / (per_call_ms["affinity"] * 1e-3) / 1e9, HBM_PEAK_GBS,
                     "GB/s", bytes_aff),
        "assign": ("hbm", bytes_assign / (per_call_ms["assign"] * 1e-3) / 1e9, HBM_PEAK_GBS,
                   "GB/s", bytes_assign),
        "permute": ("hbm", bytes_perm / (per_call_ms["permute"] * 1e-3) / 1e9, HBM_PEAK_GBS,
                    "GB/s", bytes_perm),
    }
    if unpermute:
        rl["unpermute"] = ("hbm", bytes_perm / (per_call_ms["unpermute"] * 1e-3) / 1e9,
                           HBM_PEAK_GBS, "GB/s", bytes_perm)
    # The dominant kernel: the engine (the largest part of the assign call).
    # Its modelled bytes per launch are the bids it places times the bytes a
    # bid would need if it read the token's whole score row (4E bytes) plus
    # a 16-byte key and expert, over the launches of one solve. This is an
    # upper bound: most bids read only the token's 64-byte summary, so the
    # counter-measured traffic (when a summary for this source is committed)
    # is reported beside it.
    # On the single-workgroup route (no bid placed by the engine) the timed
    # launches are those of small_solve_kernel, which places every bid.
    small_route = st.engine_bids == 0 and st.bids > 0
    kernel = "small_solve_kernel" if small_route else ENGINE_KERNEL
    kernel_bids = st.bids if small_route else st.engine_bids
    launches_per_solve = eng_launches / args.steps if eng_launches else 0.0
    eng_avg_ms = eng_ms / eng_launches if eng_launches else None
    eng_bytes = (kernel_bids * (4 * E + 16) / launches_per_solve
                 if launches_per_solve else 0.0)
    eng_ach = eng_bytes / (eng_avg_ms * 1e-3) / 1e9 if eng_launches else 0.0
    traffic = None if small_route else measured_traffic(w.name)
    spread = args.seed_spread if args.seed_spread >= 0 else (5 if w.name == wl.HEADLINE else 0)
    seeds_line = seed_spread(args, w, spread) if spread > 0 else None
    out = {
        "metric": f"tokens assigned/sec at T={T},E={E},d={d}",
        "value": T * args.steps / wall,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic (seeded generator; no dataset or trained weights)",
        "config": {"workload": w.name, "T": T, "E": E, "C": T // E, "d": d, "dist": w.dist,
                   "inputs": w.dtype, "scores": "f32",
                   "solver": "f32 auction, eps_final=1e-4",
                   **({"max_rounds": args.max_rounds, "completion": "greedy"}
                      if args.max_rounds > 0 else {}),
                   **({"unpermute": True} if unpermute else {})},
        "roofline": {"kernel": kernel, "bound": "hbm", "achieved": eng_ach,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": eng_ach / HBM_PEAK_GBS,
                     "traffic": traffic,
                     "traffic_achieved_gbs": (traffic / (eng_avg_ms * 1e-3) / 1e9
                                              if traffic and eng_launches else None),
                     "bytes_model": "bids x (4E + 16) B: an upper bound, most bids read a "
                                    "64 B summary instead of the 4E B row",
                     "algorithmic_bytes_per_launch": eng_bytes,
                     "avg_launch_ms": eng_avg_ms, "launches_per_step": launches_per_solve,
                     "share_of_step": eng_ms / args.steps / gpu_ms if gpu_ms > 0 else None},
        "per_call_ms": {k: round(v, 4) for k, v in per_call_ms.items()},
        "gpu_ms_per_step": gpu_ms,
        "step_ms_quantiles": {"p10": float(np.percentile(step_ms, 10)),
                              "median": float(np.median(step_ms)),
                              "p90": float(np.percentile(step_ms, 90))},
        "cold_step_ms_median": float(np.median(cold)),
        "per_call_roofline": {k: {"bound": v[0], "achieved": round(v[1], 2), "peak": v[2],
                                  "unit": v[3], "frac": round(v[1] / v[2], 4)}
                              for k, v in rl.items()},
        "affinity_mfma": {"achieved_tflops": flops_aff / (per_call_ms["affinity"] * 1e-3) / 1e12,
                          "peak_tflops": MFMA_BF16_PEAK_TFLOPS},
        "assign_stats": {"phases": st.phases, "rounds": st.rounds, "bids": st.bids,
                         "bids_per_token": st.bids / T, "engine_bids": st.engine_bids,
                         "eps_final": st.eps_final, "eps_last": st.eps_last,
                         "certified": st.certified, "dual_gap": st.dual_gap,
                         "gap_bound": T * st.eps_final, "converged": st.converged,
                         "fell_back": st.fell_back, "augmentations": st.augmentations},
        "balanced_solves": f"{balanced}/{checked}",
        "balanced_timed_solves": f"{timed_balanced}/{args.steps}",
        "deterministic": deterministic,
    }
    if seeds_line is not None:
        out["seed_spread"] = seeds_line
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(inp)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
